"""GPU parity of the transfer plan (App. F): the device-mapping cost matrix and the
in-flight requests' finish-or-move decisions, through the C ABI against the CPU oracle.
Both sides evaluate the same float64 expressions, so costs, times (rounded to float32) and
decisions must match exactly."""
import sys

import numpy as np
import pytest

import oracle
from conftest import golden_transfer
from oracle.check import check_transfer
from paper_2606_30391_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def parity(inp, label=""):
    from paper_2606_30391_amd import festina as F
    F.lib()
    say(f"[gpu] transfer {label}: G={inp['transfer']['n_gpus']} M={inp['n_models']} Q={inp['moves']['n_requests']}")
    dt = F.DeviceTransfer(inp, "cuda")
    dt.run_costs()
    dt.run_moves()
    torch.cuda.synchronize()
    c, d, r, m = dt.results()
    rep = check_transfer(oracle.transfer_costs(inp), oracle.request_moves(inp), c, (d, r, m))
    say(f"      {rep}; decisions {np.bincount(d + 1, minlength=4).tolist()}")
    assert rep.ok, str(rep)
    return c, d


def test_transfer_full_fleet():
    c, d = parity(W.make_transfer(), label="2048 GPUs")
    assert (d == 1).sum() > 1000 and (d == 0).sum() > 1000


def test_transfer_worked_example():
    inp, g = golden_transfer()
    c, d = parity(inp, label="worked example")
    assert list(d) == [m["decision"] for m in g["moves"]]


@pytest.mark.parametrize("G,M", [(1, 1), (3, 2), (4, 1), (5, 7), (129, 33), (1000, 31), (1001, 70), (2050, 32)])
def test_transfer_shapes(G, M):
    """Row lengths not a multiple of 4 (scalar stores), several residency words, one GPU."""
    rng = np.random.default_rng(2000 + G)
    parity(W.make_tiny_transfer(rng, G=G, M=M, NS=3, NF=4, Q=3 * G + 5), label="shapes")


def test_transfer_invalid_requests():
    rng = np.random.default_rng(2100)
    inp = W.make_tiny_transfer(rng, G=16, M=3, NS=2, NF=3, Q=200)
    mv, pl = inp["moves"], inp["plan"]
    mv["src"][:10] = 16
    mv["model"][10:20] = 3
    mv["context_tokens"][20:30] = 0
    mv["remaining_tokens"][30:40] = -1
    mv["kv_kib"][40:45] = -1
    pl["sm_cur"][0] = 5
    pl["dest"][1] = 40
    c, d = parity(inp, label="invalid requests")
    assert np.all(d[:45] == -1)


def test_transfer_unaligned_cost_matrix():
    """A cost buffer that is not 16-byte aligned takes the scalar stores."""
    from paper_2606_30391_amd import festina as F
    inp = W.make_tiny_transfer(np.random.default_rng(2200), G=64, M=5, Q=0)
    dt = F.DeviceTransfer(inp, "cuda")
    buf = torch.empty(64 * 64 + 1, dtype=torch.float32, device="cuda")
    F.festina_transfer_costs(dt.transfer, buf[1:])
    torch.cuda.synchronize()
    got = buf[1:].cpu().numpy().reshape(64, 64)
    assert np.array_equal(got, oracle.transfer_costs(inp).astype(np.float32))
