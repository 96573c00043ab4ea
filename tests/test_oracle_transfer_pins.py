"""Pins of the transfer-plan oracle (App. F): the device-mapping cost matrix and the
per-request finish-or-move decisions.

* a hand-worked four-GPU, two-node example with seven requests covering every branch,
* brute force from Python sets and lists on tiny random fleets (tests/brute.py),
* invariants: zero diagonal, non-negative costs, a destination holding all of u's models
  costs only u's state, the link class follows the nodes, more remaining work never makes
  a request stay.
"""
import numpy as np
import pytest

import oracle
from brute import brute_moves, link_ms_per_byte, transfer_mib
from conftest import golden_transfer
from paper_2606_30391_amd import workloads as W


def test_transfer_worked_example_costs():
    inp, d = golden_transfer()
    c = oracle.transfer_costs(inp)
    mib = np.array(d["expected_mib"])
    assert np.array_equal(transfer_mib(inp), mib)
    G = len(mib)
    for u in range(G):
        for v in range(G):
            assert c[u, v] == pytest.approx(mib[u, v] * 1048576 * link_ms_per_byte(inp, u, v), rel=1e-15, abs=0)
    assert c[0, 1] == pytest.approx(1100 * 1048576 * 1e3 / 100e9, rel=1e-12)    # intra-node
    assert c[0, 2] == pytest.approx(2100 * 1048576 * 1e3 / 25e9, rel=1e-12)     # inter-node


def test_transfer_worked_example_moves():
    inp, d = golden_transfer()
    dec, rem, mig = oracle.request_moves(inp)
    bdec, brem, bmig = brute_moves(inp)
    for q, e in enumerate(d["moves"]):
        assert dec[q] == e["decision"] == bdec[q], (q, e["note"])
        assert rem[q] == pytest.approx(float(e["remaining_ms"]), rel=1e-12, abs=0)
        assert mig[q] == pytest.approx(float(e["migrate_ms"]), rel=1e-12, abs=0)


@pytest.mark.parametrize("seed", range(5))
def test_transfer_matches_brute_force(seed):
    rng = np.random.default_rng(9500 + seed)
    for _ in range(30):
        inp = W.make_tiny_transfer(rng)
        c = oracle.transfer_costs(inp)
        mib = transfer_mib(inp)
        G = inp["transfer"]["n_gpus"]
        want = np.array([[mib[u, v] * 1048576 * link_ms_per_byte(inp, u, v) for v in range(G)] for u in range(G)])
        np.testing.assert_allclose(c, want.reshape(G, G), rtol=1e-15, atol=0)
        dec, rem, mig = oracle.request_moves(inp)
        bdec, brem, bmig = brute_moves(inp)
        assert np.array_equal(dec, bdec)
        np.testing.assert_allclose(rem, brem, rtol=1e-15, atol=0)
        np.testing.assert_allclose(mig, bmig, rtol=1e-15, atol=0)


def test_transfer_invariants():
    inp = W.make_transfer(n_gpus=200, requests_per_gpu=8)
    c = oracle.transfer_costs(inp)
    t = inp["transfer"]
    assert np.all(np.diag(c) == 0) and np.all(c >= 0)
    node = t["node"]
    for u in range(0, 200, 7):
        for v in range(0, 200, 5):
            if u == v:
                continue
            cu, cv = int(t["resident"][u, 0]), int(t["resident"][v, 0])
            if cu & ~cv == 0:        # v holds every model of u: only u's state moves
                gbs = t["bw_intra_gbs"] if node[u] == node[v] else t["bw_inter_gbs"]
                assert c[u, v] == pytest.approx(int(t["state_mib"][u]) * 1048576 * 1e3 / (float(np.float32(gbs)) * 1e9),
                                                rel=1e-12)
    # more remaining work never turns a move into a stay
    dec, rem, mig = oracle.request_moves(inp)
    mv = inp["moves"]
    mv["remaining_tokens"] = mv["remaining_tokens"] * 2 + 1
    dec2, _, _ = oracle.request_moves(inp)
    assert np.all((dec <= 0) | (dec2 == dec))
    moved = (dec2 > 0).sum()
    assert moved >= (dec > 0).sum() > 0
