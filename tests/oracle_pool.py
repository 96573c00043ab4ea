"""The oracle over many requests at once: the unchanged single-threaded oracle on chunks of
the request ids, in spawned worker processes (fresh interpreters that never touch the GPU).
Test infrastructure."""
import os

import numpy as np

_INP = None


def _init(inp):
    global _INP
    import oracle
    oracle.lib()
    _INP = inp


def _chunk(sel):
    import oracle
    return oracle.score_placements(_INP, sel)


def score_placements(inp, sel=None, workers=None, timeout=600):
    """oracle.score_placements(inp, sel), computed by `workers` processes (at most 16, the
    CPU share of one GPU on the box)."""
    import multiprocessing as mp
    R = inp["requests"]["n_requests"]
    sel = np.arange(R, dtype=np.int32) if sel is None else np.asarray(sel, np.int32)
    workers = workers or max(1, min(16, os.cpu_count() or 1))
    chunks = [c for c in np.array_split(sel, workers * 4) if len(c)]
    with mp.get_context("spawn").Pool(workers, initializer=_init, initargs=(inp,)) as pool:
        parts = pool.map_async(_chunk, chunks).get(timeout=timeout)
    return tuple(np.concatenate([p[i] for p in parts]) for i in range(3))
