"""The oracle's score of many candidates over worker processes (test
infrastructure, like the oracle itself).

A dense full-size parity check needs the fp64 oracle over hundreds of
thousands of candidates; one process takes minutes, the host's cores take
seconds. Workers are spawned, not forked (the parent has usually initialised
the GPU), import only NumPy and the oracle, and score tiles of candidates
with one BLAS thread each; the tiles come back in candidate order.
"""
import multiprocessing
import os

import numpy as np

_W = {}


def _init(model, cand, ref, Z):
    _W.update(model=model, cand=cand, ref=ref, Z=Z)


def _tile(bounds):
    import oracle as O
    from threadpoolctl import threadpool_limits
    i0, i1 = bounds
    with threadpool_limits(1):
        o = O.score(_W["model"], _W["cand"][i0:i1], _W["ref"], _W["Z"])
    return o["mu"], o["sigma"], o["ehvi"]


def default_workers():
    """The CPU share of this process, at most 16 (one GPU's share of a box)."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def score(model, cand, ref, Z, tile=2048, workers=None):
    """mu, sigma and EHVI of every candidate (cand [M, q, d]) as the oracle's
    score computes them, tile by tile over `workers` processes."""
    cand = np.ascontiguousarray(cand, dtype=np.float64)
    Z = np.ascontiguousarray(Z, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    M = cand.shape[0]
    tiles = [(i, min(i + tile, M)) for i in range(0, M, tile)]
    nw = min(workers or default_workers(), max(1, len(tiles)))
    ctx = multiprocessing.get_context("spawn")
    with ctx.Pool(nw, initializer=_init, initargs=(model, cand, ref, Z)) as pool:
        parts = pool.map(_tile, tiles, chunksize=1)
    return dict(mu=np.concatenate([p[0] for p in parts]),
                sigma=np.concatenate([p[1] for p in parts]),
                ehvi=np.concatenate([p[2] for p in parts]))
