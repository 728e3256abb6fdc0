"""GPU: the noisy preparation's per-draw fronts and box decompositions for
three objectives (k_sample_front3, through bo_draw_fronts3_test), on values
chosen to exercise its rules: exact duplicates, equal coordinates in every
objective, points on the reference planes, thresholds.

Fronts are index work and must equal the oracle's index sets exactly. Boxes
have no unique form, so the decomposition is checked by what it is for: the
hypervolume improvement of probe points (grid points, front points, random
points) summed over the device boxes equals the oracle's over its own
decomposition, and the boxes are disjoint and above ref.
"""
import numpy as np
import pytest

import oracle as O

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


def _device_boxes(b):
    lo = b[:, :3].astype(np.float64)
    hi = lo + b[:, 3:].astype(np.float64)       # inf widths stay inf
    return lo, hi


def _check(F, ref, lower=None, exact=True):
    """exact: small-integer data, whose boxes are exact in fp32; otherwise
    the boxes' fp32 (lo, width) form rounds each side once (relative 2^-24),
    which bounds the HVI difference well inside 1e-6 relative."""
    import torch
    import paper_2602_10729_amd as bo
    fronts, boxes = bo.draw_fronts3_test(torch.from_numpy(F).cuda(), ref, lower)
    ref64 = np.asarray(ref, dtype=np.float64)
    r = np.random.default_rng(7)
    for s in range(F.shape[0]):
        Fs = F[s]
        keep = np.arange(Fs.shape[0])
        if lower is not None:
            keep = keep[np.all(Fs >= np.asarray(lower, dtype=np.float64), axis=1)]
        want = keep[O.pareto_front(Fs[keep], ref64)]
        assert np.array_equal(fronts[s], want), (s, fronts[s], want)
        lo, hi = _device_boxes(boxes[s])
        assert np.all(lo >= ref64 - 0.0) and np.all(hi > lo)
        olo, ohi = O.box_decomposition(Fs[want], ref64)
        # probes: grid points (ties with the data), the front, random points
        g = np.arange(-1.0, 6.0, 0.5)
        grid = np.stack(np.meshgrid(g, g, g, indexing="ij"), -1).reshape(-1, 3)
        probes = np.concatenate([grid, Fs[want], r.uniform(-1, 6, (200, 3))])
        got = O.hvi(probes, lo, hi)
        exp = O.hvi(probes, olo, ohi)
        if exact:
            np.testing.assert_allclose(got, exp, rtol=1e-12, atol=1e-12)
        else:
            # each side of a box is off by at most one fp32 rounding of its
            # coordinates (2^-23 of the larger finite end); the HVI moves by at
            # most that times the other two extents, summed over the boxes
            fin = np.where(np.isfinite(hi), np.abs(hi), 0.0)
            dk = 2.0 ** -23 * np.maximum(np.abs(lo), fin)            # [B, 3]
            ext = np.maximum(np.minimum(probes[:, None, :], hi) - lo, 0.0)   # [P, B, 3]
            ext = ext + dk
            other = np.stack([ext[..., 1] * ext[..., 2], ext[..., 0] * ext[..., 2],
                              ext[..., 0] * ext[..., 1]], -1)
            bound = np.sum(dk * other, axis=(1, 2)) + 1e-12
            assert np.all(np.abs(got - exp) <= bound), float(np.max(np.abs(got - exp) / bound))
        # disjoint: the boxes' volumes inside a bounding box add up to the
        # measure of the region they cover there (the HVI of its corner)
        top = np.array([[6.0, 6.0, 6.0]])
        vol = np.sum(np.prod(np.maximum(np.minimum(top, hi) - lo, 0.0), axis=1))
        np.testing.assert_allclose(vol, O.hvi(top, olo, ohi)[0], rtol=1e-12 if exact else 1e-5)


def test_fronts_and_boxes_with_ties():
    _announce("fronts3 ties")
    r = np.random.default_rng(11)
    S, n = 24, 157
    F = r.integers(0, 5, size=(S, n, 3)).astype(np.float64)
    F[:, 10:20] = F[:, 0:10]                      # exact duplicates of lower indices
    F[3] = 2.0                                    # every point equal
    F[4, :, 0] = 1.0                              # one objective constant
    F[5, :, 2] = np.arange(n) % 3                 # heavy ties in the sweep order
    _check(F, [0.0, 0.0, 0.0])
    _check(F, [1.0, 0.5, 0.0])                    # points on the reference planes drop out


def test_fronts_and_boxes_continuous_and_thresholds():
    _announce("fronts3 continuous, thresholds")
    r = np.random.default_rng(12)
    S, n = 16, 2048
    F = r.standard_normal((S, n, 3))
    F[1] = -10.0                                  # nothing above ref: one box
    _check(F, [-2.0, -2.0, -2.0], exact=False)
    _check(F, [-2.0, -2.0, -2.0], lower=[-0.5, -np.inf, 0.25], exact=False)


def test_nonfinite_value_is_an_error():
    import torch
    import paper_2602_10729_amd as bo
    _announce("fronts3 non-finite")
    F = np.zeros((2, 9, 3))
    F[1, 4, 2] = np.inf
    with pytest.raises(bo.BoError) as ei:
        bo.draw_fronts3_test(torch.from_numpy(F).cuda(), [-1.0, -1.0, -1.0])
    assert ei.value.name == "BO_ERR_NONFINITE_INPUT"
