"""Pins for the oracle's front, boxes, HVI, (q)EHVI and argmax."""
import itertools

import numpy as np
import pytest

import oracle as O
from pins import (hv_exact, hv2d_sweep, hv3d_slices, hv_grid_count,
                  front_bruteforce, ehvi_closed_form)


def _front_cloud(n, m, seed):
    r = np.random.default_rng(seed)
    Y = r.standard_normal((n, m))
    ref = Y.min(axis=0) - 0.1
    return Y, ref


# ---- front -----------------------------------------------------------------

@pytest.mark.parametrize("m", [2, 3])
def test_front_matches_bruteforce_and_is_permutation_invariant(m):
    Y, ref = _front_cloud(120, m, seed=m)
    Y[5] = Y[17]                     # an exact duplicate
    Y[40] = Y[41] - 1.0              # a strictly dominated point
    F = O.pareto_front(Y, ref)
    assert sorted(F.tolist()) == front_bruteforce(Y, ref)
    assert np.all(np.diff(Y[F, 0]) >= 0)
    perm = np.random.default_rng(1).permutation(len(Y))
    Fp = O.pareto_front(Y[perm], ref)
    np.testing.assert_array_equal(np.sort(Y[perm][Fp], axis=0), np.sort(Y[F], axis=0))


def test_front_ref_filter_is_strict():
    Y = np.array([[1.0, 0.0], [0.0, 1.0], [0.5, 0.5]])
    F = O.pareto_front(Y, np.array([0.0, 0.0]))
    assert F.tolist() == [2]


# ---- hypervolume by grid counting ----------------------------------------

@pytest.mark.parametrize("m", [2, 3])
def test_box_volume_identity_on_integer_grids(m):
    r = np.random.default_rng(10 + m)
    for _ in range(6):
        P = r.integers(1, 7, size=(8, m))
        ref = np.zeros(m)
        idx = O.pareto_front(P, ref)
        count = hv_grid_count(P, ref)
        assert hv_exact(P, ref) == pytest.approx(count, abs=1e-12)
        lo, hi = O.box_decomposition(P[idx].astype(float), ref)
        U = np.full(m, 7.0)
        vol = np.prod(np.clip(np.minimum(hi, U) - lo, 0, None), axis=1).sum()
        assert vol + count == pytest.approx(np.prod(U - ref), abs=1e-9)


@pytest.mark.parametrize("m", [2, 3])
def test_boxes_are_disjoint_and_cover_the_nondominated_region(m):
    Y, ref = _front_cloud(60, m, seed=20 + m)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    assert np.all(lo >= ref) and np.all(hi > lo)
    pts = np.random.default_rng(3).uniform(ref, Y.max(axis=0) + 0.5, size=(20000, m))
    dominated = np.any(np.all(F[None, :, :] >= pts[:, None, :], axis=2), axis=1)
    inside = np.all((pts[:, None, :] >= lo) & (pts[:, None, :] < hi), axis=2)
    count = inside.sum(axis=1)
    assert np.all(count <= 1)
    np.testing.assert_array_equal(count == 1, ~dominated)


def test_3d_box_count_is_linear_in_front_size():
    Y, ref = _front_cloud(400, 3, seed=4)
    F = Y[O.pareto_front(Y, ref)]
    lo, _ = O.boxes_3d(F, ref)
    assert lo.shape[0] <= 2 * len(F) + 1 + len(F)


# ---- HVI -------------------------------------------------------------------

@pytest.mark.parametrize("m", [2, 3])
def test_hvi_equals_hv_difference(m):
    Y, ref = _front_cloud(80, m, seed=30 + m)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    base = hv_exact(F, ref)
    ys = np.random.default_rng(1).normal(0.5, 1.0, size=(40, m))
    got = O.hvi(ys, lo, hi)
    for i in range(40):
        want = hv_exact(np.vstack([F, ys[i]]), ref) - base
        assert got[i] == pytest.approx(want, rel=1e-10, abs=1e-12)


@pytest.mark.parametrize("m", [2, 3])
def test_hvi_invariants(m):
    Y, ref = _front_cloud(50, m, seed=40 + m)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    r = np.random.default_rng(2)
    ys = r.normal(0.0, 1.5, size=(500, m))
    h = O.hvi(ys, lo, hi)
    assert np.all(h >= 0)
    # points dominated by a front member score zero
    dom = F[r.integers(0, len(F), 100)] - r.uniform(0, 0.3, size=(100, m))
    assert np.all(O.hvi(dom, lo, hi) == 0)
    # monotone in every coordinate
    up = ys + r.uniform(0, 0.2, size=ys.shape)
    assert np.all(O.hvi(up, lo, hi) >= h - 1e-12)
    # empty front: the box [r, y]
    lo0, hi0 = O.box_decomposition(np.zeros((0, m)), ref)
    np.testing.assert_allclose(O.hvi(ys, lo0, hi0), np.prod(np.clip(ys - ref, 0, None), axis=1), rtol=1e-13)


def test_hvi_scales_with_objective_scaling():
    Y, ref = _front_cloud(50, 3, seed=9)
    c = np.array([2.0, 0.5, 3.0])
    F = Y[O.pareto_front(Y, ref)]
    ys = np.random.default_rng(3).normal(0.3, 1.0, size=(30, 3))
    lo, hi = O.box_decomposition(F, ref)
    lo2, hi2 = O.box_decomposition(F * c, ref * c)
    np.testing.assert_allclose(O.hvi(ys * c, lo2, hi2), np.prod(c) * O.hvi(ys, lo, hi), rtol=1e-12, atol=1e-14)


# ---- qHVI ------------------------------------------------------------------

@pytest.mark.parametrize("m,q", [(2, 2), (2, 3), (3, 2), (3, 4)])
def test_qhvi_equals_union_hv_difference(m, q):
    Y, ref = _front_cloud(40, m, seed=50 + m + q)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    base = hv_exact(F, ref)
    r = np.random.default_rng(6)
    for _ in range(15):
        Yq = r.normal(0.5, 1.0, size=(q, m))
        want = hv_exact(np.vstack([F, Yq]), ref) - base
        assert O.qhvi(Yq, lo, hi) == pytest.approx(want, rel=1e-9, abs=1e-12)


def test_qhvi_bounds_and_degenerate_batches():
    Y, ref = _front_cloud(40, 3, seed=77)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    r = np.random.default_rng(8)
    Yq = r.normal(0.4, 1.0, size=(200, 4, 3))
    qh = O.qhvi(Yq, lo, hi)
    single = O.hvi(Yq, lo, hi)                         # [200, 4]
    assert np.all(qh >= single.max(axis=1) - 1e-12)
    assert np.all(qh <= single.sum(axis=1) + 1e-12)
    same = np.repeat(Yq[:, :1, :], 4, axis=1)
    np.testing.assert_allclose(O.qhvi(same, lo, hi), single[:, 0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.qhvi(Yq[:, :1, :], lo, hi), single[:, 0], rtol=0, atol=0)


# ---- MC-EHVI converges to the closed form ----------------------------------

@pytest.mark.parametrize("m", [2, 3])
def test_mc_ehvi_converges_to_closed_form(m):
    Y, ref = _front_cloud(60, m, seed=60 + m)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    mu = np.full((1, m), 0.6)
    sd = np.linspace(0.4, 0.9, m)[None, :]
    cf = ehvi_closed_form(mu[0], sd[0], lo, hi)
    errs = []
    for S in (2 ** 14, 2 ** 18):
        Z = np.random.default_rng(S).standard_normal((S, 1, m))
        ys = mu + sd * Z[:, 0, :]
        h = O.hvi(ys, lo, hi)
        mc = O.ehvi_q1(mu, sd, Z, lo, hi, chunk=1)[0]
        assert mc == pytest.approx(h.mean(), rel=1e-12)
        se = h.std(ddof=1) / np.sqrt(S)
        assert abs(mc - cf) <= 5 * se
        errs.append(abs(mc - cf))
    assert cf > 0


def test_qehvi_with_q1_equals_ehvi_q1():
    Y, ref = _front_cloud(60, 3, seed=71)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    r = np.random.default_rng(0)
    mu = r.normal(0, 1, size=(7, 1, 3))
    sd = r.uniform(0.1, 1.0, size=(7, 1, 3))
    C = np.zeros((7, 3, 1, 1))
    C[:, :, 0, 0] = sd[:, 0, :]
    Z = r.standard_normal((64, 1, 3))
    np.testing.assert_allclose(O.qehvi(mu, C, Z, lo, hi), O.ehvi_q1(mu[:, 0], sd[:, 0], Z, lo, hi), rtol=1e-12)


def test_qehvi_sampling_uses_lower_factor_per_objective():
    """With a fully correlated batch (all members the same point) the
    joint samples coincide and qEHVI equals single-point EHVI."""
    Y, ref = _front_cloud(50, 3, seed=81)
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    r = np.random.default_rng(4)
    mu1 = r.normal(0, 1, size=(3,))
    sd = r.uniform(0.2, 1.0, size=(3,))
    mu = np.broadcast_to(mu1, (1, 4, 3)).copy()
    C = np.zeros((1, 3, 4, 4))
    C[0, :, :, 0] = sd[:, None]       # rank one: every member = mu + sd z_0
    Z = r.standard_normal((128, 4, 3))
    e4 = O.qehvi(mu, C, Z, lo, hi)[0]
    e1 = O.ehvi_q1(mu1[None], sd[None], Z[:, :1, :], lo, hi)[0]
    assert e4 == pytest.approx(e1, rel=1e-12)


# ---- argmax ----------------------------------------------------------------

def test_argmax_semantics():
    v = np.array([0.1, 0.5, np.nan, 0.5, 0.2])
    assert O.argmax(v) == (1, 0.5)
    assert O.argmax(np.array([np.nan, np.nan]))[0] == -1
    assert O.argmax(np.array([-np.inf, -1.0]))[0] == 1
    r = np.random.default_rng(1).random(1000)
    assert O.argmax(r)[0] == int(np.argmax(r))


# ---- end-to-end on a tiny configuration -----------------------------------

def test_score_pipeline_small_config_consistency():
    import bo_inputs as bi
    wl = bi.make_config(0, seed=0, M=32)
    mdl = O.fit(wl.X, wl.Y, wl.lengthscale, wl.outputscale, wl.noise)
    out = O.score(mdl, wl.cand, wl.ref, wl.Z)
    assert out["ehvi"].shape == (32,)
    assert np.all(out["ehvi"] >= 0)
    # same estimator recomputed from its parts with the generic box form
    ys = out["mu"][:, 0, None, :] + out["sigma"][:, 0, None, :] * wl.Z.astype(float)[None, :, 0, :]
    np.testing.assert_allclose(out["ehvi"], O.hvi(ys, out["lo"], out["hi"]).mean(axis=1), rtol=1e-12)


def test_pooled_oracle_score_matches_one_process():
    """The tile-parallel oracle used by the dense full-size parity check
    returns the one-process score, in candidate order."""
    import bo_inputs as bi
    import oracle_pool
    wl = bi.make_config(0, seed=1, M=700)
    model = O.fit(wl.X, wl.Y, wl.lengthscale, wl.outputscale, wl.noise)
    one = O.score(model, wl.cand.astype(np.float64), wl.ref, wl.Z.astype(np.float64))
    many = oracle_pool.score(model, wl.cand, wl.ref, wl.Z, tile=128, workers=2)
    for k in ("mu", "sigma", "ehvi"):
        assert many[k].shape == one[k].shape
        np.testing.assert_allclose(many[k], one[k], rtol=1e-12, atol=1e-14)
