"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Every case prints its name, seed and shape before touching the GPU so a
failing run identifies itself.
"""
import numpy as np
import pytest

import bo_inputs as bi
import oracle as O
from gpu_util import (TOL_MU, TOL_SIGMA, TOL_EHVI, gpu_run, oracle_fit,
                      oracle_score, assert_close, check_argmax, near_var_tol, to_dev)

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


def _full_parity(wl, g, o):
    assert np.array_equal(g["front"], O.nondominated(wl.Y.astype(np.float64))[
        np.argsort(wl.Y.astype(np.float64)[O.nondominated(wl.Y.astype(np.float64)), 0], kind="stable")])
    assert_close(g["mu"], o["mu"], TOL_MU, "mu")
    assert_close(g["sigma"], o["sigma"], TOL_SIGMA, "sigma")
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi")
    check_argmax(g["idx"], o["ehvi"])
    assert g["val"] == g["ehvi"][g["idx"]]


# configs at sizes the oracle finishes in seconds; M chosen ragged against
# the 16/32-point tiles and the 256-candidate EHVI blocks
SMALL = [(0, 4096), (1, 3001), (2, 2003), (4, 61)]


@pytest.mark.parametrize("cfg,M", SMALL)
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_small_config_parity(cfg, M, seed):
    _announce("small", cfg, seed, M)
    wl = bi.make_config(cfg, seed=seed, M=M)
    g = gpu_run(wl)
    o = oracle_score(oracle_fit(wl), wl)
    _full_parity(wl, g, o)


def test_config1_full_size_elementwise():
    _announce("config1 full", 0)
    wl = bi.make_config(1, seed=0)
    g = gpu_run(wl)
    o = oracle_score(oracle_fit(wl), wl)
    _full_parity(wl, g, o)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_config2_full_size_dense(seed):
    """Every one of config 2's 262,144 candidates element by element: the
    oracle runs over the host's cores (spawned workers, one BLAS thread each)."""
    import oracle_pool
    _announce("config2 full dense", seed)
    wl = bi.make_config(2, seed=seed)
    g = gpu_run(wl)
    o = oracle_pool.score(oracle_fit(wl), wl.cand, wl.ref, wl.Z)
    _full_parity(wl, g, o)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_config3_full_size_dense(seed):
    """The headline workload, all 1,048,576 candidates element by element
    (mu, sigma, EHVI) and the argmax rule, the oracle over the host's cores
    as for config 2. The benchmark's call (no mu/sigma outputs: the same
    launches into the model's workspace) gives bit for bit the same EHVI."""
    import torch
    import oracle_pool
    import paper_2602_10729_amd as bo
    _announce("config3 full dense", seed)
    wl = bi.make_config(3, seed=seed)
    g = gpu_run(wl)
    e = bo.score(g["model"], to_dev(wl.cand), wl.ref, to_dev(wl.Z))
    torch.cuda.synchronize()
    assert np.array_equal(e.cpu().numpy(), g["ehvi"])
    o = oracle_pool.score(oracle_fit(wl), wl.cand, wl.ref, wl.Z)
    _full_parity(wl, g, o)


def _sampled_full_size(cfg, nsample, seed=0):
    wl = bi.make_config(cfg, seed=seed)
    g = gpu_run(wl)
    M = wl.M
    tile = 32 if wl.n <= 1024 else 16
    pts_per_tile = tile // wl.q
    r = np.random.default_rng(99)
    edges = [0, 1, M - 1, M - 2, pts_per_tile - 1, pts_per_tile, 255, 256, M // 2]
    idx = np.unique(np.concatenate([edges, r.integers(0, M, nsample)]))
    model = oracle_fit(wl)
    o = oracle_score(model, wl, cand=wl.cand[idx])
    assert_close(g["mu"][idx], o["mu"], TOL_MU, "mu (sampled)")
    assert_close(g["sigma"][idx], o["sigma"], TOL_SIGMA, "sigma (sampled)")
    assert_close(g["ehvi"][idx], o["ehvi"], TOL_EHVI, "ehvi (sampled)")
    # argmax: any candidate the oracle could rank first has a GPU value
    # within the EHVI tolerance of the GPU maximum; score that pool exactly
    e = g["ehvi"].astype(np.float64)
    top = e.max()
    pool = np.nonzero(e >= top - 2 * (TOL_EHVI[0] * abs(top) + TOL_EHVI[1]) - 1e-3 * abs(top))[0]
    assert pool.size < 4096, pool.size
    op = oracle_score(model, wl, cand=wl.cand[pool])
    assert_close(e[pool], op["ehvi"], TOL_EHVI, "ehvi (top pool)")
    check_argmax(g["idx"], op["ehvi"], idx_pool=pool)
    assert g["idx"] == int(np.argmax(g["ehvi"]))
    return wl, g


def test_config2_full_size_sampled():
    _announce("config2 full sampled", 0)
    _sampled_full_size(2, 400)


def test_config3_full_size_sampled():
    _announce("config3 full sampled", 0)
    _sampled_full_size(3, 400)


def test_config4_full_size_sampled():
    _announce("config4 full sampled", 0)
    _sampled_full_size(4, 256)


@pytest.mark.parametrize("cfg", [0, 2, 4])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_near_data_candidates(cfg, seed):
    """Candidates at distance ~0.01 from observations: large k*, the solve
    does real work and sigma approaches the noise level, where
    sigma^2 = k(x,x) - |v|^2 cancels. sigma is compared through the variance
    with an absolute bound, NEAR_VAR_ULPS units of 2^-24 of the prior variance
    (twice the worst error these cases show); mu and the EHVI at the usual
    bar. The worst error/bound ratios are logged."""
    _announce("near-data", cfg, seed)
    wl = bi.make_config(cfg, seed=seed, M=8)
    cand = bi.near_data_candidates(wl, 512 if cfg != 4 else 64, scale=0.01)
    g = gpu_run(wl, cand=cand)
    o = oracle_score(oracle_fit(wl), wl, cand=cand)
    assert_close(g["mu"], o["mu"], TOL_MU, f"mu near data cfg{cfg} seed{seed}")
    assert_close(g["sigma"] ** 2, o["sigma"] ** 2, near_var_tol(1.0),
                 f"variance near data cfg{cfg} seed{seed}")
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, f"ehvi near data cfg{cfg} seed{seed}")


def test_small_models_and_odd_shapes():
    r = np.random.default_rng(5)
    for n, d in [(1, 3), (2, 1), (37, 5), (130, 7), (17, 32)]:
        _announce("odd shape", n, d)
        wl = bi.make_config(0, seed=1, M=50)
        X = r.random((n, d)).astype(np.float32)
        Y = r.standard_normal((n, 2)).astype(np.float32)
        wl.X, wl.Y, wl.d, wl.n = X, Y, d, n
        wl.lengthscale = r.uniform(0.2, 0.8, size=(2, d)).astype(np.float32)
        wl.cand = r.random((77, 1, d)).astype(np.float32)
        wl.ref = (Y.astype(np.float64).min(0) - 0.1).astype(np.float32)
        g = gpu_run(wl)
        o = oracle_score(oracle_fit(wl), wl)
        assert_close(g["mu"], o["mu"], TOL_MU, f"mu n={n} d={d}")
        assert_close(g["sigma"], o["sigma"], TOL_SIGMA, f"sigma n={n} d={d}")
        assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, f"ehvi n={n} d={d}")


def test_ragged_three_objective_fit():
    """n = 700 (11 fit blocks, a padded tail in the last one) with three
    objectives and q = 4: the Gram matrix in two column parts, the padded
    rows of the factor and of the row-block scales, element by element."""
    for seed in (0, 1):
        _announce("ragged m=3", seed)
        wl = bi.make_config(4, seed=seed, M=37)
        wl.X, wl.Y, wl.n = wl.X[:700].copy(), wl.Y[:700].copy(), 700
        g = gpu_run(wl)
        o = oracle_score(oracle_fit(wl), wl)
        _full_parity(wl, g, o)


def _m52_root(target):
    """Distance r with (1 + sqrt5 r + 5 r^2 / 3) exp(-sqrt5 r) = target (fp64
    bisection; the correlation falls monotonically in r)."""
    lo, hi = 0.0, 10.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        v = (1 + 5 ** 0.5 * mid + 5 * mid * mid / 3) * np.exp(-(5 ** 0.5) * mid)
        lo, hi = (mid, hi) if v > target else (lo, mid)
    return 0.5 * (lo + hi)


def test_kernel_values_at_fp16_rounding_midpoints():
    """Regression: each kernel value is split into fp16 halves hi + lo for
    the triangle's matrix-core products. Both halves must come from one value;
    a split whose high half is rounded from a different representation than
    the one the low half is taken against is off by one fp16 ulp exactly when
    the value lies at an fp16 rounding midpoint. One training point at the
    origin (unit lengthscale, unit scale), and candidates on consecutive fp32
    steps across the distances where k(x*, x) crosses the midpoints
    0.5517578125 + 2^-12 (near pair: exact differences) and 0.5 + 2^-12
    (r^2 > 1: the distance expansion)."""
    _announce("fp16 midpoints", 1, 1)
    wl = bi.make_config(0, seed=1, M=50)
    wl.X = np.zeros((1, 1), np.float32)
    wl.Y = np.array([[0.3, -0.2]], np.float32)
    wl.d, wl.n = 1, 1
    wl.lengthscale = np.ones((2, 1), np.float32)
    wl.outputscale = np.ones(2, np.float32)
    wl.noise = np.full(2, 1e-3, np.float32)
    steps = np.arange(-2048, 2048, dtype=np.int32)
    cands = []
    for mid in (0.5517578125 + 2.0 ** -12, 0.5 + 2.0 ** -12):
        r0 = np.float32(_m52_root(mid))
        cands.append((r0.view(np.int32) + steps).view(np.float32))
    wl.cand = np.concatenate(cands).reshape(-1, 1, 1)
    wl.ref = (wl.Y.astype(np.float64).min(0) - 0.1).astype(np.float32)
    g = gpu_run(wl)
    o = oracle_score(oracle_fit(wl), wl)
    assert_close(g["mu"], o["mu"], TOL_MU, "mu at fp16 midpoints")
    assert_close(g["sigma"], o["sigma"], TOL_SIGMA, "sigma at fp16 midpoints")


def test_translation_invariance_of_the_posterior():
    """The Matern kernel is stationary, so shifting the training points and
    the candidates by one offset must not change the result beyond what fp32
    inputs carry. Squared distances come from |c|^2 + |x|^2 - 2c.x over
    coordinates centred on the training mean, so large offsets must not reach
    the expansion's error. Each shifted run is held to the oracle's bar on the
    same (fp32) shifted inputs: offset 3 with near-data candidates included,
    offset 100 (scaled coordinates up to 1000) on the config's candidates."""
    for off, with_near in ((3.0, True), (100.0, False)):
        _announce("translation", off, with_near)
        wl = bi.make_config(1, seed=2, M=1500)
        if with_near:
            wl.cand = np.concatenate([wl.cand, bi.near_data_candidates(wl, 500, scale=0.01)], 0)
        wl.cand = (wl.cand.astype(np.float64) + off).astype(np.float32)
        wl.X = (wl.X.astype(np.float64) + off).astype(np.float32)
        g = gpu_run(wl)
        o = oracle_score(oracle_fit(wl), wl)
        assert_close(g["mu"], o["mu"], TOL_MU, f"mu offset {off}")
        assert_close(g["sigma"], o["sigma"], TOL_SIGMA, f"sigma offset {off}")


def test_q2_path_and_three_objectives_q1():
    """q = 2 (pairs) with m = 2, and m = 3 with q = 1, built from config 4's
    observations."""
    base = bi.make_config(4, seed=0, M=16)
    r = np.random.default_rng(3)
    for q, m in [(2, 2), (1, 3), (2, 3), (4, 2)]:
        _announce("q/m variant", q, m)
        wl = bi.make_config(4, seed=0, M=16)
        wl.Y = base.Y[:, :m].copy()
        wl.m = m
        wl.lengthscale = base.lengthscale[:m].copy()
        wl.outputscale = base.outputscale[:m].copy()
        wl.noise = base.noise[:m].copy()
        wl.ref = (wl.Y.astype(np.float64).min(0) - 0.1).astype(np.float32)
        wl.q = q
        wl.cand = r.random((40, q, wl.d)).astype(np.float32)
        wl.Z = r.standard_normal((256, q, m)).astype(np.float32)
        g = gpu_run(wl)
        o = oracle_score(oracle_fit(wl), wl)
        assert_close(g["mu"], o["mu"], TOL_MU, "mu")
        assert_close(g["sigma"], o["sigma"], TOL_SIGMA, "sigma")
        assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi")


def test_q4_marginals_match_q1_path():
    _announce("q4 vs q1 marginals")
    wl = bi.make_config(4, seed=1, M=40)
    g4 = gpu_run(wl)
    flat = wl.cand.reshape(-1, 1, wl.d)
    Z1 = wl.Z[:, :1, :].copy()
    g1 = gpu_run(wl, cand=flat, Z=Z1)
    np.testing.assert_allclose(g4["mu"].reshape(-1, wl.m), g1["mu"][:, 0, :], rtol=0, atol=0)
    np.testing.assert_allclose(g4["sigma"].reshape(-1, wl.m), g1["sigma"][:, 0, :], rtol=1e-5, atol=1e-6)


def test_empty_front_and_extreme_reference():
    _announce("empty front")
    wl = bi.make_config(0, seed=0, M=300)
    ref = (wl.Y.astype(np.float64).max(0) + 0.5).astype(np.float32)   # above every point
    g = gpu_run(wl, ref=ref)
    o = oracle_score(oracle_fit(wl), wl, ref=ref)
    assert o["lo"].shape[0] == 1
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi with empty front")


def test_single_sample_and_single_candidate():
    _announce("S=1, M=1")
    wl = bi.make_config(1, seed=2, M=1)
    Z = wl.Z[:1].copy()
    g = gpu_run(wl, Z=Z)
    o = oracle_score(oracle_fit(wl), wl, Z=Z)
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi S=1")
    assert g["idx"] == 0


def test_zero_candidates_is_noop():
    import torch
    import paper_2602_10729_amd as bo
    _announce("M=0")
    wl = bi.make_config(0, seed=0, M=4)
    model = bo.fit(to_dev(wl.X), to_dev(wl.Y), wl.lengthscale, wl.outputscale, wl.noise)
    cand = torch.empty((0, 1, wl.d), dtype=torch.float32, device="cuda")
    e = bo.score(model, cand, wl.ref, to_dev(wl.Z))
    idx, val = bo.argmax(e)
    torch.cuda.synchronize()
    assert e.numel() == 0 and int(idx.item()) == -1 and np.isnan(float(val.item()))


def test_deterministic_repeat():
    _announce("determinism cfg2")
    wl = bi.make_config(2, seed=0, M=5000)
    a = gpu_run(wl)
    b = gpu_run(wl)
    for k in ("mu", "sigma", "ehvi"):
        assert np.array_equal(a[k], b[k]), k
    assert a["idx"] == b["idx"]


def test_score_reuses_model_with_new_reference_point():
    import torch
    import paper_2602_10729_amd as bo
    _announce("ref change")
    wl = bi.make_config(0, seed=0, M=500)
    model = bo.fit(to_dev(wl.X), to_dev(wl.Y), wl.lengthscale, wl.outputscale, wl.noise)
    om = oracle_fit(wl)
    c, z = to_dev(wl.cand), to_dev(wl.Z)
    for shift in (0.0, 0.3, -0.2, 0.0):
        ref = (wl.ref + shift).astype(np.float32)
        e = bo.score(model, c, ref, z)
        torch.cuda.synchronize()
        o = oracle_score(om, wl, ref=ref)
        assert_close(e.cpu().numpy(), o["ehvi"], TOL_EHVI, f"ehvi ref shift {shift}")


def test_low_dimension_batches():
    """d <= 4 (one float4 of coordinates) with q = 2 and 4: every column of a
    64-point tile, including the prior cross-covariances of batch mates kept
    next to the staging area."""
    r = np.random.default_rng(31)
    # lengthscales short enough for a well-conditioned K (cond < 50)
    for d, q, n, lo, hi in [(3, 2, 40, 0.05, 0.12), (4, 4, 40, 0.08, 0.16), (2, 4, 32, 0.03, 0.06)]:
        _announce("low-d batches", d, q)
        wl = bi.make_config(0, seed=1, M=8)
        X = r.random((n, d)).astype(np.float32)
        Y = r.standard_normal((n, 2)).astype(np.float32)
        wl.X, wl.Y, wl.d, wl.n, wl.q = X, Y, d, n, q
        wl.lengthscale = r.uniform(lo, hi, size=(2, d)).astype(np.float32)
        wl.cand = r.random((300, q, d)).astype(np.float32)
        wl.Z = r.standard_normal((128, q, 2)).astype(np.float32)
        wl.ref = (Y.astype(np.float64).min(0) - 0.1).astype(np.float32)
        g = gpu_run(wl)
        o = oracle_score(oracle_fit(wl), wl)
        assert_close(g["mu"], o["mu"], TOL_MU, f"mu d={d} q={q}")
        assert_close(g["sigma"], o["sigma"], TOL_SIGMA, f"sigma d={d} q={q}")
        assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, f"ehvi d={d} q={q}")


@pytest.mark.parametrize("cfg,shift", [(2, 5), (4, 3)])
def test_tile_position_invariance(cfg, shift):
    """A candidate's results do not depend on where it falls in a tile: the
    same points scored from an offset start (every tile boundary moves) are
    bitwise identical."""
    _announce("tile invariance", cfg, shift)
    wl = bi.make_config(cfg, seed=0, M=1000 if cfg == 2 else 120)
    a = gpu_run(wl)
    wl2 = bi.make_config(cfg, seed=0, M=1000 if cfg == 2 else 120)
    wl2.cand = wl.cand[shift:].copy()
    wl2.M = wl.M - shift
    b = gpu_run(wl2)
    for k in ("mu", "sigma", "ehvi"):
        assert np.array_equal(a[k][shift:], b[k]), k
