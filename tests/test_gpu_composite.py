"""GPU parity of the composite surrogate kernel (bo_fit_composite + bo_score)
against the fp64 oracle."""
import numpy as np
import pytest

import bo_inputs as bi
from gpu_util import (TOL_MU, TOL_SIGMA, TOL_EHVI, gpu_run, oracle_fit, oracle_score,
                      assert_close, check_argmax, to_dev, near_var_tol, log_ratio)

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("cfg,M,seed,d_route,q", [(2, 2003, 0, None, 1), (2, 2003, 1, None, 1),
                                                  (1, 3001, 0, 5, 1), (0, 777, 2, 2, 1),
                                                  (4, 300, 0, 9, 1), (4, 61, 0, None, 4),
                                                  (0, 501, 1, 2, 2), (2, 333, 2, None, 4)])
def test_composite_parity(cfg, M, seed, d_route, q):
    wl = bi.make_config(cfg, seed=seed, M=M * q if q != bi.CONFIGS[cfg]["q"] else M)
    if wl.q != q:   # re-batch the candidate stream (config 4's points as singles or pairs)
        wl.cand = wl.cand.reshape(-1, wl.d)[:M * q].reshape(M, q, wl.d).copy()
        wl.Z = np.random.default_rng(seed + 5).standard_normal((wl.S, q, wl.m)).astype(np.float32)
        wl.q, wl.M = q, M
    comp = bi.composite_hyperparameters(wl, d_route)
    _announce("composite", cfg, seed, M, comp.d_route, q)
    g = gpu_run(wl, comp=comp)
    o = oracle_score(oracle_fit(wl, comp), wl)
    assert_close(g["mu"], o["mu"], TOL_MU, "mu")
    assert_close(g["sigma"], o["sigma"], TOL_SIGMA, "sigma")
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi")
    check_argmax(g["idx"], o["ehvi"])


def test_composite_near_data():
    _announce("composite near data")
    wl = bi.make_config(2, seed=2, M=8)
    comp = bi.composite_hyperparameters(wl)
    cand = bi.near_data_candidates(wl, 600, scale=0.01)
    g = gpu_run(wl, cand=cand, comp=comp)
    o = oracle_score(oracle_fit(wl, comp), wl, cand=cand)
    assert_close(g["mu"], o["mu"], TOL_MU, "mu near data")
    # variance through sigma^2 with the absolute bound of the plain kernel's
    # near-data test, scaled by the largest prior variance
    # s_route + s_dep w^2 + s_int of these points
    c = cand[:, 0, :].astype(np.float64)
    w = np.exp(c[:, comp.d_route:] @ comp.pref.astype(np.float64).T)       # [N, m]
    prior_max = float(np.max(comp.s_route + comp.s_int + comp.s_dep * w * w))
    assert_close(g["sigma"] ** 2, o["sigma"] ** 2, near_var_tol(prior_max), "variance near data")
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi near data")


def test_composite_config3_full_size_sampled():
    _announce("composite config3 full sampled")
    wl = bi.make_config(3, seed=0)
    comp = bi.composite_hyperparameters(wl)
    g = gpu_run(wl, comp=comp)
    r = np.random.default_rng(21)
    idx = np.unique(np.concatenate([[0, 1, wl.M - 1, wl.M // 2], r.integers(0, wl.M, 300)]))
    model = oracle_fit(wl, comp)
    o = oracle_score(model, wl, cand=wl.cand[idx])
    assert_close(g["mu"][idx], o["mu"], TOL_MU, "mu (sampled)")
    assert_close(g["sigma"][idx], o["sigma"], TOL_SIGMA, "sigma (sampled)")
    assert_close(g["ehvi"][idx], o["ehvi"], TOL_EHVI, "ehvi (sampled)")
    e = g["ehvi"].astype(np.float64)
    top = e.max()
    pool = np.nonzero(e >= top - 2 * (TOL_EHVI[0] * abs(top) + TOL_EHVI[1]) - 1e-3 * abs(top))[0]
    assert pool.size < 4096, pool.size
    op = oracle_score(model, wl, cand=wl.cand[pool])
    assert_close(e[pool], op["ehvi"], TOL_EHVI, "ehvi (top pool)")
    check_argmax(g["idx"], op["ehvi"], idx_pool=pool)


def test_composite_config3_full_size_dense():
    """The composite model on all 1,048,576 headline candidates, element by
    element, the oracle over the host's cores. Its preference weights make
    the mean cancel hard at some points (mu = sum_i k_i alpha_i with
    sum_i |k_i alpha_i| up to thousands of times |mu|), where fp32 kernel
    values bound the error absolutely: a mean outside the plain bar must lie
    within the fp32 error model |mu_g - mu_o| <= 1e-4 |mu_o| + 1e-5 +
    2^-18 sum_i |k_i alpha_i| (the learned-hyperparameter bound); how many
    need it, and the worst plain-bar ratio, are logged."""
    import oracle_pool
    _announce("composite config3 full dense")
    wl = bi.make_config(3, seed=0)
    comp = bi.composite_hyperparameters(wl)
    g = gpu_run(wl, comp=comp)
    model = oracle_fit(wl, comp)
    o = oracle_pool.score(model, wl.cand, wl.ref, wl.Z)
    err = np.abs(g["mu"].astype(np.float64) - o["mu"])
    plain = TOL_MU[0] * np.abs(o["mu"]) + TOL_MU[1]
    log_ratio("composite mu, plain bar (informational)", float(np.max(err / plain)))
    out = np.argwhere(err > plain)      # (candidate, member, objective)
    print(f"[composite] {len(out)} of {err.size} means outside the plain bar", flush=True)
    assert len(out) <= 0.001 * err.size, len(out)
    for k in range(wl.m):
        rows = out[out[:, 2] == k, 0]
        if rows.size:
            P = wl.cand[rows, 0, :].astype(np.float64)
            sabs = np.abs(model.cov(k, P, model.X)) @ np.abs(model.alpha[k])
            bound = plain[rows, 0, k] + 2.0 ** -18 * sabs
            assert_close(g["mu"][rows, 0, k], o["mu"][rows, 0, k], (0.0, bound),
                         f"composite mu k={k}, fp32 error model")
    assert_close(g["sigma"], o["sigma"], TOL_SIGMA, "sigma")
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "ehvi")
    check_argmax(g["idx"], o["ehvi"])


def test_composite_bad_arguments():
    import paper_2602_10729_amd as bo
    _announce("composite argument checks")
    wl = bi.make_config(4, seed=0, M=4)
    comp = bi.composite_hyperparameters(wl)
    X, Y = to_dev(wl.X), to_dev(wl.Y)
    model = bo.fit_composite(X, Y, comp.d_route, wl.lengthscale, comp.s_route, comp.s_dep,
                             comp.s_int, comp.pref, wl.noise)
    for dr in (0, wl.d):
        with pytest.raises(bo.BoError) as ei:
            bo.fit_composite(X, Y, dr, wl.lengthscale, comp.s_route, comp.s_dep, comp.s_int,
                             np.zeros((wl.m, max(wl.d - dr, 0)), np.float32), wl.noise)
        assert ei.value.name == "BO_ERR_INVALID_ARGUMENT"
    # d = 32 with one routing coordinate: padded groups need 4 + 32 slots
    r = np.random.default_rng(0)
    X32 = to_dev(r.random((8, 32)).astype(np.float32))
    Y32 = to_dev(r.standard_normal((8, 2)).astype(np.float32))
    with pytest.raises(bo.BoError) as ei:
        bo.fit_composite(X32, Y32, 1, np.ones((2, 32), np.float32), np.ones(2, np.float32),
                         np.ones(2, np.float32), np.zeros(2, np.float32),
                         np.zeros((2, 31), np.float32), np.full(2, 1e-4, np.float32))
    assert ei.value.name == "BO_ERR_CAPACITY"
