"""GPU parity of the noisy acquisition (bo_nehvi_prepare + bo_score_nehvi)
against the fp64 oracle.

Per-sample fronts are index work: their index sets must equal the oracle's
exactly. The acquisition meets the EHVI bar; with feasibility thresholds the
decision y >= t is taken by each side on its own candidate sample, so the
samples within the posterior tolerances of a threshold are bounded on both
sides.
"""
import numpy as np
import pytest

import bo_inputs as bi
import oracle as O
from gpu_util import TOL_EHVI, to_dev, oracle_fit, assert_close, assert_within_bounds, check_argmax

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


def _gpu(wl, cand, ZX, Zs, ref=None, lower=None, model=None, comp=None):
    import torch
    import paper_2602_10729_amd as bo
    if model is None and comp is None:
        model = bo.fit(to_dev(wl.X), to_dev(wl.Y), wl.lengthscale, wl.outputscale, wl.noise)
    elif model is None:
        model = bo.fit_composite(to_dev(wl.X), to_dev(wl.Y), comp.d_route, wl.lengthscale,
                                 comp.s_route, comp.s_dep, comp.s_int, comp.pref, wl.noise)
    bo.nehvi_prepare(model, to_dev(ZX), wl.ref if ref is None else ref, lower=lower)
    e = bo.score_nehvi(model, to_dev(np.ascontiguousarray(cand)), to_dev(np.ascontiguousarray(Zs)))
    idx, val = bo.argmax(e)
    torch.cuda.synchronize()
    return dict(ehvi=e.cpu().numpy(), idx=int(idx.item()), val=float(val.item()), model=model)


def _oracle(wl, cand, ZX, Zs, ref=None, lower=None, model=None):
    om = oracle_fit(wl) if model is None else model
    return O.nehvi(om, cand, wl.ref if ref is None else ref, ZX, Zs,
                   lower=None if lower is None else np.asarray(lower, dtype=np.float64))


def _oracle_fronts(o, ref, lower, samples):
    out = []
    for s in samples:
        F = o["F"][s]
        keep = np.arange(F.shape[0])
        if lower is not None:
            keep = keep[np.all(F >= np.asarray(lower, dtype=np.float64), axis=1)]
        out.append(keep[O.pareto_front(F[keep], np.asarray(ref, dtype=np.float64))])
    return out


def _check_fronts(g, o, ref, lower, samples):
    want = _oracle_fronts(o, ref, lower, samples)
    for s, w in zip(samples, want):
        got = g["model"].nehvi_front(s)
        assert np.array_equal(got, w), (s, got, w)


def _workload(cfg, seed, M, n=None, S=None):
    wl = bi.make_config(cfg, seed=seed, M=M)
    if n is not None:
        wl.X, wl.Y, wl.n = wl.X[:n].copy(), wl.Y[:n].copy(), n
    ZX = bi.insample_base_samples(wl, S)
    Zs = wl.Z[:, 0, :] if S is None else np.random.default_rng(seed + 99).standard_normal(
        (S, wl.m)).astype(np.float32)
    return wl, ZX, Zs


@pytest.mark.parametrize("cfg,M,seed,n,S", [(0, 4096, 0, None, None), (0, 1000, 1, None, None),
                                            (1, 3001, 1, None, None), (1, 1000, 0, 77, 200),
                                            (2, 2003, 0, None, None)])
def test_noisy_parity(cfg, M, seed, n, S):
    _announce("nehvi", cfg, M, seed, n, S)
    wl, ZX, Zs = _workload(cfg, seed, M, n, S)
    cand = wl.cand[:, 0, :]
    g = _gpu(wl, cand, ZX, Zs)
    o = _oracle(wl, cand, ZX, Zs)
    # the noisy form differs from the plain one (the test is not vacuous)
    plain = O.score(oracle_fit(wl), wl.cand.astype(np.float64), wl.ref,
                    Zs[:, None, :].astype(np.float64))["ehvi"]
    assert np.max(np.abs(o["ehvi"] - plain)) > 1e-4
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "nehvi")
    check_argmax(g["idx"], o["ehvi"])
    assert g["val"] == g["ehvi"][g["idx"]]
    _check_fronts(g, o, wl.ref, None, range(0, ZX.shape[0], max(1, ZX.shape[0] // 16)))


def test_noisy_near_data_candidates():
    _announce("nehvi near data")
    wl, ZX, Zs = _workload(2, 1, 8)
    cand = bi.near_data_candidates(wl, 700, scale=0.02)[:, 0, :]
    g = _gpu(wl, cand, ZX, Zs)
    o = _oracle(wl, cand, ZX, Zs)
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "nehvi near data")


def _noisy_constrained_bounds(om, cand, ZX, Zs, o, lower, safety=4.0):
    """Range of the constrained noisy acquisition over the candidate samples
    whose feasibility the GPU may decide differently (see the module doc):
    a sample within `safety` times the mean/std tolerance of a threshold
    counts in the upper bound only."""
    F, Ls = O.insample_samples(om, ZX)
    ys = O.candidate_samples(om, cand, ZX, Zs, Ls)              # [M, S, m]
    lower = np.asarray(lower, dtype=np.float64)
    band = safety * (1e-4 * np.abs(ys) + 1e-4 * np.abs(Zs)[None] + 1e-5)
    h = np.empty(ys.shape[:2])
    for s in range(ys.shape[1]):
        lo, hi = o["boxes"][s]
        h[:, s] = O.hvi(ys[:, s, :], lo, hi)
    d = ys - lower
    sure = np.all(d > band, axis=-1)
    maybe = np.all(d >= -band, axis=-1)
    return np.mean(h * sure, axis=1), np.mean(h * maybe, axis=1)


@pytest.mark.parametrize("cfg,M,seed", [(0, 2048, 0), (2, 1000, 2)])
def test_noisy_constrained_parity(cfg, M, seed):
    _announce("nehvi constrained", cfg, M, seed)
    wl, ZX, Zs = _workload(cfg, seed, M)
    cand = wl.cand[:, 0, :]
    lower = bi.feasibility_thresholds(wl, 0.3)
    g = _gpu(wl, cand, ZX, Zs, lower=lower)
    om = oracle_fit(wl)
    o = _oracle(wl, cand, ZX, Zs, lower=lower, model=om)
    u = _oracle(wl, cand[:300], ZX, Zs, model=om)
    # the constraint binds: it removes infeasible in-sample points from the
    # fronts (raising the HVI) and infeasible candidate samples (lowering it)
    assert np.mean(np.abs(o["ehvi"][:300] - u["ehvi"]) > 1e-6 * u["ehvi"]) > 0.2
    lo, hi = _noisy_constrained_bounds(om, cand, ZX, Zs.astype(np.float64), o, lower)
    assert_within_bounds(g["ehvi"], lo, hi, TOL_EHVI, "constrained nehvi")
    exact = lo == hi
    assert exact.mean() > 0.5, exact.mean()
    assert_close(g["ehvi"][exact], o["ehvi"][exact], TOL_EHVI, "constrained nehvi (unambiguous)")
    _check_fronts(g, o, wl.ref, lower, range(0, ZX.shape[0], max(1, ZX.shape[0] // 16)))


def test_noisy_headline_size_sampled():
    # the full headline workload in the bench's launch configuration (four
    # chunks of candidates); the oracle checks a spread of sampled candidates
    import torch
    _announce("nehvi headline size, sampled")
    wl, ZX, Zs = _workload(3, 0, None)
    g = _gpu(wl, wl.cand[:, 0, :], ZX, Zs)
    assert g["ehvi"].shape == (wl.M,) and np.all(np.isfinite(g["ehvi"]))
    pick = np.unique(np.concatenate([np.linspace(0, wl.M - 1, 384).astype(np.int64),
                                     np.arange(262140, 262150), [wl.M - 1, g["idx"]]]))
    o = _oracle(wl, wl.cand[pick, 0, :], ZX, Zs)
    assert_close(g["ehvi"][pick], o["ehvi"], TOL_EHVI, "nehvi (sampled)")
    assert g["ehvi"][g["idx"]] == g["ehvi"].max()
    torch.cuda.synchronize()


def test_noisy_reprepare_and_edges():
    import torch
    import paper_2602_10729_amd as bo
    _announce("nehvi re-prepare and edge cases")
    wl, ZX, Zs = _workload(0, 3, 500)
    cand = wl.cand[:, 0, :]
    model = bo.fit(to_dev(wl.X), to_dev(wl.Y), wl.lengthscale, wl.outputscale, wl.noise)
    with pytest.raises(bo.BoError, match="INVALID_ARGUMENT"):
        bo.score_nehvi(model, to_dev(cand), to_dev(Zs))               # not prepared
    g1 = _gpu(wl, cand, ZX, Zs, model=model)
    ZX2 = -ZX[:64].copy()
    Zs2 = Zs[:64].copy()
    g2 = _gpu(wl, cand, ZX2, Zs2, model=model)                         # smaller S, new draws
    assert_close(g2["ehvi"], _oracle(wl, cand, ZX2, Zs2)["ehvi"], TOL_EHVI, "re-prepared")
    assert not np.allclose(g1["ehvi"], g2["ehvi"])
    with pytest.raises(bo.BoError, match="INVALID_ARGUMENT"):
        bo.score_nehvi(model, to_dev(cand), to_dev(Zs))               # S differs from prepared
    e = torch.full((1,), 7.0, device="cuda")
    bo.score_nehvi(model, to_dev(cand[:0].copy()), to_dev(Zs2), ehvi=e)   # M = 0: nothing written
    torch.cuda.synchronize()
    assert e.item() == 7.0
    big = np.zeros((513, wl.n, 2), dtype=np.float32)
    with pytest.raises(bo.BoError, match="CAPACITY"):
        bo.nehvi_prepare(model, to_dev(big), wl.ref)
    # batches of three are not supported
    with pytest.raises(bo.BoError, match="INVALID_ARGUMENT"):
        bo.score_nehvi(model, to_dev(np.ascontiguousarray(wl.cand[:6, 0, :].reshape(2, 3, -1))),
                       to_dev(np.zeros((64, 3, 2), np.float32)))
    torch.cuda.synchronize()


def _batched(wl, ZX, M, q, seed):
    """q-batches from the workload's candidate stream and their base samples."""
    d = wl.cand.shape[-1]
    pts = wl.cand.reshape(-1, d)[:M * q]
    Zs = np.random.default_rng(seed + 7).standard_normal((ZX.shape[0], q, wl.m)).astype(np.float32)
    return np.ascontiguousarray(pts.reshape(M, q, d)), Zs


@pytest.mark.parametrize("cfg,M,q,seed", [(0, 1500, 2, 0), (1, 700, 4, 1), (0, 333, 4, 2)])
def test_noisy_batch_parity_two_objectives(cfg, M, q, seed):
    _announce("nehvi batches", cfg, M, q, seed)
    wl = bi.make_config(cfg, seed=seed, M=M * q)
    ZX = bi.insample_base_samples(wl)
    cand, Zs = _batched(wl, ZX, M, q, seed)
    g = _gpu(wl, cand, ZX, Zs)
    o = _oracle(wl, cand, ZX, Zs)
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "nehvi batches")
    check_argmax(g["idx"], o["ehvi"])


@pytest.mark.parametrize("q,M,S,seed", [(1, 400, 128, 0), (4, 48, 512, 0), (2, 96, 200, 1)])
def test_noisy_three_objectives(q, M, S, seed):
    # config 4's observations (n = 2048, d = 24, three objectives): per-draw
    # fronts and 3-D boxes built on the device, boxes read from global memory;
    # every draw's front is checked
    _announce("nehvi three objectives", q, M, S, seed)
    wl = bi.make_config(4, seed=seed, M=M)
    ZX = bi.insample_base_samples(wl, S)
    if q == 4 and S == wl.S:
        cand, Zs = np.ascontiguousarray(wl.cand), wl.Z
    else:
        cand, Zs = _batched(wl, ZX, M, q, seed)
        if q == 1:
            cand, Zs = cand[:, 0, :], Zs[:, 0, :]
    g = _gpu(wl, cand, ZX, Zs)
    o = _oracle(wl, cand, ZX, Zs)
    assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "nehvi three objectives")
    check_argmax(g["idx"], o["ehvi"])
    _check_fronts(g, o, wl.ref, None, range(S))


def test_noisy_three_objectives_constrained():
    _announce("nehvi three objectives constrained")
    wl = bi.make_config(4, seed=2, M=40)
    ZX = bi.insample_base_samples(wl, 256)
    cand, Zs = _batched(wl, ZX, 40, 4, 2)
    lower = bi.feasibility_thresholds(wl, [0.3, None, 0.2])
    g = _gpu(wl, cand, ZX, Zs, lower=lower)
    om = oracle_fit(wl)
    o = _oracle(wl, cand, ZX, Zs, lower=lower, model=om)
    # bounds over the member draws whose feasibility is ambiguous (module doc)
    F, Ls = O.insample_samples(om, ZX)
    ys = O.batch_samples(om, cand, ZX, Zs, Ls)                       # [M, S, q, m]
    low = np.asarray(lower, dtype=np.float64)
    # each side's member draw differs by at most the mean tolerance plus the
    # std tolerance times sum_t |z_t| (factor entries are at most sqrt(s) = 1)
    zsum = np.abs(Zs).sum(axis=1)[None, :, None, :]                  # [1, S, 1, m]
    band = 4.0 * (1e-4 * np.abs(ys) + 1e-4 * zsum + 1e-5)
    d = ys - low
    sure = np.all(d > band, axis=-1).astype(float)
    maybe = np.all(d >= -band, axis=-1).astype(float)
    lo = np.empty(len(cand))
    hi = np.empty(len(cand))
    hs_lo = np.empty((len(cand), ZX.shape[0]))
    hs_hi = np.empty_like(hs_lo)
    for s in range(ZX.shape[0]):
        blo, bhi = o["boxes"][s]
        hs_lo[:, s] = O.qhvi(ys[:, s], blo, bhi, sure[:, s])
        hs_hi[:, s] = O.qhvi(ys[:, s], blo, bhi, maybe[:, s])
    lo, hi = hs_lo.mean(axis=1), hs_hi.mean(axis=1)
    assert_within_bounds(g["ehvi"], lo, hi, TOL_EHVI, "constrained nehvi, three objectives")
    exact = lo == hi
    assert exact.mean() > 0.3, exact.mean()
    assert_close(g["ehvi"][exact], o["ehvi"][exact], TOL_EHVI, "constrained nehvi (unambiguous)")
    _check_fronts(g, o, wl.ref, lower, range(0, 256, 32))


@pytest.mark.parametrize("cfg,M,q,seed,d_route,cons", [(2, 1500, 1, 0, None, False),
                                                       (0, 400, 2, 1, 2, False),
                                                       (4, 40, 4, 0, None, False),
                                                       (2, 800, 1, 2, None, True)])
def test_noisy_composite_kernel(cfg, M, q, seed, d_route, cons):
    """The paper's surrogate (composite kernel) inside its acquisition (the
    noisy form, optionally constrained)."""
    _announce("nehvi composite", cfg, M, q, seed, d_route, cons)
    wl = bi.make_config(cfg, seed=seed, M=M * q if q != wl_q(cfg) else M)
    comp = bi.composite_hyperparameters(wl, d_route)
    S = 256 if cfg == 4 else None
    ZX = bi.insample_base_samples(wl, S)
    if q == 1:
        cand, Zs = np.ascontiguousarray(wl.cand[:M, 0, :]), np.ascontiguousarray(wl.Z[:, 0, :])
        if S is not None:
            Zs = Zs[:S]
    else:
        cand, Zs = _batched(wl, ZX, M, q, seed)
    lower = bi.feasibility_thresholds(wl, 0.3) if cons else None
    g = _gpu(wl, cand, ZX, Zs, lower=lower, comp=comp)
    om = oracle_fit(wl, comp)
    o = _oracle(wl, cand, ZX, Zs, lower=lower, model=om)
    if not cons:
        assert_close(g["ehvi"], o["ehvi"], TOL_EHVI, "nehvi composite")
        check_argmax(g["idx"], o["ehvi"])
    else:
        lo, hi = _noisy_constrained_bounds(om, cand, ZX, Zs.astype(np.float64), o, lower)
        assert_within_bounds(g["ehvi"], lo, hi, TOL_EHVI, "constrained nehvi composite")
        exact = lo == hi
        assert exact.mean() > 0.5, exact.mean()
        assert_close(g["ehvi"][exact], o["ehvi"][exact], TOL_EHVI, "constrained nehvi composite")
    _check_fronts(g, o, wl.ref, lower, range(0, ZX.shape[0], max(1, ZX.shape[0] // 8)))


def wl_q(cfg):
    return bi.CONFIGS[cfg]["q"]
