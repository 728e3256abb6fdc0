"""The fit's fp64 scratch is kept per device and grown on demand: models
fitted before and after larger fits, likelihood evaluations and a noisy
preparation (which share that device state) must score bit for bit alike,
and a model must stay valid while later fits reuse the scratch."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


def _score(bo, torch, model, wl):
    cand = torch.from_numpy(wl.cand).cuda()
    Z = torch.from_numpy(wl.Z).cuda()
    M, q, _ = wl.cand.shape
    mu = torch.empty((M, q, wl.m), dtype=torch.float32, device="cuda")
    sd = torch.empty_like(mu)
    e = bo.score(model, cand, wl.ref, Z, mu=mu, sigma=sd)
    torch.cuda.synchronize()
    return mu.cpu().numpy(), sd.cpu().numpy(), e.cpu().numpy()


def _fit(bo, torch, wl, f64=False):
    X = torch.from_numpy(wl.X).cuda()
    Y = torch.from_numpy(wl.Y).cuda()
    return bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, f64=f64)


def test_fit_scratch_reuse_is_bitwise_stable():
    import torch
    import bo_inputs as bi
    import paper_2602_10729_amd as bo
    small = bi.make_config(0, seed=1, M=777)
    large = bi.make_config(4, seed=0, M=61)
    mid = bi.make_config(2, seed=2, M=513)

    _announce("fit reuse: small first")
    m_small = _fit(bo, torch, small)
    ref_small = _score(bo, torch, m_small, small)

    _announce("fit reuse: large (scratch grows), then mid and likelihood")
    m_large = _fit(bo, torch, large)
    ref_large = _score(bo, torch, m_large, large)
    m_mid = _fit(bo, torch, mid)
    Xm = torch.from_numpy(mid.X).cuda()
    Ym = torch.from_numpy(mid.Y).cuda()
    bo.mll(Xm, Ym, mid.lengthscale, mid.outputscale, mid.noise)

    _announce("fit reuse: earlier models unchanged by later fits")
    for got, want in zip(_score(bo, torch, m_small, small), ref_small):
        np.testing.assert_array_equal(got, want)
    for got, want in zip(_score(bo, torch, m_large, large), ref_large):
        np.testing.assert_array_equal(got, want)

    _announce("fit reuse: refit after a noisy preparation and an fp64 fit")
    ZX = torch.from_numpy(bi.insample_base_samples(mid, S=64)).cuda()
    bo.nehvi_prepare(m_mid, ZX, mid.ref)
    _fit(bo, torch, large, f64=True)
    torch.cuda.synchronize()
    m_small2 = _fit(bo, torch, small)
    for got, want in zip(_score(bo, torch, m_small2, small), ref_small):
        np.testing.assert_array_equal(got, want)
    m_large2 = _fit(bo, torch, large)
    for got, want in zip(_score(bo, torch, m_large2, large), ref_large):
        np.testing.assert_array_equal(got, want)
