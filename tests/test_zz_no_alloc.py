"""bo_score_noalloc through the C ABI against bo_score.

The no-allocation entry point runs bo_score's kernels with its workspace and
boxes in the library's fixed per-device scratch; its acquisition must equal
bo_score's (mu = sigma = NULL) on the same inputs, bitwise. Two calls in a row
each time, the second with a smaller input (the scratch keeps the first
call's contents), on a q = 1 and a q = 4 workload, and a call beyond the
scratch's limit is refused before any device work.
"""
import numpy as np
import pytest

import bo_inputs as bi
from gpu_util import TOL_EHVI, assert_close, to_dev

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("cfg,M1,M2", [(2, 5003, 1777), (4, 61, 17)])
def test_noalloc_matches_bo_score_on_two_calls(cfg, M1, M2):
    import torch
    import paper_2602_10729_amd as bo
    _announce("noalloc vs bo_score", cfg, M1, M2)
    wl = bi.make_config(cfg, seed=1, M=M1)
    model = bo.fit(to_dev(wl.X), to_dev(wl.Y), wl.lengthscale, wl.outputscale, wl.noise)
    Z = to_dev(wl.Z)
    calls = [(to_dev(wl.cand), wl.ref),
             (to_dev(wl.cand[M1 - M2:]), (wl.ref - 0.05).astype(np.float32))]
    for i, (cand, ref) in enumerate(calls):
        M = cand.shape[0]
        e_ref = bo.score(model, cand, ref, Z)
        i_ref, v_ref = bo.argmax(e_ref)
        e_na = torch.full((M,), float("nan"), dtype=torch.float32, device="cuda")
        bo.score_noalloc(model, cand, ref, Z, e_na)
        i_na, v_na = bo.argmax(e_na)
        torch.cuda.synchronize()
        a, b = e_ref.cpu().numpy(), e_na.cpu().numpy()
        assert_close(b, a, TOL_EHVI, f"noalloc ehvi cfg{cfg} call {i}")
        assert np.array_equal(a, b), f"call {i}: not bitwise equal"
        assert int(i_na.item()) == int(i_ref.item())


def test_noalloc_refuses_a_call_beyond_its_scratch():
    import torch
    import paper_2602_10729_amd as bo
    _announce("noalloc capacity")
    wl = bi.make_config(0, seed=0, M=4)
    model = bo.fit(to_dev(wl.X), to_dev(wl.Y), wl.lengthscale, wl.outputscale, wl.noise)
    M = 2_091_009            # one point beyond 2 objectives x (mu, sigma) in the scratch
    cand = torch.zeros((M, 1, wl.d), dtype=torch.float32, device="cuda")
    e = torch.zeros(M, dtype=torch.float32, device="cuda")
    with pytest.raises(bo.BoError) as ei:
        bo.score_noalloc(model, cand, wl.ref, to_dev(wl.Z), e)
    assert ei.value.name == "BO_ERR_CAPACITY"
    bo.score_noalloc(model, cand[:M - 1], wl.ref, to_dev(wl.Z), e[:M - 1])
    torch.cuda.synchronize()
    assert np.isfinite(e[:M - 1].cpu().numpy()).all()
