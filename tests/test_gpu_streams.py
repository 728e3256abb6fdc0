"""Calls on one model from different streams are ordered by the library: a
scoring call on another stream waits for the model's previous call before it
rewrites the model's boxes and workspace, so back-to-back calls with
different reference points on two streams, enqueued without any host
synchronisation between them, give bit for bit the results of the same
calls made one after another on one stream. The fit on a caller's stream is
covered the same way (its side-stream work joins before it returns)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _announce(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("cfg,M", [(1, 65536), (4, 4096)])
def test_calls_on_two_streams_match_one_stream(cfg, M):
    import torch
    import bo_inputs as bi
    import paper_2602_10729_amd as bo
    _announce("two streams", cfg, M)
    wl = bi.make_config(cfg, seed=0, M=M)
    X = torch.from_numpy(wl.X).cuda()
    Y = torch.from_numpy(wl.Y).cuda()
    cand = torch.from_numpy(wl.cand).cuda()
    Z = torch.from_numpy(wl.Z).cuda()
    ref_a = np.asarray(wl.ref, np.float32)
    # a second reference point below the first: a different box set
    ref_b = ref_a - np.float32(0.25)

    # one stream, one call after another
    m1 = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise)
    ea1 = bo.score(m1, cand, ref_a, Z).cpu().numpy()
    eb1 = bo.score(m1, cand, ref_b, Z).cpu().numpy()
    torch.cuda.synchronize()

    # two streams of default priority, no host synchronisation in between
    s1 = torch.cuda.Stream()
    s2 = torch.cuda.Stream()
    ea2 = torch.empty(cand.shape[0], device="cuda")
    eb2 = torch.empty(cand.shape[0], device="cuda")
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    m2 = bo.fit(X, Y, wl.lengthscale, wl.outputscale, wl.noise, stream=s1)
    bo.score(m2, cand, ref_a, Z, ehvi=ea2, stream=s1)
    bo.score(m2, cand, ref_b, Z, ehvi=eb2, stream=s2)
    bo.score(m2, cand, ref_a, Z, ehvi=ea2, stream=s1)
    torch.cuda.synchronize()
    assert np.array_equal(ea2.cpu().numpy(), ea1)
    assert np.array_equal(eb2.cpu().numpy(), eb1)
    assert not np.array_equal(ea1, eb1)
