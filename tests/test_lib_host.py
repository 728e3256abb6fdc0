"""The C-ABI library without a GPU: it loads, exports every declared symbol,
validates arguments before touching a device, and its host geometry agrees
with the oracle's independently written front and boxes."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bo():
    import paper_2602_10729_amd as bo
    if not os.path.exists(bo.lib_path()):
        from paper_2602_10729_amd import build
        build.build()
    bo.lib()
    return bo


def _declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for mt in re.finditer(r"\b(bo_[a-z0-9_]+)\s*\(", text):
            names.add(mt.group(1))
    return sorted(names)


def test_library_exports_every_declared_symbol(bo):
    names = _declared_functions()
    assert {"bo_fit", "bo_score", "bo_argmax", "bo_free"} <= set(names)
    L = bo.lib()
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing


def test_status_strings(bo):
    L = bo.lib()
    for s in range(8):
        assert L.bo_status_string(s) != b"unknown status"
    assert L.bo_status_string(99) == b"unknown status"


def test_fit_validation_before_device_work(bo):
    L = bo.lib()
    h = ctypes.c_void_p()
    ls = np.full(4, 0.3, dtype=np.float32)
    one = np.ones(2, dtype=np.float32)
    nz = np.full(2, 1e-4, dtype=np.float32)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    fake = ctypes.c_void_p(0x1000)
    # out == NULL
    assert L.bo_fit(fake, fake, 4, 2, 2, p(ls), p(one), p(nz), None, None) == 1
    # m outside {2, 3}
    assert L.bo_fit(fake, fake, 4, 2, 4, p(ls), p(one), p(nz), None, ctypes.byref(h)) == 1
    # n < 1, d < 1
    assert L.bo_fit(fake, fake, 0, 2, 2, p(ls), p(one), p(nz), None, ctypes.byref(h)) == 1
    assert L.bo_fit(fake, fake, 4, 0, 2, p(ls), p(one), p(nz), None, ctypes.byref(h)) == 1
    # beyond compiled limits
    assert L.bo_fit(fake, fake, 5000, 2, 2, p(ls), p(one), p(nz), None, ctypes.byref(h)) == 3
    assert L.bo_fit(fake, fake, 4, 64, 2, p(np.ones(128, np.float32)), p(one), p(nz), None,
                    ctypes.byref(h)) == 3
    # bad hyperparameters
    bad = ls.copy(); bad[1] = 0.0
    assert L.bo_fit(fake, fake, 4, 2, 2, p(bad), p(one), p(nz), None, ctypes.byref(h)) == 1
    bad[1] = np.nan
    assert L.bo_fit(fake, fake, 4, 2, 2, p(bad), p(one), p(nz), None, ctypes.byref(h)) == 6
    assert L.bo_fit(fake, fake, 4, 2, 2, p(ls), p(-one), p(nz), None, ctypes.byref(h)) == 1
    assert L.bo_fit(fake, fake, 4, 2, 2, p(ls), p(one), p(-nz), None, ctypes.byref(h)) == 1
    assert h.value is None
    assert b"noise" in L.bo_last_error_message()
    # outside the accepted range: outputscale in [2^-64, 2^64], noise <= 2^64
    for s_bad in (2.0 ** -65, 2.0 ** 65):
        sb = np.full(2, s_bad, dtype=np.float32)
        assert L.bo_fit(fake, fake, 4, 2, 2, p(ls), p(sb), p(nz), None, ctypes.byref(h)) == 1
        assert b"2^64" in L.bo_last_error_message()
    for s_ok in (2.0 ** -64, 2.0 ** 64):
        # in range: validation passes and the fake device pointer is refused next
        sb = np.full(2, s_ok, dtype=np.float32)
        assert L.bo_fit(fake, fake, 4, 2, 2, p(ls), p(sb), p(nz), None, ctypes.byref(h)) != 1 \
            or b"2^64" not in L.bo_last_error_message()
    big = np.full(2, 2.0 ** 65, dtype=np.float32)
    assert L.bo_fit(fake, fake, 4, 2, 2, p(ls), p(one), p(big), None, ctypes.byref(h)) == 1
    assert h.value is None


def test_score_and_argmax_validation(bo):
    L = bo.lib()
    ref = np.zeros(2, dtype=np.float32)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    fake = ctypes.c_void_p(0x1000)
    assert L.bo_score(None, fake, 4, 1, p(ref), fake, 8, fake, None, None, None) == 1
    assert L.bo_argmax(fake, -1, fake, fake, None) == 1
    assert L.bo_argmax(fake, 1 << 31, fake, fake, None) == 1
    assert L.bo_cholesky_test(fake, 0, fake, None) == 1
    assert L.bo_cholesky_test(fake, 4096, fake, None) == 3
    r3 = np.zeros(3, dtype=np.float32)
    assert L.bo_draw_fronts3_test(fake, 0, 4, p(r3), None, fake, fake, fake, None) == 1
    assert L.bo_draw_fronts3_test(fake, 8, 0, p(r3), None, fake, fake, fake, None) == 1
    assert L.bo_draw_fronts3_test(fake, 4096, 4, p(r3), None, fake, fake, fake, None) == 3
    assert L.bo_draw_fronts3_test(fake, 8, 4, None, None, fake, fake, fake, None) == 1
    bad = np.array([0, np.nan, 0], dtype=np.float32)
    assert L.bo_draw_fronts3_test(fake, 8, 4, p(bad), None, fake, fake, fake, None) == 6
    assert L.bo_model_front_size(None) == -1


@pytest.mark.parametrize("m", [2, 3])
def test_host_front_and_boxes_match_oracle(bo, m):
    r = np.random.default_rng(40 + m)
    for trial in range(12):
        n = int(r.integers(1, 400))
        Y = r.standard_normal((n, m)).astype(np.float32)
        if n > 5:
            Y[3] = Y[1]                                   # duplicate
            Y[4, :] = np.round(Y[4, :], 1)                # ties on a grid
        ref = (Y.astype(np.float64).min(0) - 0.1).astype(np.float32)
        f_lib = bo.pareto_front(Y, ref)
        f_or = O.pareto_front(Y.astype(np.float64), ref.astype(np.float64))
        np.testing.assert_array_equal(f_lib, f_or)
        lo, hi = bo.box_decomposition(Y[f_lib], ref)
        lo2, hi2 = O.box_decomposition(Y[f_or].astype(np.float64), ref.astype(np.float64))
        ys = r.normal(0.3, 1.2, size=(300, m))
        np.testing.assert_allclose(O.hvi(ys, lo.astype(np.float64), hi.astype(np.float64)),
                                   O.hvi(ys, lo2, hi2), rtol=1e-9, atol=1e-12)
        # disjointness and coverage of the library's boxes
        pts = r.uniform(ref, Y.max(0) + 0.5, size=(3000, m))
        F = Y[f_lib].astype(np.float64)
        dominated = np.any(np.all(F[None] >= pts[:, None], axis=2), axis=1) if len(F) else np.zeros(3000, bool)
        inside = np.all((pts[:, None, :] >= lo) & (pts[:, None, :] < hi), axis=2).sum(1)
        assert np.all(inside <= 1)
        np.testing.assert_array_equal(inside == 1, ~dominated)


def test_host_boxes_on_integer_grid(bo):
    from pins import hv_grid_count
    r = np.random.default_rng(1)
    for m in (2, 3):
        for _ in range(5):
            P = r.integers(1, 6, size=(7, m)).astype(np.float32)
            ref = np.zeros(m, dtype=np.float32)
            f = bo.pareto_front(P, ref)
            lo, hi = bo.box_decomposition(P[f], ref)
            U = np.full(m, 6.0)
            vol = np.prod(np.clip(np.minimum(hi, U) - lo, 0, None), axis=1).sum()
            assert vol + hv_grid_count(P.astype(int), ref.astype(int)) == pytest.approx(6.0 ** m)


def test_box_decomposition_rejects_rows_below_reference(bo):
    with pytest.raises(bo.BoError) as ei:
        bo.box_decomposition(np.array([[1.0, -1.0]], dtype=np.float32), np.zeros(2, np.float32))
    assert ei.value.status == 1


def test_host_front_with_ties_and_duplicates_matches_oracle(bo):
    """Coarse values (many exact ties and duplicate rows) in two and three
    objectives, with and without the reference filter."""
    r = np.random.default_rng(0)
    for trial in range(300):
        m = 2 if trial % 2 else 3
        Y = (np.round(r.standard_normal((int(r.integers(1, 60)), m)) * 2) / 2).astype(np.float32)
        ref = None if trial % 3 == 0 else (Y.min(0) - 0.1).astype(np.float32)
        got = bo.pareto_front(Y, ref)
        if ref is None:
            o = O.nondominated(Y.astype(np.float64))
            o = o[np.lexsort((o, Y[o, 0]))]
        else:
            o = O.pareto_front(Y.astype(np.float64), ref.astype(np.float64))
        assert list(got) == list(o), (trial, got, o)
