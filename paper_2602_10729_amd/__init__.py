"""Python binding of libbo, the MI355X batch acquisition scorer.

Argument marshalling only: every step of fitting, scoring and the argmax runs
in the HIP kernels of ``libbo.so``; torch tensors supply device memory and the
current stream. There is no CPU fallback: if the library is missing or a
tensor is not on the GPU, the call raises.

Functions mirror the C ABI in ``include/bo.h``:
``fit`` (``bo_fit``), ``fit_composite`` (``bo_fit_composite``), ``mll``
(``bo_mll``), ``score`` (``bo_score``, or ``bo_score_constrained`` when feasibility
thresholds are given), ``nehvi_prepare`` / ``score_nehvi`` / ``Model.nehvi_front``
(``bo_nehvi_prepare``, ``bo_score_nehvi``, ``bo_nehvi_front``), ``argmax``,
``cholesky_test`` (device) and
``pareto_front``, ``box_decomposition`` (host geometry, no GPU needed).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

__all__ = ["BoError", "Model", "lib", "lib_path", "fit", "fit_composite", "mll", "score", "score_noalloc", "nehvi_prepare", "score_nehvi", "argmax",
           "cholesky_test", "draw_fronts3_test", "profile_enable", "profile_read", "measure_peak", "pareto_front", "box_decomposition", "STATUS",
           "MAX_N", "MAX_D", "MAX_S", "MAX_BOXES"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libbo.so")
_lib = None

STATUS = {
    0: "BO_OK", 1: "BO_ERR_INVALID_ARGUMENT", 2: "BO_ERR_NOT_POSITIVE_DEFINITE",
    3: "BO_ERR_CAPACITY", 4: "BO_ERR_DEVICE", 5: "BO_ERR_OUT_OF_MEMORY",
    6: "BO_ERR_NONFINITE_INPUT", 7: "BO_ERR_ILL_CONDITIONED",
}
MAX_N, MAX_D, MAX_S, MAX_BOXES = 2048, 32, 4096, 4096


class BoError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        self.name = STATUS.get(status, str(status))
        super().__init__(f"{where}: {self.name}: {detail}")


def lib_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load libbo.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2602_10729_amd.build`")
    L = ctypes.CDLL(_LIB_PATH)
    vp, i64, i32, fp = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    L.bo_fit.argtypes = [vp, vp, i64, i32, i32, fp, fp, fp, vp, ctypes.POINTER(vp)]
    L.bo_fit.restype = ctypes.c_int
    L.bo_fit_composite.argtypes = [vp, vp, i64, i32, i32, i32, fp, fp, fp, fp, fp, fp, vp,
                                   ctypes.POINTER(vp)]
    L.bo_fit_f64.argtypes = L.bo_fit.argtypes
    L.bo_fit_f64.restype = ctypes.c_int
    L.bo_fit_composite_f64.argtypes = L.bo_fit_composite.argtypes
    L.bo_fit_composite_f64.restype = ctypes.c_int
    L.bo_fit_composite.restype = ctypes.c_int
    L.bo_mll.argtypes = [vp, vp, i64, i32, i32, fp, fp, fp, vp, vp, vp]
    L.bo_mll.restype = ctypes.c_int
    L.bo_score.argtypes = [vp, vp, i64, i32, fp, vp, i32, vp, vp, vp, vp]
    L.bo_score.restype = ctypes.c_int
    L.bo_score_constrained.argtypes = [vp, vp, i64, i32, fp, fp, vp, i32, vp, vp, vp, vp]
    L.bo_score_constrained.restype = ctypes.c_int
    L.bo_score_noalloc.argtypes = [vp, vp, i64, i32, fp, vp, i32, vp, vp]
    L.bo_score_noalloc.restype = ctypes.c_int
    L.bo_nehvi_prepare.argtypes = [vp, vp, i32, fp, fp, vp]
    L.bo_nehvi_prepare.restype = ctypes.c_int
    L.bo_score_nehvi.argtypes = [vp, vp, i64, i32, vp, i32, vp, vp]
    L.bo_score_nehvi.restype = ctypes.c_int
    L.bo_nehvi_front.argtypes = [vp, i32, vp, i32, ctypes.POINTER(i32)]
    L.bo_nehvi_front.restype = ctypes.c_int
    L.bo_argmax.argtypes = [vp, i64, vp, vp, vp]
    L.bo_argmax.restype = ctypes.c_int
    L.bo_model_front_size.argtypes = [vp]
    L.bo_model_front_size.restype = i32
    L.bo_model_front_indices.argtypes = [vp, vp, i32]
    L.bo_model_front_indices.restype = ctypes.c_int
    L.bo_cholesky_test.argtypes = [vp, i64, vp, vp]
    L.bo_cholesky_test.restype = ctypes.c_int
    L.bo_draw_fronts3_test.argtypes = [vp, i64, i32, vp, vp, vp, vp, vp, vp]
    L.bo_draw_fronts3_test.restype = ctypes.c_int
    L.bo_pareto_front.argtypes = [vp, i64, i32, vp, vp, i32, ctypes.POINTER(i32)]
    L.bo_pareto_front.restype = ctypes.c_int
    L.bo_box_decomposition.argtypes = [vp, i32, i32, vp, vp, vp, i32, ctypes.POINTER(i32)]
    L.bo_box_decomposition.restype = ctypes.c_int
    L.bo_profile_enable.argtypes = [i32]
    L.bo_profile_enable.restype = ctypes.c_int
    L.bo_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(i64), ctypes.POINTER(i64)]
    L.bo_profile_read.restype = ctypes.c_int
    L.bo_measure_peak.argtypes = [i32, i64, ctypes.POINTER(ctypes.c_double), vp]
    L.bo_measure_peak.restype = ctypes.c_int
    L.bo_free.argtypes = [vp]
    L.bo_free.restype = None
    L.bo_status_string.argtypes = [ctypes.c_int]
    L.bo_status_string.restype = ctypes.c_char_p
    L.bo_last_error_message.argtypes = []
    L.bo_last_error_message.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int, where: str):
    if status != 0:
        detail = lib().bo_last_error_message().decode(errors="replace")
        raise BoError(status, where, detail)


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(int(stream.cuda_stream))


def _dev(t, name, dtype=None):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor on the GPU")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on a GPU (got {t.device})")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _host_f32(a, shape, name):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    if a.size != int(np.prod(shape)):
        raise ValueError(f"{name} must have {int(np.prod(shape))} elements")
    return a


class Model:
    """A fitted model (opaque handle owned by the library)."""

    def __init__(self, handle: int, n: int, d: int, m: int):
        self._h = ctypes.c_void_p(handle)
        self.n, self.d, self.m = n, d, m

    @property
    def handle(self):
        return self._h

    def front_indices(self) -> np.ndarray:
        L = lib()
        P = L.bo_model_front_size(self._h)
        out = np.zeros(max(P, 0), dtype=np.int32)
        _check(L.bo_model_front_indices(self._h, out.ctypes.data_as(ctypes.c_void_p), P),
               "bo_model_front_indices")
        return out

    def nehvi_front(self, sample: int) -> np.ndarray:
        """Front of one prepared in-sample draw (bo_nehvi_front): indices into
        the observations, sorted by objective 0 ascending."""
        L = lib()
        cnt = ctypes.c_int32(0)
        _check(L.bo_nehvi_front(self._h, int(sample), None, 0, ctypes.byref(cnt)), "bo_nehvi_front")
        out = np.zeros(cnt.value, dtype=np.int32)
        _check(L.bo_nehvi_front(self._h, int(sample), out.ctypes.data_as(ctypes.c_void_p),
                                cnt.value, ctypes.byref(cnt)), "bo_nehvi_front")
        return out

    def close(self):
        if self._h is not None and self._h.value:
            lib().bo_free(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def fit(X, Y, lengthscale, outputscale, noise, stream=None, f64=False) -> Model:
    """bo_fit (bo_fit_f64 when f64: scoring in double precision): X [n, d],
    Y [n, m] fp32 GPU tensors; hyperparameters on host."""
    import torch
    n, d = X.shape
    m = Y.shape[1]
    ls = _host_f32(lengthscale, (m, d), "lengthscale")
    os_ = _host_f32(outputscale, (m,), "outputscale")
    nz = _host_f32(noise, (m,), "noise")
    h = ctypes.c_void_p()
    fn = lib().bo_fit_f64 if f64 else lib().bo_fit
    st = fn(_dev(X, "X", torch.float32), _dev(Y, "Y", torch.float32), n, d, m,
            ls.ctypes.data_as(ctypes.c_void_p), os_.ctypes.data_as(ctypes.c_void_p),
            nz.ctypes.data_as(ctypes.c_void_p), _stream(stream), ctypes.byref(h))
    _check(st, "bo_fit_f64" if f64 else "bo_fit")
    return Model(h.value, n, d, m)


def fit_composite(X, Y, d_route, lengthscale, scale_route, scale_dep, scale_int, pref, noise,
                  stream=None, f64=False) -> Model:
    """bo_fit_composite (bo_fit_composite_f64 when f64): the composite kernel
    (routing Matern-5/2 + preference-weighted deployment Matern-3/2 +
    interaction). X [n, d], Y [n, m] fp32 GPU tensors; hyperparameters on host
    (pref [m, d - d_route])."""
    import torch
    n, d = X.shape
    m = Y.shape[1]
    ls = _host_f32(lengthscale, (m, d), "lengthscale")
    sr = _host_f32(scale_route, (m,), "scale_route")
    sd = _host_f32(scale_dep, (m,), "scale_dep")
    si = _host_f32(scale_int, (m,), "scale_int")
    pf = _host_f32(pref, (m, max(d - int(d_route), 0)), "pref")
    nz = _host_f32(noise, (m,), "noise")
    h = ctypes.c_void_p()
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    fn = lib().bo_fit_composite_f64 if f64 else lib().bo_fit_composite
    st = fn(_dev(X, "X", torch.float32), _dev(Y, "Y", torch.float32), n, d,
            m, int(d_route), p(ls), p(sr), p(sd), p(si), p(pf), p(nz),
            _stream(stream), ctypes.byref(h))
    _check(st, "bo_fit_composite_f64" if f64 else "bo_fit_composite")
    return Model(h.value, n, d, m)


def mll(X, Y, lengthscale, outputscale, noise, stream=None):
    """bo_mll: (value [m], gradient [m, d + 2]) of the exact log marginal
    likelihood with respect to (log lengthscales, log outputscale, log noise)."""
    import torch
    n, d = X.shape
    m = Y.shape[1]
    ls = _host_f32(lengthscale, (m, d), "lengthscale")
    os_ = _host_f32(outputscale, (m,), "outputscale")
    nz = _host_f32(noise, (m,), "noise")
    val = np.zeros(m, dtype=np.float64)
    grad = np.zeros((m, d + 2), dtype=np.float64)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    st = lib().bo_mll(_dev(X, "X", torch.float32), _dev(Y, "Y", torch.float32), n, d, m, p(ls),
                      p(os_), p(nz), _stream(stream), p(val), p(grad))
    _check(st, "bo_mll")
    return val, grad


def score(model: Model, cand, ref, Z, ehvi=None, mu=None, sigma=None, stream=None,
          lower=None):
    """bo_score: cand [M, q, d], Z [S, q, m] fp32 GPU tensors; ref host [m].

    Returns the ehvi tensor [M] (allocated if not given). mu/sigma
    [M, q, m] are written only when passed. ``lower`` (host [m], optional)
    selects bo_score_constrained with these feasibility thresholds.
    """
    import torch
    M, q, d = cand.shape
    S = Z.shape[0]
    r = _host_f32(ref, (model.m,), "ref")
    if ehvi is None:
        ehvi = torch.empty(M, dtype=torch.float32, device=cand.device)
    mu_p = _dev(mu, "mu", torch.float32) if mu is not None else ctypes.c_void_p(0)
    sg_p = _dev(sigma, "sigma", torch.float32) if sigma is not None else ctypes.c_void_p(0)
    args = (_dev(cand, "cand", torch.float32), M, q, r.ctypes.data_as(ctypes.c_void_p))
    tail = (_dev(Z, "Z", torch.float32), S, _dev(ehvi, "ehvi", torch.float32), mu_p, sg_p,
            _stream(stream))
    if lower is None:
        st = lib().bo_score(model.handle, *args, *tail)
        _check(st, "bo_score")
    else:
        lw = _host_f32(lower, (model.m,), "lower")
        st = lib().bo_score_constrained(model.handle, *args, lw.ctypes.data_as(ctypes.c_void_p),
                                        *tail)
        _check(st, "bo_score_constrained")
    return ehvi


def score_noalloc(model: Model, cand, ref, Z, ehvi, stream=None):
    """bo_score_noalloc: bo_score without mu/sigma outputs that allocates no
    device memory (its workspace is the library's fixed per-device scratch).
    cand [M, q, d], Z [S, q, m], ehvi [M] fp32 GPU tensors (ehvi must be
    given: this call allocates nothing, the binding neither); ref host [m]."""
    import torch
    M, q, d = cand.shape
    S = Z.shape[0]
    r = _host_f32(ref, (model.m,), "ref")
    st = lib().bo_score_noalloc(model.handle, _dev(cand, "cand", torch.float32), M, q,
                                r.ctypes.data_as(ctypes.c_void_p), _dev(Z, "Z", torch.float32), S,
                                _dev(ehvi, "ehvi", torch.float32), _stream(stream))
    _check(st, "bo_score_noalloc")
    return ehvi


def nehvi_prepare(model: Model, ZX, ref, lower=None, stream=None):
    """bo_nehvi_prepare: ZX [S, n, m] fp32 GPU tensor (in-sample base
    samples); ref host [m]; lower host [m] or None. Synchronous."""
    import torch
    S = ZX.shape[0]
    r = _host_f32(ref, (model.m,), "ref")
    lw = None if lower is None else _host_f32(lower, (model.m,), "lower")
    st = lib().bo_nehvi_prepare(model.handle, _dev(ZX, "ZX", torch.float32), S,
                                r.ctypes.data_as(ctypes.c_void_p),
                                lw.ctypes.data_as(ctypes.c_void_p) if lw is not None else None,
                                _stream(stream))
    _check(st, "bo_nehvi_prepare")


def score_nehvi(model: Model, cand, Z, ehvi=None, stream=None):
    """bo_score_nehvi: cand [M, d] or [M, q, d] and Z [S, m] or [S, q, m] fp32
    GPU tensors. Returns the ehvi tensor [M] (allocated if not given)."""
    import torch
    M = cand.shape[0]
    q = cand.shape[1] if cand.dim() == 3 else 1
    S = Z.shape[0]
    if ehvi is None:
        ehvi = torch.empty(M, dtype=torch.float32, device=cand.device)
    st = lib().bo_score_nehvi(model.handle, _dev(cand, "cand", torch.float32), M, q,
                              _dev(Z, "Z", torch.float32), S, _dev(ehvi, "ehvi", torch.float32),
                              _stream(stream))
    _check(st, "bo_score_nehvi")
    return ehvi


def argmax(values, index=None, value=None, stream=None):
    """bo_argmax into device scalars (int64 index, float32 value)."""
    import torch
    dev = values.device
    if index is None:
        index = torch.empty(1, dtype=torch.int64, device=dev)
    if value is None:
        value = torch.empty(1, dtype=torch.float32, device=dev)
    st = lib().bo_argmax(_dev(values, "values", torch.float32), values.numel(),
                         _dev(index, "index", torch.int64), _dev(value, "value", torch.float32),
                         _stream(stream))
    _check(st, "bo_argmax")
    return index, value


def profile_enable(on: bool = True):
    """Start (or stop) per-phase event timing of bo_score calls."""
    _check(lib().bo_profile_enable(1 if on else 0), "bo_profile_enable")


def profile_read():
    """(posterior_ms, ehvi_ms, calls, posterior_launches) since the last read."""
    a, b = ctypes.c_double(), ctypes.c_double()
    c, n = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().bo_profile_read(ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                                 ctypes.byref(n)), "bo_profile_read")
    return a.value, b.value, c.value, n.value


PEAK_VALU_FMA, PEAK_VALU_CLAMP, PEAK_MFMA_F32, PEAK_HBM_COPY, PEAK_MFMA_F16 = 0, 1, 2, 3, 4


def measure_peak(what: int, iters: int = 4096, stream=None) -> float:
    """Achieved rate of a synthetic probe (see bo_measure_peak in bo.h)."""
    r = ctypes.c_double()
    _check(lib().bo_measure_peak(what, iters, ctypes.byref(r), _stream(stream)), "bo_measure_peak")
    return r.value


def cholesky_test(A, L=None, stream=None):
    """bo_cholesky_test: lower factor of a symmetric fp32 GPU matrix."""
    import torch
    n = A.shape[0]
    if L is None:
        L = torch.empty_like(A)
    st = lib().bo_cholesky_test(_dev(A, "A", torch.float32), n, _dev(L, "L", torch.float32),
                                _stream(stream))
    _check(st, "bo_cholesky_test")
    return L


def draw_fronts3_test(F, ref, lower=None, stream=None):
    """bo_draw_fronts3_test: per-draw fronts and boxes of three-objective
    values F (fp64 GPU tensor [S][n][3]). Returns (fronts, boxes): per draw the
    front's indices (objective 0 ascending) and its boxes [nb][6]
    (lo0, lo1, lo2, w0, w1, w2)."""
    import torch
    S, n, m = F.shape
    if m != 3:
        raise ValueError("F must be [S][n][3]")
    front = torch.empty((S, n), dtype=torch.int32, device=F.device)
    boxes = torch.empty((S, 3 * n + 1, 6), dtype=torch.float32, device=F.device)
    counts = torch.empty(2 * S, dtype=torch.int32, device=F.device)
    r = np.ascontiguousarray(np.asarray(ref, dtype=np.float32))
    lo = None if lower is None else np.ascontiguousarray(np.asarray(lower, dtype=np.float32))
    st = lib().bo_draw_fronts3_test(
        _dev(F, "F", torch.float64), n, S, r.ctypes.data_as(ctypes.c_void_p),
        None if lo is None else lo.ctypes.data_as(ctypes.c_void_p),
        _dev(front, "front"), _dev(boxes, "boxes"), _dev(counts, "counts"), _stream(stream))
    _check(st, "bo_draw_fronts3_test")
    c = counts.cpu().numpy()
    fr, bx = front.cpu().numpy(), boxes.cpu().numpy()
    return ([fr[s, :c[S + s]].copy() for s in range(S)],
            [bx[s, :c[s]].copy() for s in range(S)])


def pareto_front(Y, ref: Optional[np.ndarray] = None) -> np.ndarray:
    """Host: front indices (sorted by objective 0) of Y [n, m] (fp32)."""
    Y = np.ascontiguousarray(np.asarray(Y, dtype=np.float32))
    n, m = Y.shape
    rp = ctypes.c_void_p(0)
    if ref is not None:
        ref = _host_f32(ref, (m,), "ref")
        rp = ref.ctypes.data_as(ctypes.c_void_p)
    idx = np.zeros(max(n, 1), dtype=np.int32)
    cnt = ctypes.c_int32(0)
    _check(lib().bo_pareto_front(Y.ctypes.data_as(ctypes.c_void_p), n, m, rp,
                                 idx.ctypes.data_as(ctypes.c_void_p), n, ctypes.byref(cnt)),
           "bo_pareto_front")
    return idx[:cnt.value].copy()


def box_decomposition(F, ref):
    """Host: disjoint boxes (lo, hi) [B, m] of the region F does not dominate."""
    F = np.ascontiguousarray(np.asarray(F, dtype=np.float32))
    m = np.asarray(ref).shape[0]
    F = F.reshape(-1, m)
    r = _host_f32(ref, (m,), "ref")
    cnt = ctypes.c_int32(0)
    L = lib()
    cap = 4 * F.shape[0] + 8
    while True:
        lo = np.zeros((cap, m), dtype=np.float32)
        hi = np.zeros((cap, m), dtype=np.float32)
        st = L.bo_box_decomposition(F.ctypes.data_as(ctypes.c_void_p), F.shape[0], m,
                                    r.ctypes.data_as(ctypes.c_void_p),
                                    lo.ctypes.data_as(ctypes.c_void_p),
                                    hi.ctypes.data_as(ctypes.c_void_p), cap, ctypes.byref(cnt))
        if st == 3 and cnt.value > cap:
            cap = cnt.value
            continue
        _check(st, "bo_box_decomposition")
        return lo[:cnt.value].copy(), hi[:cnt.value].copy()
