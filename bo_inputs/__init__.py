"""Seeded synthetic workloads for batch acquisition scoring.

This module only draws and prepares inputs. It holds none of the scoring
arithmetic (no kernel function, no posterior, no hypervolume): both the fp64
oracle and the GPU path consume the arrays it returns and share nothing else.

Workload recipe (five configurations, all objectives maximised):

====  ====  ==  ====  ========  ===  =========================================
cfg   m,q   d   n     M         S    inputs / objectives
====  ====  ==  ====  ========  ===  =========================================
0     2,1   6   32    4096      128  U[0,1]^6; y1=-|x-0.3|^2, y2=-|x-0.7|^2
1     2,1   12  256   65536     256  U[0,1]^12; y1=sum sin(3x_j)/12,
                                     y2=-sum (x_j-.5)^2 + 0.5 x0 x1
2     2,1   16  1024  262144    512  dims 0-3 U[0,1], dims 4-15 k/8 with
                                     k uniform on {0..8};
                                     y1=sum w_j x_j (1-0.3 x_j),
                                     y2=sigmoid(4 sum_{j<4} x_j - 2)
3     2,1   16  1024  1048576   512  as 2 (same X, Y, lengthscales, Z; the
                                     candidates extend config 2's stream)
4     3,4   24  2048  131072x4  512  U[0,1]^24; y1, y2 as 2 over 24 dims,
                                     y3=-sum x_j^2/24
====  ====  ==  ====  ========  ===  =========================================

The encoded decision vector stands in for the paper's theta = (tau, c)
(routing thresholds / load fractions plus per-GPU-type deployment choices,
Section "Online Optimization Phase", structural information S1), and the two
or three objectives stand in for latency and quality outcomes of Eq. (1).
The paper's own workloads (request traces, the simulator database, the router)
are not used.

Every array is drawn in fp64 and rounded to fp32 once; both sides read the
rounded values (the oracle up-casts them). Observation noise N(0, sigma^2) is
added, then each objective is standardised with its mean and unbiased (ddof=1)
standard deviation in fp64, as the outcome transform "Standardize" of the
paper's implementation section does, and rounded to fp32. The reference point
is the per-objective minimum of the standardised fp32 Y minus 0.1.

Feasibility thresholds (for the constrained acquisition): per objective the
given quantile (default 0.3) of the standardised fp32 Y, in fp64, rounded to
fp32 — a latency cap and a quality floor that 70% of the observations meet
on each objective. ``None`` in place of a quantile leaves that objective
unconstrained (-inf).

Composite-kernel hyperparameters (for the paper's additive surrogate): the
routing features are the first d/4 coordinates (4 for configs 2 and 3, the
routing fractions), the rest are deployment features; output scales 0.7
(routing Matern-5/2), 0.3 (preference-weighted deployment Matern-3/2) and
0.05 (interaction); preference slopes 0.08 * U[0,1] per objective and
deployment dimension (stream 6), so the weights exp(p . c) stay within
[1, e^{0.96}]. Lengthscales are the workload's.

In-sample base samples (for the noisy acquisition, which also samples the
latent objectives at the observed points): iid N(0,1) of shape [S, n, m]
from stream 7, rounded to fp32.

Random streams: ``numpy.random.Generator(PCG64(SeedSequence(seed,
spawn_key=(family, stream))))`` with streams 0 X, 1 candidates, 2 noise,
3 lengthscales, 4 weights w, 5 base samples Z, 6 preference slopes, 7 the
in-sample base samples of the noisy acquisition; family is
the config number
except that configs 2 and 3 share family 2. Candidates are drawn row by row,
so a prefix of a larger M equals the smaller-M draw.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = ["CONFIGS", "Workload", "make_config", "near_data_candidates",
           "feasibility_thresholds", "CompositeParams", "composite_hyperparameters",
           "insample_base_samples"]

# (m, q, d, n, M, S, noise_sd, family)
CONFIGS = {
    0: dict(m=2, q=1, d=6, n=32, M=4096, S=128, noise_sd=0.01, family=0),
    1: dict(m=2, q=1, d=12, n=256, M=65536, S=256, noise_sd=0.02, family=1),
    2: dict(m=2, q=1, d=16, n=1024, M=262144, S=512, noise_sd=0.01, family=2),
    3: dict(m=2, q=1, d=16, n=1024, M=1048576, S=512, noise_sd=0.01, family=2),
    4: dict(m=3, q=4, d=24, n=2048, M=131072, S=512, noise_sd=0.01, family=4),
}

OUTPUTSCALE = 1.0
NOISE_VAR = 1e-4
REF_OFFSET = 0.1

(STREAM_X, STREAM_CAND, STREAM_NOISE, STREAM_LS, STREAM_W, STREAM_Z, STREAM_PREF,
 STREAM_ZX) = range(8)


@dataclass
class Workload:
    cfg: int
    seed: int
    m: int
    q: int
    d: int
    n: int
    M: int
    S: int
    X: np.ndarray            # [n, d] fp32
    Y: np.ndarray            # [n, m] fp32, standardised
    cand: np.ndarray         # [M, q, d] fp32
    lengthscale: np.ndarray  # [m, d] fp32
    outputscale: np.ndarray  # [m] fp32
    noise: np.ndarray        # [m] fp32 (noise variance)
    ref: np.ndarray          # [m] fp32
    Z: np.ndarray            # [S, q, m] fp32
    meta: dict = field(default_factory=dict)


def _rng(seed: int, family: int, stream: int) -> np.random.Generator:
    ss = np.random.SeedSequence(seed, spawn_key=(family, stream))
    return np.random.Generator(np.random.PCG64(ss))


def _draw_points(cfg: int, rng: np.random.Generator, rows: int, d: int) -> np.ndarray:
    """Encoded configurations in [0,1]^d, drawn row-major from one stream."""
    u = rng.random((rows, d))
    if cfg in (2, 3):
        # dims 0-3: continuous routing fractions; dims 4..: integers {0..8}/8
        k = np.floor(u[:, 4:] * 9.0)
        u[:, 4:] = np.minimum(k, 8.0) / 8.0
    return u


def _objectives(cfg: int, X: np.ndarray, w: Optional[np.ndarray]) -> np.ndarray:
    if cfg == 0:
        y1 = -np.sum((X - 0.3) ** 2, axis=1)
        y2 = -np.sum((X - 0.7) ** 2, axis=1)
        return np.stack([y1, y2], axis=1)
    if cfg == 1:
        y1 = np.sum(np.sin(3.0 * X), axis=1) / 12.0
        y2 = -np.sum((X - 0.5) ** 2, axis=1) + 0.5 * X[:, 0] * X[:, 1]
        return np.stack([y1, y2], axis=1)
    y1 = np.sum(w[None, :] * X * (1.0 - 0.3 * X), axis=1)
    y2 = 1.0 / (1.0 + np.exp(-(4.0 * np.sum(X[:, :4], axis=1) - 2.0)))
    if cfg in (2, 3):
        return np.stack([y1, y2], axis=1)
    y3 = -np.sum(X ** 2, axis=1) / X.shape[1]
    return np.stack([y1, y2, y3], axis=1)


def make_config(cfg: int, seed: int = 0, M: Optional[int] = None) -> Workload:
    """Build the seeded workload of configuration ``cfg``.

    ``M`` overrides the number of candidates (q-batches for config 4); the
    first ``M`` rows are identical to those of the full-size draw.
    """
    if cfg not in CONFIGS:
        raise ValueError(f"unknown config {cfg}")
    c = CONFIGS[cfg]
    m, q, d, n, S, fam = c["m"], c["q"], c["d"], c["n"], c["S"], c["family"]
    Mv = c["M"] if M is None else int(M)
    if Mv < 0:
        raise ValueError("M must be >= 0")

    X = _draw_points(cfg, _rng(seed, fam, STREAM_X), n, d).astype(np.float32)
    cand = _draw_points(cfg, _rng(seed, fam, STREAM_CAND), Mv * q, d)
    cand = cand.astype(np.float32).reshape(Mv, q, d)

    w = None
    if cfg >= 2:
        w = _rng(seed, fam, STREAM_W).uniform(0.5, 1.5, size=d)
    Yraw = _objectives(cfg, X.astype(np.float64), w)
    Yraw = Yraw + c["noise_sd"] * _rng(seed, fam, STREAM_NOISE).standard_normal((n, m))
    mean = Yraw.mean(axis=0)
    sd = Yraw.std(axis=0, ddof=1)
    Y = ((Yraw - mean) / sd).astype(np.float32)

    if cfg == 0:
        ls = np.full((m, d), 0.3)
    elif cfg == 1:
        ls = _rng(seed, fam, STREAM_LS).uniform(0.1, 0.5, size=(m, d))
    else:
        ls = _rng(seed, fam, STREAM_LS).uniform(0.1, 0.6, size=(m, d))
    ls = ls.astype(np.float32)

    ref = (Y.astype(np.float64).min(axis=0) - REF_OFFSET).astype(np.float32)
    Z = _rng(seed, fam, STREAM_Z).standard_normal((S, q, m)).astype(np.float32)

    return Workload(
        cfg=cfg, seed=seed, m=m, q=q, d=d, n=n, M=Mv, S=S,
        X=X, Y=Y, cand=cand, lengthscale=ls,
        outputscale=np.full(m, OUTPUTSCALE, dtype=np.float32),
        noise=np.full(m, NOISE_VAR, dtype=np.float32),
        ref=ref, Z=Z,
        meta=dict(y_mean=mean, y_sd=sd, w=w),
    )


def near_data_candidates(wl: Workload, count: int, scale: float = 0.01,
                         seed: int = 12345) -> np.ndarray:
    """Candidates placed near observed points: X[i] + N(0, scale^2), clipped.

    These exercise the triangular solve where the cross-covariance is large,
    which random candidates in 16-24 dimensions rarely do.
    """
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    idx = rng.integers(0, wl.n, size=count * wl.q)
    pts = wl.X.astype(np.float64)[idx] + scale * rng.standard_normal((count * wl.q, wl.d))
    pts = np.clip(pts, 0.0, 1.0)
    return pts.astype(np.float32).reshape(count, wl.q, wl.d)


def feasibility_thresholds(wl: Workload, quantiles=0.3) -> np.ndarray:
    """Lower bounds [m] on the standardised objectives for the constrained
    acquisition: the per-objective quantile of the observed Y (fp32).
    ``quantiles`` is one value or one per objective (None: unconstrained)."""
    qs = [quantiles] * wl.m if np.isscalar(quantiles) or quantiles is None else list(quantiles)
    Y = wl.Y.astype(np.float64)
    out = np.empty(wl.m)
    for k, qk in enumerate(qs):
        out[k] = -np.inf if qk is None else np.quantile(Y[:, k], qk)
    return out.astype(np.float32)


@dataclass
class CompositeParams:
    d_route: int
    s_route: np.ndarray      # [m] fp32
    s_dep: np.ndarray        # [m] fp32
    s_int: np.ndarray        # [m] fp32
    pref: np.ndarray         # [m, d - d_route] fp32


def composite_hyperparameters(wl: Workload, d_route: Optional[int] = None) -> CompositeParams:
    """Seeded hyperparameters of the composite kernel for a workload."""
    dr = max(1, wl.d // 4) if d_route is None else int(d_route)
    if not 1 <= dr < wl.d:
        raise ValueError("need 1 <= d_route < d")
    fam = CONFIGS[wl.cfg]["family"]
    pref = 0.08 * _rng(wl.seed, fam, STREAM_PREF).random((wl.m, wl.d - dr))
    f = lambda v: np.full(wl.m, v, dtype=np.float32)
    return CompositeParams(dr, f(0.7), f(0.3), f(0.05), pref.astype(np.float32))


def insample_base_samples(wl: Workload, S: Optional[int] = None) -> np.ndarray:
    """Base samples [S, n, m] (fp32) of the latent objectives at the observed
    points, for the noisy acquisition; S defaults to the workload's."""
    Sv = wl.S if S is None else int(S)
    fam = CONFIGS[wl.cfg]["family"]
    z = _rng(wl.seed, fam, STREAM_ZX).standard_normal((Sv, wl.n, wl.m))
    return z.astype(np.float32)
