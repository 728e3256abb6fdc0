"""Hypervolume improvement, Monte-Carlo (q)EHVI and argmax, fp64.

Test infrastructure only. Paper: constrained qNEHVI paragraph — the
acquisition is the expectation, over samples of the joint posterior of the
objectives, of the hypervolume improvement (HVI) of a candidate, estimated by
Monte-Carlo integration; "Overall MOBO workflow" step (ii) picks the candidate
that maximises it. Here (readings):

* HVI is the Lebesgue measure, in standardised objective space, of the part
  of the region dominated by the candidate (or, for a q-batch, by any member)
  and bounded below by r that the current front does not already dominate.
  With the region {z > r : z not weakly dominated by F} split into disjoint
  boxes [lo_c, hi_c):
      HVI(y) = sum_c prod_k [min(y_k, hi_ck) - lo_ck]_+ .
  For a batch Y = {y_1..y_q} the union of the boxes [r, y_a] is expanded by
  inclusion-exclusion over non-empty subsets J (the q-batch form of
  Daulton, Balandat & Bakshy, NeurIPS 2020):
      qHVI(Y) = sum_{J} (-1)^{|J|+1} sum_c prod_k [min(min_{a in J} y_ak, hi_ck) - lo_ck]_+ .
* MC estimator: the plain mean over the S given base samples (common to all
  candidates). q = 1: y_s = mu + sigma * z_s.
  q > 1: y_s[a, k] = mu[a, k] + sum_b C_k[a, b] z_s[b, k] with C_k the PSD
  Cholesky factor of the batch covariance of objective k (objectives are
  independent GPs, so each has its own factor).
* Feasibility (optional): the constrained form of the same paragraph
  multiplies each sample's HVI by the indicator that every constraint
  g_i <= 0 holds on that sample. Its constraints bound the objectives
  themselves (a latency cap and a quality floor), so in the maximised,
  standardised objectives each reads y_k >= t_k, one lower threshold per
  objective (-inf: unconstrained). For a q-batch, a member counts only on
  the samples where it is feasible: every inclusion-exclusion term of a
  subset J is multiplied by the product of its members' indicators (the
  constrained qEHVI of Daulton, Balandat & Bakshy 2020), i.e. the HVI of the
  feasible members.
* argmax: first index of the maximum, NaN never wins; all-NaN gives -1.
"""
from __future__ import annotations

import itertools

import numpy as np

from .gp import GPModel, posterior, chol_psd
from .pareto import pareto_front, box_decomposition


def hvi(y: np.ndarray, lo: np.ndarray, hi: np.ndarray) -> np.ndarray:
    """HVI of points y [..., m] against disjoint boxes lo/hi [B, m]."""
    y = np.asarray(y, dtype=np.float64)
    ext = np.minimum(y[..., None, :], hi) - lo          # [..., B, m]
    ext = np.maximum(ext, 0.0)
    return np.sum(np.prod(ext, axis=-1), axis=-1)


def _subsets(q: int):
    out = []
    for size in range(1, q + 1):
        for J in itertools.combinations(range(q), size):
            out.append((J, 1.0 if size % 2 == 1 else -1.0))
    return out


def feasible(ys: np.ndarray, lower) -> np.ndarray:
    """Indicator [...] that a sample ys [..., m] meets every constraint
    g_k = lower_k - y_k <= 0 (lower_k = -inf: objective k unconstrained)."""
    ys = np.asarray(ys, dtype=np.float64)
    lower = np.asarray(lower, dtype=np.float64)
    return np.all(ys >= lower, axis=-1).astype(np.float64)


def qhvi(Y: np.ndarray, lo: np.ndarray, hi: np.ndarray, feas=None) -> np.ndarray:
    """Joint HVI of q-batches Y [..., q, m] by inclusion-exclusion.

    feas [..., q] (optional): member feasibility indicators; the term of a
    subset J is weighted by prod_{a in J} feas[..., a]."""
    Y = np.asarray(Y, dtype=np.float64)
    q = Y.shape[-2]
    total = np.zeros(Y.shape[:-2])
    for J, sign in _subsets(q):
        corner = np.min(Y[..., list(J), :], axis=-2)      # [..., m]
        term = hvi(corner, lo, hi)
        if feas is not None:
            term = term * np.prod(np.asarray(feas)[..., list(J)], axis=-1)
        total = total + sign * term
    return total


def ehvi_q1(mu: np.ndarray, sigma: np.ndarray, Z: np.ndarray,
            lo: np.ndarray, hi: np.ndarray, chunk: int = 256,
            lower=None) -> np.ndarray:
    """MC-EHVI of single points. mu, sigma [N, m]; Z [S, 1, m] or [S, m].
    lower [m] (optional): feasibility thresholds; each sample's HVI is
    multiplied by its feasibility indicator."""
    mu = np.asarray(mu, dtype=np.float64)
    sigma = np.asarray(sigma, dtype=np.float64)
    Z = np.asarray(Z, dtype=np.float64).reshape(Z.shape[0], -1)
    N = mu.shape[0]
    out = np.empty(N)
    for i0 in range(0, N, chunk):
        i1 = min(N, i0 + chunk)
        ys = mu[i0:i1, None, :] + sigma[i0:i1, None, :] * Z[None, :, :]   # [c, S, m]
        h = hvi(ys, lo, hi)
        if lower is not None:
            h = h * feasible(ys, lower)
        out[i0:i1] = np.mean(h, axis=1)
    return out


def qehvi(mu: np.ndarray, C: np.ndarray, Z: np.ndarray,
          lo: np.ndarray, hi: np.ndarray, chunk: int = 8,
          lower=None) -> np.ndarray:
    """MC-qEHVI. mu [N, q, m]; C [N, m, q, q] lower factors; Z [S, q, m].
    lower [m] (optional): feasibility thresholds applied per member."""
    mu = np.asarray(mu, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    Z = np.asarray(Z, dtype=np.float64)
    N = mu.shape[0]
    out = np.empty(N)
    for i0 in range(0, N, chunk):
        i1 = min(N, i0 + chunk)
        # ys[c, s, a, k] = mu[c, a, k] + sum_b C[c, k, a, b] Z[s, b, k]
        corr = np.einsum("ckab,sbk->csak", C[i0:i1], Z)
        ys = mu[i0:i1, None, :, :] + corr
        feas = None if lower is None else feasible(ys, lower)   # [c, S, q]
        out[i0:i1] = np.mean(qhvi(ys, lo, hi, feas), axis=1)
    return out


def score(model: GPModel, cand: np.ndarray, ref: np.ndarray, Z: np.ndarray,
          lower=None):
    """Posterior plus MC acquisition of M candidates (q-batches).

    cand [M, q, d]; ref [m]; Z [S, q, m]; lower [m] optional feasibility
    thresholds (None: no constraint). Returns a dict with ``ehvi`` [M],
    ``mu`` [M, q, m], ``sigma`` [M, q, m] (marginal posterior std),
    ``front`` (indices into Y) and the boxes ``lo``/``hi``.
    """
    cand = np.asarray(cand, dtype=np.float64)
    M, q, _ = cand.shape
    ref = np.asarray(ref, dtype=np.float64)
    front = pareto_front(model.Y, ref)
    lo, hi = box_decomposition(model.Y[front], ref)
    mu, cov = posterior(model, cand)
    var = np.diagonal(cov, axis1=-2, axis2=-1)             # [M, m, q]
    sigma = np.sqrt(np.transpose(var, (0, 2, 1)))          # [M, q, m]
    if q == 1:
        e = ehvi_q1(mu[:, 0, :], sigma[:, 0, :], Z, lo, hi, lower=lower)
    else:
        Cf = chol_psd(cov, model.s[None, :])
        e = qehvi(mu, Cf, Z, lo, hi, lower=lower)
    return dict(ehvi=e, mu=mu, sigma=sigma, front=front, lo=lo, hi=hi, cov=cov)


def argmax(values: np.ndarray):
    """(index, value) of the maximum; lowest index on ties; NaN never wins."""
    v = np.asarray(values, dtype=np.float64)
    ok = ~np.isnan(v)
    if not np.any(ok):
        return -1, float("nan")
    best = np.max(v[ok])
    idx = int(np.nonzero(ok & (v == best))[0][0])
    return idx, float(v[idx])
