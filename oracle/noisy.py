"""Noisy expected hypervolume improvement (qNEHVI) of candidates and q-batches, fp64.

Test infrastructure only: the GPU library never imports this module.

Paper: "Overall MOBO workflow" step (ii) and the constrained qNEHVI
paragraph (after Daulton, Balandat & Bakshy, NeurIPS 2021). The noisy form
does not trust the observed Y as the current front: the observations are
noisy, so the latent objective values at the observed points are uncertain
as well. Each Monte-Carlo sample draws the latent objectives jointly at the
observed points X and at the candidate x* from the GP posterior; the
candidate's improvement in that sample is measured against the Pareto front
of that sample's in-sample values.

Readings (the paper names the acquisition but does not spell it out):

* Joint posterior of the latent f (no noise term) at [X; x*], per objective
  (independent GPs), with K = K_XX + eta I:
      mu_X      = K_XX K^{-1} y,            mu* = k*^T K^{-1} y,
      Sigma_XX  = K_XX - K_XX K^{-1} K_XX,  Sigma_*X = k*^T - k*^T K^{-1} K_XX,
      Sigma_**  = s - k*^T K^{-1} k*.
* Sampling by the lower Cholesky factor of that joint covariance, written
  in block form: with L_XX = chol(Sigma_XX) and base samples z_X [n],
  z* (iid N(0, 1)),
      f_X = mu_X + L_XX z_X,
      f*  = mu* + B^T z_X + c z*,   B = L_XX^{-1} Sigma_X*,  c^2 = Sigma_** - |B|^2
  (the factor of [[Sigma_XX, Sigma_X*], [Sigma_*X, Sigma_**]] is
  [[L_XX, 0], [B^T, c]]); c^2 is clamped at 0.
* Base samples z_X [S, n, m] and z* [S, m] are common to all candidates
  (common random numbers), so the in-sample fronts are shared.
* Front of sample s: the non-dominated in-sample vectors f_X^s (maximise,
  duplicates keep the lowest index) strictly above r; with feasibility
  thresholds, only in-sample vectors meeting all of them take part.
* HVI of f*^s against the disjoint boxes of that front; the constrained
  form multiplies it by the feasibility indicator of f*^s.
* qNEHVI = plain mean over the S samples.
* q-batches (the paper's q): the members x*_1..x*_q are drawn jointly with
  f_X the same way, with B = L_XX^{-1} Sigma_XB [n, q] and the conditional
  batch covariance Sigma_BB - B^T B factored by the PSD Cholesky rule of
  ``gp.chol_psd``; the batch improvement of a draw is the joint HVI of its
  members (inclusion-exclusion, ``acq.qhvi``) against that draw's boxes, a
  member counting only where it is feasible.
"""
from __future__ import annotations

import numpy as np
from scipy.linalg import cho_solve, solve_triangular

from .gp import GPModel, chol_psd
from .pareto import pareto_front, box_decomposition
from .acq import hvi, qhvi, feasible


def insample_posterior(model: GPModel):
    """Posterior of the latent objectives at the observed points.

    Returns mu_X [n, m] and a list of m covariance matrices Sigma_XX [n, n]."""
    X = model.X
    mu = np.empty((model.n, model.m))
    cov = []
    for k in range(model.m):
        Kxx = model.cov(k, X, X)
        KinvKxx = cho_solve((model.L[k], True), Kxx)
        mu[:, k] = Kxx @ model.alpha[k]
        S = Kxx - Kxx @ KinvKxx
        cov.append(0.5 * (S + S.T))
    return mu, cov


def insample_samples(model: GPModel, ZX: np.ndarray):
    """f_X^s = mu_X + L_XX z_X^s for every sample: F [S, n, m].

    Also returns the factors L_XX (list of m [n, n])."""
    ZX = np.asarray(ZX, dtype=np.float64)
    mu, cov = insample_posterior(model)
    Ls = [np.linalg.cholesky(c) for c in cov]
    F = np.empty(ZX.shape)
    for k in range(model.m):
        F[:, :, k] = mu[None, :, k] + ZX[:, :, k] @ Ls[k].T
    return F, Ls


def candidate_samples(model: GPModel, cand: np.ndarray, ZX: np.ndarray, Zs: np.ndarray,
                      Ls=None, Kxx=None):
    """Joint-posterior samples of the candidates: f* [M, S, m].

    cand [M, d]; ZX [S, n, m]; Zs [S, m]. Ls: the in-sample factors, Kxx: the
    noise-free training covariances (both lists over objectives; computed
    when not given)."""
    cand = np.asarray(cand, dtype=np.float64).reshape(-1, model.X.shape[1])
    ZX = np.asarray(ZX, dtype=np.float64)
    Zs = np.asarray(Zs, dtype=np.float64).reshape(ZX.shape[0], model.m)
    if Ls is None:
        _, Ls = insample_samples(model, ZX)
    X = model.X
    M = cand.shape[0]
    out = np.empty((M, ZX.shape[0], model.m))
    for k in range(model.m):
        Ks = model.cov(k, cand, X)                              # [M, n] = k*^T
        Kk = model.cov(k, X, X) if Kxx is None else Kxx[k]
        mu_s = Ks @ model.alpha[k]
        KinvKs = cho_solve((model.L[k], True), Ks.T)            # [n, M] = K^{-1} k*
        var_s = model.pair_cov(k, cand, cand) - np.sum(Ks.T * KinvKs, axis=0)
        Sx = Ks.T - Kk @ KinvKs                                 # [n, M] = Sigma_X*
        Bm = solve_triangular(Ls[k], Sx, lower=True)            # [n, M]
        c2 = np.maximum(var_s - np.sum(Bm * Bm, axis=0), 0.0)
        out[:, :, k] = (mu_s[:, None] + Bm.T @ ZX[:, :, k].T
                        + np.sqrt(c2)[:, None] * Zs[None, :, k])
    return out


def batch_samples(model: GPModel, cand: np.ndarray, ZX: np.ndarray, Zs: np.ndarray,
                  Ls=None, Kxx=None):
    """Joint-posterior samples of q-batches: f* [M, S, q, m].

    cand [M, q, d]; ZX [S, n, m]; Zs [S, q, m]. The batch block of the joint
    factor is the PSD Cholesky factor of Sigma_BB - B^T B (B = L_XX^{-1}
    Sigma_XB), applied to z*_s."""
    cand = np.asarray(cand, dtype=np.float64)
    M, q, d = cand.shape
    ZX = np.asarray(ZX, dtype=np.float64)
    S = ZX.shape[0]
    Zs = np.asarray(Zs, dtype=np.float64).reshape(S, q, model.m)
    if Ls is None:
        _, Ls = insample_samples(model, ZX)
    X = model.X
    P = cand.reshape(M * q, d)
    out = np.empty((M, S, q, model.m))
    for k in range(model.m):
        Ks = model.cov(k, P, X)                                 # [Mq, n]
        Kk = model.cov(k, X, X) if Kxx is None else Kxx[k]
        mu_s = (Ks @ model.alpha[k]).reshape(M, q)
        KinvKs = cho_solve((model.L[k], True), Ks.T)            # [n, Mq]
        Sx = Ks.T - Kk @ KinvKs                                 # [n, Mq] = Sigma_X*
        Bm = solve_triangular(Ls[k], Sx, lower=True)            # [n, Mq]
        Bb = Bm.T.reshape(M, q, -1)                             # [M, q, n]
        prior = np.empty((M, q, q))
        for a in range(q):
            for c in range(q):
                prior[:, a, c] = model.pair_cov(k, cand[:, a, :], cand[:, c, :])
        Kb = Ks.reshape(M, q, -1)
        KinvKb = KinvKs.T.reshape(M, q, -1)
        post = prior - np.einsum("mai,mbi->mab", Kb, KinvKb)    # Sigma_BB
        cond = post - np.einsum("mai,mbi->mab", Bb, Bb)
        C = chol_psd(cond, model.s[k])                          # [M, q, q]
        off = np.einsum("mai,si->msa", Bb, ZX[:, :, k])         # [M, S, q]
        out[:, :, :, k] = (mu_s[:, None, :] + off
                           + np.einsum("mab,sb->msa", C, Zs[:, :, k]))
    return out


def sample_boxes(F: np.ndarray, ref: np.ndarray, lower=None):
    """Boxes of each sample's in-sample front: list of (lo, hi) per sample.

    F [S, n, m]; rows failing a feasibility threshold are left out."""
    ref = np.asarray(ref, dtype=np.float64)
    out = []
    for s in range(F.shape[0]):
        Fs = F[s]
        if lower is not None:
            Fs = Fs[feasible(Fs, lower) > 0]
        front = pareto_front(Fs, ref)
        out.append(box_decomposition(Fs[front], ref))
    return out


def nehvi(model: GPModel, cand: np.ndarray, ref: np.ndarray, ZX: np.ndarray,
          Zs: np.ndarray, lower=None, chunk: int = 1024):
    """qNEHVI of M candidates [M, d] (q = 1) or q-batches [M, q, d].

    ZX [S, n, m] in-sample base samples; Zs [S, m] (q = 1) or [S, q, m]
    candidate base samples; lower [m] optional feasibility thresholds.
    Returns a dict with ``ehvi`` [M], the in-sample samples ``F`` [S, n, m]
    and the per-sample ``boxes``.
    """
    cand = np.asarray(cand, dtype=np.float64)
    ZX = np.asarray(ZX, dtype=np.float64)
    S = ZX.shape[0]
    batched = cand.ndim == 3 and cand.shape[1] > 1
    if not batched:
        cand = cand.reshape(cand.shape[0], -1)
        Zs = np.asarray(Zs, dtype=np.float64).reshape(S, model.m)
    F, Ls = insample_samples(model, ZX)
    Kxx = [model.cov(k, model.X, model.X) for k in range(model.m)]
    boxes = sample_boxes(F, ref, lower)
    M = cand.shape[0]
    out = np.empty(M)
    if batched:
        chunk = max(1, chunk // cand.shape[1])
    for i0 in range(0, M, chunk):
        i1 = min(M, i0 + chunk)
        if not batched:
            ys = candidate_samples(model, cand[i0:i1], ZX, Zs, Ls, Kxx)    # [c, S, m]
            h = np.empty((i1 - i0, S))
            for s in range(S):
                lo, hi = boxes[s]
                h[:, s] = hvi(ys[:, s, :], lo, hi)
            if lower is not None:
                h = h * feasible(ys, lower)
        else:
            ys = batch_samples(model, cand[i0:i1], ZX, Zs, Ls, Kxx)        # [c, S, q, m]
            feas = None if lower is None else feasible(ys, lower)           # [c, S, q]
            h = np.empty((i1 - i0, S))
            for s in range(S):
                lo, hi = boxes[s]
                h[:, s] = qhvi(ys[:, s], lo, hi, None if feas is None else feas[:, s])
        out[i0:i1] = np.mean(h, axis=1)
    return dict(ehvi=out, F=F, boxes=boxes)
