"""Gaussian-process surrogate, fp64 (test infrastructure, not the product path).

Paper: "Overall MOBO workflow" step (i) fits one GP per objective
(``SingleTaskGP`` models combined by ``ModelListGP``, implementation section),
with an ARD Matern kernel of smoothness 5/2 wrapped in a scale kernel, in
double precision. Hyperparameters are given here, not learned.

The paper's own surrogate (paragraphs "Additive kernels" and S5 "Model-GPU
preference encoding", and the implementation section's list of kernels) is
the composite kernel of ``composite_cov``: an ARD Matern-5/2 term on the
routing features, a preference-weighted ARD Matern-3/2 term on the
deployment features and their product as a low-weight interaction, each with
its own output scale.

Readings of points the paper does not state:

* Matern-5/2 is the standard form k(rho) = s (1 + sqrt5 rho + 5/3 rho^2)
  exp(-sqrt5 rho) with rho the lengthscale-scaled Euclidean distance
  (Rasmussen & Williams 2006, Section 4.2), s the output scale.
* Observation noise is homoscedastic Gaussian with variance eta added to the
  diagonal of the training covariance.
* The posterior is that of the latent function (no noise added to the
  predictive variance); variance is clamped at 0.
* The q x q batch covariance is factorised without jitter; a Schur pivot
  <= 1e-10 * s zeroes that column of the factor.
* Composite kernel (readings): the routing features are the first d_route
  coordinates and the deployment features the rest; the interaction is the
  product of the two unscaled Matern correlations with its own scale (the
  preference weight wraps only the deployment term, as the paper writes
  k~_c = w(c) w(c*) k_c); the weight is w(c) = exp(sum_j p_j c_j) with
  p_j = beta * (preference of the GPU type whose count dimension j encodes)
  folded into one slope per objective and deployment dimension. The
  pivot scale s of the batch factorisation is the sum of the three scales.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
from scipy.linalg import solve_triangular

SQRT5 = math.sqrt(5.0)
SQRT3 = math.sqrt(3.0)
PIVOT_RTOL = 1e-10


class NotPositiveDefinite(ValueError):
    """The training covariance matrix of some objective is not PD."""


def scaled_distance(U: np.ndarray, V: np.ndarray, ls: np.ndarray, rows: int = 16) -> np.ndarray:
    """rho[i, j] = sqrt(sum_t ((U[i,t] - V[j,t]) / ls[t])^2), direct differences.

    Computed ``rows`` rows of U at a time, so the [rows, len(V), d] array of
    differences stays small."""
    U = np.asarray(U, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    ls = np.asarray(ls, dtype=np.float64)
    out = np.empty((U.shape[0], V.shape[0]))
    for i0 in range(0, U.shape[0], rows):
        D = (U[i0:i0 + rows, None, :] - V[None, :, :]) / ls
        out[i0:i0 + rows] = np.sqrt(np.einsum("ijt,ijt->ij", D, D))
    return out


def matern52(rho: np.ndarray, s: float) -> np.ndarray:
    """Matern nu=5/2 covariance of scaled distance ``rho`` with output scale s."""
    rho = np.asarray(rho, dtype=np.float64)
    return float(s) * (1.0 + SQRT5 * rho + (5.0 / 3.0) * rho * rho) * np.exp(-SQRT5 * rho)


def matern32(rho: np.ndarray, s: float) -> np.ndarray:
    """Matern nu=3/2 covariance: s (1 + sqrt3 rho) exp(-sqrt3 rho)
    (Rasmussen & Williams 2006, eq. 4.17)."""
    rho = np.asarray(rho, dtype=np.float64)
    return float(s) * (1.0 + SQRT3 * rho) * np.exp(-SQRT3 * rho)


@dataclass
class Composite:
    """Hyperparameters of the composite kernel for all objectives.

    d_route: number of routing features (the first coordinates);
    s_route, s_dep, s_int [m]: output scales of the routing term, the
    preference-weighted deployment term and the interaction;
    pref [m, d - d_route]: log-weight slopes of the deployment features."""
    d_route: int
    s_route: np.ndarray
    s_dep: np.ndarray
    s_int: np.ndarray
    pref: np.ndarray


def pref_weight(C: np.ndarray, p: np.ndarray) -> np.ndarray:
    """w(c) = exp(sum_j p_j c_j) for deployment features C [N, d_c]."""
    return np.exp(np.asarray(C, dtype=np.float64) @ np.asarray(p, dtype=np.float64))


def composite_cov(U, V, ls, comp: Composite, k: int) -> np.ndarray:
    """k(u, v) = s_route M52(rho_route) + s_dep w(u_c) w(v_c) M32(rho_dep)
                 + s_int M52(rho_route) M32(rho_dep)
    for objective k; M52, M32 unit-scale Matern correlations, rho_* the
    ARD-scaled distances over the routing / deployment coordinates."""
    U = np.asarray(U, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    dr = comp.d_route
    k5 = matern52(scaled_distance(U[:, :dr], V[:, :dr], ls[:dr]), 1.0)
    k3 = matern32(scaled_distance(U[:, dr:], V[:, dr:], ls[dr:]), 1.0)
    wu = pref_weight(U[:, dr:], comp.pref[k])
    wv = pref_weight(V[:, dr:], comp.pref[k])
    return (comp.s_route[k] * k5 + comp.s_dep[k] * np.outer(wu, wv) * k3
            + comp.s_int[k] * k5 * k3)


@dataclass
class GPModel:
    X: np.ndarray            # [n, d]
    Y: np.ndarray            # [n, m]
    ls: np.ndarray           # [m, d]
    s: np.ndarray            # [m]
    eta: np.ndarray          # [m]
    L: List[np.ndarray] = field(default_factory=list)      # m x [n, n] lower
    alpha: List[np.ndarray] = field(default_factory=list)  # m x [n]
    comp: Optional[Composite] = None                       # None: Matern-5/2

    def cov(self, k: int, U, V) -> np.ndarray:
        """Covariance matrix of objective k between point sets U and V."""
        if self.comp is None:
            return matern52(scaled_distance(U, V, self.ls[k]), self.s[k])
        return composite_cov(U, V, self.ls[k], self.comp, k)

    def pair_cov(self, k: int, U, V) -> np.ndarray:
        """k(U[i], V[i]) for paired rows (the diagonal of cov(k, U, V))."""
        U = np.asarray(U, dtype=np.float64)
        V = np.asarray(V, dtype=np.float64)

        def rho(a, b, ls):
            diff = (a - b) / ls
            return np.sqrt(np.sum(diff * diff, axis=1))
        if self.comp is None:
            return matern52(rho(U, V, self.ls[k]), self.s[k])
        c, dr, ls = self.comp, self.comp.d_route, self.ls[k]
        k5 = matern52(rho(U[:, :dr], V[:, :dr], ls[:dr]), 1.0)
        k3 = matern32(rho(U[:, dr:], V[:, dr:], ls[dr:]), 1.0)
        w = pref_weight(U[:, dr:], c.pref[k]) * pref_weight(V[:, dr:], c.pref[k])
        return c.s_route[k] * k5 + c.s_dep[k] * w * k3 + c.s_int[k] * k5 * k3

    @property
    def n(self) -> int:
        return self.X.shape[0]

    @property
    def m(self) -> int:
        return self.Y.shape[1]


def fit(X, Y, ls, s, eta, composite: Optional[Composite] = None) -> GPModel:
    """Condition one GP per objective on (X, Y[:, k]).

    K_k = [k_k(x_i, x_j)] + eta_k I;  L_k = chol(K_k) (lower);
    alpha_k = L_k^T \\ (L_k \\ y_k).
    k_k is the ARD Matern-5/2 with output scale s_k, or the composite kernel
    when ``composite`` is given (then ``s`` is ignored).
    Raises NotPositiveDefinite when a factorisation fails.
    """
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    ls = np.asarray(ls, dtype=np.float64).reshape(Y.shape[1], X.shape[1])
    eta = np.asarray(eta, dtype=np.float64).reshape(-1)
    if composite is not None:
        c = composite
        composite = Composite(int(c.d_route), *[np.asarray(v, dtype=np.float64) for v in
                                                (c.s_route, c.s_dep, c.s_int, c.pref)])
        s = composite.s_route + composite.s_dep + composite.s_int
    s = np.asarray(s, dtype=np.float64).reshape(-1)
    model = GPModel(X=X, Y=Y, ls=ls, s=s, eta=eta, comp=composite)
    n = X.shape[0]
    for k in range(Y.shape[1]):
        K = model.cov(k, X, X) + eta[k] * np.eye(n)
        try:
            L = np.linalg.cholesky(K)
        except np.linalg.LinAlgError as e:  # pragma: no cover - message path
            raise NotPositiveDefinite(f"objective {k}: {e}") from e
        if not np.all(np.isfinite(L)):
            raise NotPositiveDefinite(f"objective {k}: non-finite factor")
        w = solve_triangular(L, Y[:, k], lower=True)
        alpha = solve_triangular(L.T, w, lower=False)
        model.L.append(L)
        model.alpha.append(alpha)
    return model


def posterior(model: GPModel, cand: np.ndarray, chunk: int = 512):
    """Posterior of every objective at a set of q-batches.

    cand: [B, q, d]. Returns (mu [B, q, m], cov [B, m, q, q]).
    For each point x*: k* = k(x*, X), mu = k*^T alpha, v = L \\ k* (forward
    substitution), and for a batch Sigma[a, b] = k(x*_a, x*_b) - v_a^T v_b.
    The diagonal is clamped at 0 (variance of the latent function).
    """
    cand = np.asarray(cand, dtype=np.float64)
    B, q, d = cand.shape
    m = model.m
    mu = np.zeros((B, q, m))
    cov = np.zeros((B, m, q, q))
    for b0 in range(0, B, chunk):
        b1 = min(B, b0 + chunk)
        P = cand[b0:b1].reshape(-1, d)
        nb = b1 - b0
        for k in range(m):
            Ks = model.cov(k, P, model.X)
            mu[b0:b1, :, k] = (Ks @ model.alpha[k]).reshape(nb, q)
            V = solve_triangular(model.L[k], Ks.T, lower=True)   # [n, nb*q]
            Vb = V.T.reshape(nb, q, -1)
            Pb = cand[b0:b1]
            prior = np.empty((nb, q, q))
            for a in range(q):
                for c in range(q):
                    prior[:, a, c] = model.pair_cov(k, Pb[:, a, :], Pb[:, c, :])
            S = prior - Vb @ np.transpose(Vb, (0, 2, 1))
            idx = np.arange(q)
            S[:, idx, idx] = np.maximum(S[:, idx, idx], 0.0)
            cov[b0:b1, k] = S
    return mu, cov


def chol_psd(Sig: np.ndarray, s) -> np.ndarray:
    """Lower Cholesky factor of a batch of PSD q x q matrices, no jitter.

    Sig: [..., q, q]; s: output scale (broadcast over the leading axes).
    Column j is computed from the Schur pivot p = Sig[j,j] - sum_{t<j} C[j,t]^2;
    if p <= 1e-10 * s the whole column j of C is zero, otherwise
    C[j,j] = sqrt(p) and C[i,j] = (Sig[i,j] - sum_{t<j} C[i,t] C[j,t]) / C[j,j].
    """
    Sig = np.asarray(Sig, dtype=np.float64)
    q = Sig.shape[-1]
    s = np.broadcast_to(np.asarray(s, dtype=np.float64), Sig.shape[:-2])
    C = np.zeros_like(Sig)
    for j in range(q):
        p = Sig[..., j, j] - np.sum(C[..., j, :j] ** 2, axis=-1)
        ok = p > PIVOT_RTOL * s
        cjj = np.where(ok, np.sqrt(np.where(ok, p, 1.0)), 0.0)
        C[..., j, j] = cjj
        for i in range(j + 1, q):
            num = Sig[..., i, j] - np.sum(C[..., i, :j] * C[..., j, :j], axis=-1)
            C[..., i, j] = np.where(ok, num / np.where(ok, cjj, 1.0), 0.0)
    return C


def mll(X, Y, ls, s, eta):
    """Exact log marginal likelihood of each objective's GP and its gradient.

    Paper: implementation section (lengthscales learned by maximising the GP
    marginal likelihood). For objective k with K = s M52 + eta I:
      log p(y) = -1/2 y^T K^{-1} y - 1/2 log det K - n/2 log(2 pi),
    log det K = 2 sum_i log L_ii. Gradient with respect to
    theta = (log l_1 .. log l_d, log s, log eta):
      d log p / d theta_j = 1/2 tr((alpha alpha^T - K^{-1}) dK/dtheta_j),
    with dK/dlog l_t = (5/3) s (1 + sqrt5 r) exp(-sqrt5 r) u_t^2
    (u_t = (x_it - x_i't) / l_t), dK/dlog s = s M52, dK/dlog eta = eta I.
    Returns (value [m], grad [m, d + 2]).
    """
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    n, d = X.shape
    m = Y.shape[1]
    ls = np.asarray(ls, dtype=np.float64).reshape(m, d)
    s = np.asarray(s, dtype=np.float64).reshape(-1)
    eta = np.asarray(eta, dtype=np.float64).reshape(-1)
    value = np.zeros(m)
    grad = np.zeros((m, d + 2))
    for k in range(m):
        U = X / ls[k]                                      # scaled coordinates
        D = U[:, None, :] - U[None, :, :]                  # [n, n, d]
        r = np.sqrt(np.sum(D * D, axis=2))
        K0 = matern52(r, s[k])
        K = K0 + eta[k] * np.eye(n)
        L = np.linalg.cholesky(K)
        alpha = solve_triangular(L.T, solve_triangular(L, Y[:, k], lower=True), lower=False)
        value[k] = (-0.5 * Y[:, k] @ alpha - np.sum(np.log(np.diag(L)))
                    - 0.5 * n * math.log(2.0 * math.pi))
        Linv = solve_triangular(L, np.eye(n), lower=True)
        A = np.outer(alpha, alpha) - Linv.T @ Linv
        common = (5.0 / 3.0) * s[k] * (1.0 + SQRT5 * r) * np.exp(-SQRT5 * r)
        for t in range(d):
            grad[k, t] = 0.5 * np.sum(A * common * D[:, :, t] ** 2)
        grad[k, d] = 0.5 * np.sum(A * K0)
        grad[k, d + 1] = 0.5 * eta[k] * np.trace(A)
    return value, grad
