"""Independent reference routines used to pin the oracle.

None of these calls into ``oracle``; each computes a quantity the oracle also
computes, by a different algorithm or a closed form, so a mistake in either
shows up as a disagreement.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
from scipy.special import gamma, kv, ndtr


def matern_bessel(rho: np.ndarray, nu: float) -> np.ndarray:
    """General Matern correlation through the modified Bessel function K_nu:
    2^{1-nu}/Gamma(nu) (sqrt(2 nu) rho)^nu K_nu(sqrt(2 nu) rho), 1 at rho = 0
    (Rasmussen & Williams 2006, eq. 4.14)."""
    rho = np.asarray(rho, dtype=np.float64)
    t = np.sqrt(2.0 * nu) * rho
    out = np.ones_like(t)
    pos = t > 0
    out[pos] = (2.0 ** (1.0 - nu) / gamma(nu)) * t[pos] ** nu * kv(nu, t[pos])
    return out


def hv2d_sweep(P: np.ndarray, ref: np.ndarray) -> float:
    """Dominated hypervolume (maximisation) of 2-D points above ref, by a
    sweep over x descending."""
    P = np.asarray(P, dtype=np.float64).reshape(-1, 2)
    P = P[np.all(P > ref, axis=1)]
    if len(P) == 0:
        return 0.0
    order = np.argsort(-P[:, 0], kind="stable")
    area = 0.0
    best_y = ref[1]
    for i, j in enumerate(order):
        x, y = P[j]
        best_y = max(best_y, y)
        x_next = P[order[i + 1], 0] if i + 1 < len(order) else ref[0]
        area += (x - x_next) * (best_y - ref[1])
    return area


def hv3d_slices(P: np.ndarray, ref: np.ndarray) -> float:
    """Dominated hypervolume of 3-D points above ref: slices along z, each
    slice's area by the 2-D sweep."""
    P = np.asarray(P, dtype=np.float64).reshape(-1, 3)
    P = P[np.all(P > ref, axis=1)]
    if len(P) == 0:
        return 0.0
    zs = np.unique(P[:, 2])[::-1]
    vol = 0.0
    for i, z in enumerate(zs):
        z_next = zs[i + 1] if i + 1 < len(zs) else ref[2]
        act = P[P[:, 2] >= z][:, :2]
        vol += hv2d_sweep(act, ref[:2]) * (z - z_next)
    return vol


def hv_exact(P: np.ndarray, ref: np.ndarray) -> float:
    ref = np.asarray(ref, dtype=np.float64)
    return hv2d_sweep(P, ref) if ref.shape[0] == 2 else hv3d_slices(P, ref)


def hv_grid_count(P: np.ndarray, ref: np.ndarray) -> int:
    """Count of unit cells dominated by integer points P above integer ref."""
    P = np.asarray(P, dtype=np.int64)
    ref = np.asarray(ref, dtype=np.int64)
    m = ref.shape[0]
    top = P.max(axis=0)
    count = 0
    for cell in itertools.product(*[range(int(ref[k]), int(top[k])) for k in range(m)]):
        upper = np.asarray(cell) + 1
        if np.any(np.all(P >= upper, axis=1)):
            count += 1
    return count


def front_bruteforce(Y: np.ndarray, ref: np.ndarray) -> list:
    """Non-dominated (maximise), deduplicated (lowest index), strictly above
    ref; returned as a set of indices."""
    Y = np.asarray(Y, dtype=np.float64)
    n = Y.shape[0]
    keep = []
    for i in range(n):
        if not np.all(Y[i] > ref):
            continue
        dominated = False
        for j in range(n):
            if j == i:
                continue
            if np.all(Y[j] >= Y[i]) and np.any(Y[j] > Y[i]):
                dominated = True
                break
            if np.all(Y[j] == Y[i]) and j < i:
                dominated = True
                break
        if not dominated:
            keep.append(i)
    return sorted(keep)


def psi(mu, sd, c):
    """E[(Y - c)_+] for Y ~ N(mu, sd^2); 0 for c = +inf."""
    mu = np.asarray(mu, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    out = np.zeros(np.broadcast(mu, c).shape)
    fin = np.broadcast_to(np.isfinite(c), out.shape)
    with np.errstate(invalid="ignore"):
        t = (mu - c) / sd
        val = sd * np.exp(-0.5 * t * t) / math.sqrt(2 * math.pi) + (mu - c) * ndtr(t)
    out[fin] = np.broadcast_to(val, out.shape)[fin]
    return out


def ehvi_closed_form(mu, sd, lo, hi) -> float:
    """Exact EHVI of one point with independent Gaussian objectives over
    disjoint boxes: sum_c prod_k (psi_k(lo_ck) - psi_k(hi_ck)), using
    [min(y,u) - l]_+ = (y - l)_+ - (y - u)_+ for l <= u."""
    mu = np.asarray(mu, dtype=np.float64)
    sd = np.asarray(sd, dtype=np.float64)
    total = 0.0
    for c in range(lo.shape[0]):
        prod = 1.0
        for k in range(lo.shape[1]):
            prod *= float(psi(mu[k], sd[k], lo[c, k]) - psi(mu[k], sd[k], hi[c, k]))
        total += prod
    return total


def _tail_first_moment(mu, sd, l, a):
    """E[(Y - l) 1[Y >= a]] for Y ~ N(mu, sd^2); 0 for a = +inf."""
    if not np.isfinite(a):
        return 0.0 if a > 0 else mu - l
    t = (a - mu) / sd
    return sd * math.exp(-0.5 * t * t) / math.sqrt(2 * math.pi) + (mu - l) * (1.0 - ndtr(t))


def _tail_prob(mu, sd, a):
    """P(Y >= a)."""
    if not np.isfinite(a):
        return 0.0 if a > 0 else 1.0
    return 1.0 - ndtr((a - mu) / sd)


def constrained_ehvi_closed_form(mu, sd, lo, hi, lower) -> float:
    """Exact E[HVI(Y) * prod_k 1[Y_k >= t_k]] for independent Gaussian
    objectives over disjoint boxes. The integrand factorises per objective;
    with a = max(l, t) each factor is
      E[(min(Y,u) - l) 1[Y >= a]]
        = (u - l) P(Y >= a)                                   if a >= u
        = E[(Y-l)1[Y>=a]] - E[(Y-l)1[Y>=u]] + (u-l) P(Y>=u)  otherwise,
    since [min(y,u) - l]_+ vanishes below l and the indicator below t."""
    mu = np.asarray(mu, dtype=np.float64)
    sd = np.asarray(sd, dtype=np.float64)
    lower = np.asarray(lower, dtype=np.float64)
    total = 0.0
    for c in range(lo.shape[0]):
        prod = 1.0
        for k in range(lo.shape[1]):
            l, u, t = float(lo[c, k]), float(hi[c, k]), float(lower[k])
            a = max(l, t)
            if a >= u:
                f = (u - l) * _tail_prob(mu[k], sd[k], a)
            else:
                f = _tail_first_moment(mu[k], sd[k], l, a)
                if np.isfinite(u):
                    f += -_tail_first_moment(mu[k], sd[k], l, u) + (u - l) * _tail_prob(mu[k], sd[k], u)
            prod *= f
        total += prod
    return total
