"""Planted mistakes in the oracle must be caught by the pins.

Each test swaps one oracle routine for a subtly wrong variant (on the CPU)
and checks that the corresponding pin rejects it.
"""
import numpy as np

import oracle as O
from oracle import acq as oacq
from pins import hv_exact, ehvi_closed_form


def _setup(m, seed):
    r = np.random.default_rng(seed)
    Y = r.standard_normal((50, m))
    ref = Y.min(axis=0) - 0.1
    F = Y[O.pareto_front(Y, ref)]
    return F, ref, O.box_decomposition(F, ref)


def test_wrong_inclusion_exclusion_sign_is_caught(monkeypatch):
    F, ref, (lo, hi) = _setup(3, 1)
    Yq = np.random.default_rng(2).normal(0.5, 1.0, size=(4, 3))
    want = hv_exact(np.vstack([F, Yq]), ref) - hv_exact(F, ref)
    assert abs(O.qhvi(Yq, lo, hi) - want) < 1e-9
    orig = oacq._subsets
    monkeypatch.setattr(oacq, "_subsets", lambda q: [(J, 1.0) for J, _ in orig(q)])
    assert abs(oacq.qhvi(Yq, lo, hi) - want) > 1e-6


def test_missing_clamp_in_hvi_is_caught(monkeypatch):
    F, ref, (lo, hi) = _setup(2, 3)
    ys = np.random.default_rng(4).normal(0.0, 1.0, size=(50, 2))
    bad = lambda y, lo, hi: np.sum(np.prod(np.minimum(y[..., None, :], hi) - lo, axis=-1), axis=-1)
    base = hv_exact(F, ref)
    want = np.array([hv_exact(np.vstack([F, y]), ref) - base for y in ys])
    np.testing.assert_allclose(O.hvi(ys, lo, hi), want, rtol=1e-9, atol=1e-12)
    assert not np.allclose(bad(ys, lo, hi), want, rtol=1e-6, atol=1e-9)


def test_sigma_instead_of_variance_in_sampling_is_caught():
    F, ref, (lo, hi) = _setup(2, 5)
    mu = np.array([[1.0, 0.9]])
    sd = np.array([[0.5, 0.6]])
    cf = ehvi_closed_form(mu[0], sd[0], lo, hi)
    Z = np.random.default_rng(0).standard_normal((2 ** 17, 1, 2))
    h = O.hvi(mu + sd * Z[:, 0, :], lo, hi)
    se = h.std(ddof=1) / np.sqrt(len(h))
    good = O.ehvi_q1(mu, sd, Z, lo, hi)[0]
    bad = O.ehvi_q1(mu, sd ** 2, Z, lo, hi)[0]
    assert abs(good - cf) < 5 * se
    assert abs(bad - cf) > 50 * se
