"""Pins for the feasibility-weighted acquisition of the oracle (the
constrained form: each sample's HVI times the indicator that every
constraint holds on it; thresholds are lower bounds on the maximised,
standardised objectives)."""
import numpy as np
import pytest

import oracle as O
from oracle import acq as oacq
from pins import hv_exact, constrained_ehvi_closed_form, ehvi_closed_form


def _front(m, seed, n=60):
    r = np.random.default_rng(seed)
    Y = r.standard_normal((n, m))
    ref = Y.min(axis=0) - 0.1
    F = Y[O.pareto_front(Y, ref)]
    lo, hi = O.box_decomposition(F, ref)
    return F, ref, lo, hi


@pytest.mark.parametrize("m", [2, 3])
def test_minus_inf_thresholds_reduce_to_unconstrained(m):
    F, ref, lo, hi = _front(m, 1)
    r = np.random.default_rng(2)
    mu = r.normal(0.5, 0.5, size=(40, m))
    sd = r.uniform(0.1, 1.0, size=(40, m))
    Z = r.standard_normal((256, 1, m))
    a = O.ehvi_q1(mu, sd, Z, lo, hi)
    b = O.ehvi_q1(mu, sd, Z, lo, hi, lower=np.full(m, -np.inf))
    np.testing.assert_array_equal(a, b)
    c = O.ehvi_q1(mu, sd, Z, lo, hi, lower=np.full(m, np.inf))
    assert np.all(c == 0.0)


@pytest.mark.parametrize("m", [2, 3])
def test_mc_converges_to_closed_form(m):
    F, ref, lo, hi = _front(m, 10 + m)
    mu = np.full(m, 0.8)
    sd = np.linspace(0.4, 0.9, m)
    # one threshold inside the front's span, one below the reference point
    # (inactive), and for m = 3 one above every box's lower corner
    lower = [np.median(F[:, 0]), ref[1] - 1.0]
    if m == 3:
        lower.append(F[:, 2].max())
    lower = np.array(lower)
    cf = constrained_ehvi_closed_form(mu, sd, lo, hi, lower)
    assert cf < ehvi_closed_form(mu, sd, lo, hi)
    for S in (2 ** 14, 2 ** 18):
        Z = np.random.default_rng(S).standard_normal((S, 1, m))
        ys = mu + sd * Z[:, 0, :]
        h = O.hvi(ys, lo, hi) * np.all(ys >= lower, axis=1)
        se = h.std(ddof=1) / np.sqrt(S)
        e = O.ehvi_q1(mu[None, :], sd[None, :], Z, lo, hi, lower=lower)[0]
        assert abs(e - cf) < 5 * se, (S, e, cf, se)


@pytest.mark.parametrize("m,q", [(2, 2), (2, 4), (3, 3), (3, 4)])
def test_batch_term_weighting_equals_hv_of_feasible_members(m, q):
    F, ref, lo, hi = _front(m, 30 + 7 * q + m, n=40)
    base = hv_exact(F, ref)
    r = np.random.default_rng(q * 10 + m)
    for _ in range(12):
        Yq = r.normal(0.3, 1.0, size=(q, m))
        feas = (r.random(q) < 0.6).astype(float)
        want = hv_exact(np.vstack([F, Yq[feas > 0]]), ref) - base
        got = O.qhvi(Yq, lo, hi, feas)
        assert got == pytest.approx(want, abs=1e-9)


def test_qehvi_feasibility_per_member_matches_q1_path():
    F, ref, lo, hi = _front(2, 7)
    r = np.random.default_rng(8)
    mu = r.normal(0.5, 0.4, size=(10, 1, 2))
    sd = r.uniform(0.2, 0.8, size=(10, 1, 2))
    C = np.zeros((10, 2, 1, 1))
    C[:, :, 0, 0] = sd[:, 0, :]
    Z = r.standard_normal((300, 1, 2))
    lower = np.array([0.2, -np.inf])
    a = O.qehvi(mu, C, Z, lo, hi, lower=lower)
    b = O.ehvi_q1(mu[:, 0], sd[:, 0], Z, lo, hi, lower=lower)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-15)


def test_raising_a_threshold_never_increases_the_acquisition():
    F, ref, lo, hi = _front(2, 9)
    r = np.random.default_rng(10)
    mu = r.normal(0.5, 0.5, size=(30, 2))
    sd = r.uniform(0.1, 1.0, size=(30, 2))
    Z = r.standard_normal((512, 1, 2))
    prev = O.ehvi_q1(mu, sd, Z, lo, hi)
    for t in np.linspace(-2.0, 2.0, 9):
        cur = O.ehvi_q1(mu, sd, Z, lo, hi, lower=np.array([t, -np.inf]))
        assert np.all(cur <= prev + 1e-15)
        prev = cur


def test_reversed_constraint_direction_is_caught(monkeypatch):
    F, ref, lo, hi = _front(2, 11)
    mu = np.array([0.9, 0.9])
    sd = np.array([0.5, 0.6])
    lower = np.array([np.median(F[:, 0]), np.median(F[:, 1]) - 0.5])
    cf = constrained_ehvi_closed_form(mu, sd, lo, hi, lower)
    Z = np.random.default_rng(0).standard_normal((2 ** 17, 1, 2))
    good = O.ehvi_q1(mu[None], sd[None], Z, lo, hi, lower=lower)[0]
    monkeypatch.setattr(oacq, "feasible",
                        lambda ys, lo_: np.all(np.asarray(ys) <= lo_, axis=-1).astype(float))
    bad = oacq.ehvi_q1(mu[None], sd[None], Z, lo, hi, lower=lower)[0]
    ys = mu + sd * Z[:, 0, :]
    se = (O.hvi(ys, lo, hi) * np.all(ys >= lower, axis=1)).std(ddof=1) / np.sqrt(len(Z))
    assert abs(good - cf) < 5 * se
    assert abs(bad - cf) > 30 * se
