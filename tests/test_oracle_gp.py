"""Pins for the oracle's GP part: closed forms, library routes, invariants."""
import math

import numpy as np
import pytest

import oracle as O
from oracle import gp as ogp
from pins import matern_bessel

RNG = np.random.default_rng(7)


def _rand_problem(n=40, d=5, m=2, eta=1e-4, seed=0):
    r = np.random.default_rng(seed)
    X = r.random((n, d))
    Y = r.standard_normal((n, m))
    ls = r.uniform(0.2, 0.7, size=(m, d))
    s = r.uniform(0.5, 2.0, size=m)
    return X, Y, ls, s, np.full(m, eta)


# ---- Matern-5/2 -----------------------------------------------------------

def test_matern_equals_bessel_form():
    rho = np.concatenate([np.linspace(0.0, 6.0, 601), [1e-6, 10.0, 20.0]])
    got = O.matern52(rho, 1.0)
    ref = matern_bessel(rho, 2.5)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-15)


def test_matern_special_values():
    assert O.matern52(0.0, 2.5) == pytest.approx(2.5, rel=0, abs=0)
    # rho = 1 through the general Bessel form (independent of the polynomial)
    assert O.matern52(1.0, 3.0) == pytest.approx(3.0 * matern_bessel(np.array([1.0]), 2.5)[0], rel=1e-13)
    rho = np.linspace(0, 8, 400)
    k = O.matern52(rho, 1.0)
    assert np.all(np.diff(k) < 0)
    assert O.matern52(60.0, 1.0) < 1e-50


def test_scaled_distance_ard_and_symmetry():
    r = np.random.default_rng(3)
    U, V = r.random((7, 4)), r.random((5, 4))
    ls = np.array([0.1, 0.5, 2.0, 1.0])
    D = O.scaled_distance(U, V, ls)
    for i in range(7):
        for j in range(5):
            direct = math.sqrt(sum(((U[i, t] - V[j, t]) / ls[t]) ** 2 for t in range(4)))
            assert D[i, j] == pytest.approx(direct, rel=1e-14)
    np.testing.assert_allclose(O.scaled_distance(V, U, ls), D.T, rtol=0, atol=0)


def test_gram_is_psd():
    X, Y, ls, s, eta = _rand_problem(n=60, d=3)
    K = O.matern52(O.scaled_distance(X, X, ls[0]), s[0])
    np.testing.assert_allclose(K, K.T, rtol=0, atol=0)
    assert np.linalg.eigvalsh(K).min() > -1e-10


# ---- fit ---------------------------------------------------------------

def test_cholesky_reconstruction_and_lu_route():
    X, Y, ls, s, eta = _rand_problem()
    mdl = O.fit(X, Y, ls, s, eta)
    for k in range(2):
        K = O.matern52(O.scaled_distance(X, X, ls[k]), s[k]) + eta[k] * np.eye(len(X))
        L = mdl.L[k]
        assert np.allclose(np.triu(L, 1), 0.0)
        assert np.linalg.norm(L @ L.T - K) / np.linalg.norm(K) < 1e-13
        # alpha through LU (numpy.linalg.solve), not through the factor
        np.testing.assert_allclose(mdl.alpha[k], np.linalg.solve(K, Y[:, k]), rtol=1e-8, atol=1e-10)


def test_not_pd_is_reported():
    X, Y, ls, s, eta = _rand_problem(n=6)
    X[1] = X[0]
    with pytest.raises(O.NotPositiveDefinite):
        O.fit(X, Y, ls, s, np.zeros(2))


# ---- posterior ---------------------------------------------------------

def test_posterior_n1_closed_form():
    r = np.random.default_rng(11)
    x1 = r.random((1, 4))
    y1 = np.array([[0.7, -1.3]])
    ls = np.array([[0.3, 0.4, 0.5, 0.6], [0.2, 0.2, 0.9, 0.9]])
    s = np.array([1.7, 0.6])
    eta = np.array([1e-3, 0.2])
    mdl = O.fit(x1, y1, ls, s, eta)
    cand = r.random((9, 1, 4))
    mu, cov = O.posterior(mdl, cand)
    for k in range(2):
        rho = np.sqrt(np.sum(((cand[:, 0, :] - x1[0]) / ls[k]) ** 2, axis=1))
        kk = s[k] * matern_bessel(rho, 2.5)
        np.testing.assert_allclose(mu[:, 0, k], kk * y1[0, k] / (s[k] + eta[k]), rtol=1e-12)
        np.testing.assert_allclose(cov[:, k, 0, 0], s[k] - kk ** 2 / (s[k] + eta[k]), rtol=1e-12)


def test_posterior_matches_dense_inverse_route():
    X, Y, ls, s, eta = _rand_problem(n=30, d=3, eta=1e-2)
    mdl = O.fit(X, Y, ls, s, eta)
    cand = np.random.default_rng(5).random((11, 3, 3))
    mu, cov = O.posterior(mdl, cand)
    for k in range(2):
        K = O.matern52(O.scaled_distance(X, X, ls[k]), s[k]) + eta[k] * np.eye(30)
        Kinv = np.linalg.inv(K)
        for b in range(11):
            P = cand[b]
            Ks = O.matern52(O.scaled_distance(P, X, ls[k]), s[k])
            Kpp = O.matern52(O.scaled_distance(P, P, ls[k]), s[k])
            np.testing.assert_allclose(mu[b, :, k], Ks @ Kinv @ Y[:, k], rtol=1e-8, atol=1e-10)
            np.testing.assert_allclose(cov[b, k], Kpp - Ks @ Kinv @ Ks.T, rtol=1e-8, atol=1e-10)


def test_variance_at_training_inputs_collapses_to_noise_level():
    X, Y, ls, s, eta = _rand_problem(n=50, d=4, eta=1e-4)
    mdl = O.fit(X, Y, ls, s, eta)
    mu, cov = O.posterior(mdl, X[:, None, :])
    for k in range(2):
        v = cov[:, k, 0, 0]
        bound = s[k] * eta[k] / (s[k] + eta[k])
        assert np.all(v >= 0)
        assert np.all(v <= bound * (1 + 1e-6))


def test_isolated_training_point_attains_bound():
    # two far-apart points: each is isolated, so the bound holds with equality
    X = np.array([[0.0, 0.0], [50.0, 50.0]])
    Y = np.array([[1.0], [-1.0]])
    mdl = O.fit(X, Y, np.array([[0.5, 0.5]]), np.array([2.0]), np.array([0.1]))
    _, cov = O.posterior(mdl, X[:, None, :])
    np.testing.assert_allclose(cov[:, 0, 0, 0], 2.0 * 0.1 / 2.1, rtol=1e-12)


def test_far_field_reverts_to_prior():
    X, Y, ls, s, eta = _rand_problem(n=20, d=3)
    mdl = O.fit(X, Y, ls, s, eta)
    far = np.full((3, 1, 3), 1e3)
    mu, cov = O.posterior(mdl, far)
    np.testing.assert_allclose(mu, 0.0, atol=1e-300)
    np.testing.assert_allclose(cov[:, :, 0, 0], np.broadcast_to(s, (3, 2)), rtol=1e-15)


def test_q_batch_consistent_with_single_points():
    X, Y, ls, s, eta = _rand_problem(n=25, d=4)
    mdl = O.fit(X, Y, ls, s, eta)
    cand = np.random.default_rng(9).random((6, 4, 4))
    mu4, cov4 = O.posterior(mdl, cand)
    mu1, cov1 = O.posterior(mdl, cand.reshape(-1, 1, 4))
    np.testing.assert_allclose(mu4.reshape(-1, 2), mu1[:, 0, :], rtol=1e-12, atol=1e-14)
    d4 = np.diagonal(cov4, axis1=-2, axis2=-1)                 # [6, m, 4]
    d1 = cov1[:, :, 0, 0].reshape(6, 4, 2).transpose(0, 2, 1)
    np.testing.assert_allclose(d4, d1, rtol=1e-12, atol=1e-14)
    for b in range(6):
        for k in range(2):
            np.testing.assert_allclose(cov4[b, k], cov4[b, k].T, atol=1e-14)
            assert np.linalg.eigvalsh(cov4[b, k]).min() > -1e-10


# ---- chol_psd ------------------------------------------------------------

def test_chol_psd_reconstructs_pd_matrices():
    r = np.random.default_rng(2)
    A = r.standard_normal((20, 4, 4))
    S = A @ A.transpose(0, 2, 1) + 0.1 * np.eye(4)
    C = O.chol_psd(S, 1.0)
    np.testing.assert_allclose(C @ C.transpose(0, 2, 1), S, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(C, np.linalg.cholesky(S), rtol=1e-10, atol=1e-12)


def test_chol_psd_degenerate_pivot_zeroes_column():
    v = np.array([1.0, 2.0, 0.5, -1.0])
    S = np.outer(v, v)[None]             # rank one: pivots 2..4 are zero
    C = O.chol_psd(S, 1.0)[0]
    np.testing.assert_allclose(C[:, 0], v / 1.0, rtol=1e-14)
    np.testing.assert_allclose(C[:, 1:], 0.0, atol=0)
    np.testing.assert_allclose(C @ C.T, S[0], rtol=1e-14, atol=1e-14)
    Z = np.zeros((1, 4, 4))
    assert np.all(O.chol_psd(Z, 1.0) == 0)


def test_pins_catch_planted_matern_mistake(monkeypatch):
    """A dropped quadratic term in the kernel must break the Bessel pin."""
    bad = lambda rho, s: s * (1 + ogp.SQRT5 * rho) * np.exp(-ogp.SQRT5 * rho)
    rho = np.linspace(0.0, 4.0, 50)
    assert not np.allclose(bad(rho, 1.0), matern_bessel(rho, 2.5), rtol=1e-6)
