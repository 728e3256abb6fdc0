"""Pins for the oracle's composite kernel (routing Matern-5/2 + preference-
weighted deployment Matern-3/2 + their product), each term against the
general Bessel-function Matern and the weight against a direct sum."""
import math

import numpy as np
import pytest

import oracle as O
from pins import matern_bessel


def _points(n, d, seed):
    return np.random.default_rng(seed).random((n, d))


def _comp(m, dr, dc, s_route, s_dep, s_int, pref_scale, seed=0):
    r = np.random.default_rng(seed)
    return O.Composite(dr, np.full(m, s_route), np.full(m, s_dep), np.full(m, s_int),
                       pref_scale * r.random((m, dc)))


def _rho(U, V, ls):
    out = np.zeros((len(U), len(V)))
    for i in range(len(U)):
        for j in range(len(V)):
            out[i, j] = math.sqrt(sum(((U[i, t] - V[j, t]) / ls[t]) ** 2 for t in range(len(ls))))
    return out


def test_each_term_matches_the_bessel_matern():
    dr, dc = 3, 5
    U, V = _points(7, dr + dc, 1), _points(6, dr + dc, 2)
    ls = np.random.default_rng(3).uniform(0.2, 0.9, dr + dc)
    r_t = _rho(U[:, :dr], V[:, :dr], ls[:dr])
    r_c = _rho(U[:, dr:], V[:, dr:], ls[dr:])
    only_route = O.composite_cov(U, V, ls, _comp(1, dr, dc, 0.7, 0.0, 0.0, 0.3), 0)
    np.testing.assert_allclose(only_route, 0.7 * matern_bessel(r_t, 2.5), rtol=1e-12, atol=1e-15)
    only_dep = O.composite_cov(U, V, ls, _comp(1, dr, dc, 0.0, 0.4, 0.0, 0.0), 0)
    np.testing.assert_allclose(only_dep, 0.4 * matern_bessel(r_c, 1.5), rtol=1e-12, atol=1e-15)
    only_int = O.composite_cov(U, V, ls, _comp(1, dr, dc, 0.0, 0.0, 0.05, 0.3), 0)
    np.testing.assert_allclose(only_int, 0.05 * matern_bessel(r_t, 2.5) * matern_bessel(r_c, 1.5),
                               rtol=1e-12, atol=1e-17)


def test_preference_weight_scales_the_deployment_term_only():
    dr, dc = 2, 6
    U, V = _points(5, dr + dc, 4), _points(4, dr + dc, 5)
    ls = np.full(dr + dc, 0.5)
    c = _comp(1, dr, dc, 0.0, 1.0, 0.0, 0.4, seed=6)
    flat = _comp(1, dr, dc, 0.0, 1.0, 0.0, 0.0)
    w = lambda X: np.array([math.exp(sum(c.pref[0][j] * X[i, dr + j] for j in range(dc)))
                            for i in range(len(X))])
    got = O.composite_cov(U, V, ls, c, 0)
    np.testing.assert_allclose(got, np.outer(w(U), w(V)) * O.composite_cov(U, V, ls, flat, 0),
                               rtol=1e-13)
    assert np.all(w(U) >= 1.0)       # non-negative slopes on [0,1] features
    # the interaction term ignores the preference
    ci = _comp(1, dr, dc, 0.0, 0.0, 1.0, 0.4, seed=6)
    np.testing.assert_allclose(O.composite_cov(U, V, ls, ci, 0),
                               O.composite_cov(U, V, ls, _comp(1, dr, dc, 0.0, 0.0, 1.0, 0.0), 0),
                               rtol=1e-14)


def test_composite_gram_is_symmetric_psd_with_the_right_diagonal():
    dr, dc = 4, 12
    X = _points(80, dr + dc, 7)
    ls = np.random.default_rng(8).uniform(0.1, 0.6, dr + dc)
    c = _comp(1, dr, dc, 0.7, 0.3, 0.05, 0.08, seed=9)
    K = O.composite_cov(X, X, ls, c, 0)
    np.testing.assert_allclose(K, K.T, rtol=0, atol=1e-15)
    assert np.linalg.eigvalsh(K).min() > -1e-12 * np.abs(K).max()
    w = O.pref_weight(X[:, dr:], c.pref[0])
    np.testing.assert_allclose(np.diag(K), 0.7 + 0.3 * w * w + 0.05, rtol=1e-14)


def test_composite_posterior_limits():
    dr, dc, m = 2, 4, 2
    r = np.random.default_rng(10)
    X = r.random((25, dr + dc))
    Y = r.standard_normal((25, m))
    ls = r.uniform(0.3, 0.7, (m, dr + dc))
    c = _comp(m, dr, dc, 0.6, 0.35, 0.05, 0.1, seed=11)
    eta = np.full(m, 1e-4)
    model = O.fit(X, Y, ls, np.ones(m), eta, composite=c)
    mu, cov = O.posterior(model, X[:, None, :])
    prior = np.stack([model.pair_cov(k, X, X) for k in range(m)], axis=1)      # [n, m]
    var = cov[:, :, 0, 0]
    bound = prior * eta / (prior + eta)
    assert np.all(var >= 0) and np.all(var <= bound * (1 + 1e-6))
    # far field: posterior mean 0, variance the prior k(x, x)
    far = np.concatenate([np.full((3, dr), 50.0), r.random((3, dc))], axis=1)
    far[:, dr:] += 50.0
    mu_f, cov_f = O.posterior(model, far[:, None, :])
    np.testing.assert_allclose(mu_f, 0.0, atol=1e-12)
    for k in range(m):
        w = O.pref_weight(far[:, dr:], c.pref[k])
        np.testing.assert_allclose(cov_f[:, k, 0, 0], 0.6 + 0.35 * w * w + 0.05, rtol=1e-12)
    # mean through the Cholesky route equals a direct dense solve
    for k in range(m):
        K = model.cov(k, X, X) + eta[k] * np.eye(25)
        P = r.random((5, dr + dc))
        want = model.cov(k, P, X) @ np.linalg.solve(K, Y[:, k])
        got, _ = O.posterior(model, P[:, None, :])
        np.testing.assert_allclose(got[:, 0, k], want, rtol=1e-9, atol=1e-12)


def test_plain_model_unchanged_by_the_kernel_switch():
    r = np.random.default_rng(12)
    X, Y = r.random((20, 5)), r.standard_normal((20, 2))
    ls = r.uniform(0.3, 0.7, (2, 5))
    m0 = O.fit(X, Y, ls, np.ones(2), np.full(2, 1e-4))
    K = O.matern52(O.scaled_distance(X, X, ls[1]), 1.0)
    np.testing.assert_array_equal(m0.cov(1, X, X), K)
