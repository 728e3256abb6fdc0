"""Pins for the oracle's log marginal likelihood: the value against SciPy's
multivariate normal density, the gradient against central differences of
that independent value."""
import numpy as np
import pytest
from scipy.stats import multivariate_normal

import oracle as O
from pins import matern_bessel


def _problem(n, d, seed):
    r = np.random.default_rng(seed)
    X = r.random((n, d))
    Y = np.stack([np.sin(3 * X).sum(1), -((X - 0.5) ** 2).sum(1)], axis=1)
    Y = Y + 0.05 * r.standard_normal(Y.shape)
    Y = (Y - Y.mean(0)) / Y.std(0, ddof=1)
    ls = r.uniform(0.2, 0.6, (2, d))
    return X, Y, ls, np.array([1.3, 0.7]), np.array([1e-2, 3e-3])


def _logpdf(X, y, ls, s, eta):
    """log N(y; 0, s M52 + eta I) with the Matern built from the Bessel form."""
    D = (X[:, None, :] - X[None, :, :]) / ls
    rho = np.sqrt((D * D).sum(2))
    K = s * matern_bessel(rho, 2.5) + eta * np.eye(len(X))
    return multivariate_normal(mean=np.zeros(len(X)), cov=K).logpdf(y)


@pytest.mark.parametrize("n,d", [(30, 3), (60, 5)])
def test_value_matches_scipy_density(n, d):
    X, Y, ls, s, eta = _problem(n, d, n + d)
    val, _ = O.mll(X, Y, ls, s, eta)
    for k in range(2):
        assert val[k] == pytest.approx(_logpdf(X, Y[:, k], ls[k], s[k], eta[k]), rel=1e-10)


def test_gradient_matches_central_differences():
    X, Y, ls, s, eta = _problem(25, 3, 7)
    _, g = O.mll(X, Y, ls, s, eta)
    h = 1e-5
    for k in range(2):
        theta = np.concatenate([np.log(ls[k]), [np.log(s[k]), np.log(eta[k])]])

        def f(th):
            return _logpdf(X, Y[:, k], np.exp(th[:3]), np.exp(th[3]), np.exp(th[4]))
        for j in range(5):
            e = np.zeros(5)
            e[j] = h
            fd = (f(theta + e) - f(theta - e)) / (2 * h)
            assert g[k, j] == pytest.approx(fd, rel=1e-5, abs=1e-7), (k, j)


def test_gradient_vanishes_at_the_scale_optimum():
    # for K = s C (no noise), d log p / d log s = (y^T C^{-1} y / s - n) / 2,
    # zero at s* = y^T C^{-1} y / n
    X, Y, ls, _, _ = _problem(40, 2, 3)
    y = Y[:, :1]
    D = (X[:, None, :] - X[None, :, :]) / ls[0]
    C = O.matern52(np.sqrt((D * D).sum(2)), 1.0)
    s_star = float(y[:, 0] @ np.linalg.solve(C + 1e-12 * np.eye(40), y[:, 0]) / 40)
    _, g = O.mll(X, np.repeat(y, 2, axis=1), np.repeat(ls[:1], 2, 0),
                 np.array([s_star, 2 * s_star]), np.array([1e-12, 1e-12]))
    assert abs(g[0, 2]) < 1e-5 * 40
    assert g[1, 2] == pytest.approx(0.5 * (40 / 2 - 40), rel=1e-6)
