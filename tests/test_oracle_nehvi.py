"""Pins for the oracle's noisy acquisition (qNEHVI, q = 1).

Each check reaches the same quantity by another route: the joint posterior
factored by the library Cholesky on the union of points, the noise-free
interpolation form of the conditional, exact hypervolumes of each sample's
front, and the noise-to-zero limit in which the noisy form reduces to the
plain EHVI.
"""
import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle as O
from oracle import noisy as onehvi
from pins import matern_bessel, hv_exact, front_bruteforce


def _kernel(U, V, ls, s):
    """Matern-5/2 through the Bessel form and a library distance."""
    return s * matern_bessel(cdist(U / ls, V / ls), 2.5)


def _problem(n=12, d=3, m=2, M=5, S=8, eta=1e-2, seed=0):
    r = np.random.default_rng(seed)
    X = r.random((n, d))
    Y = r.standard_normal((n, m))
    ls = r.uniform(0.3, 0.8, size=(m, d))
    s = r.uniform(0.5, 1.5, size=m)
    etas = np.full(m, eta)
    cand = r.random((M, d))
    ZX = r.standard_normal((S, n, m))
    Zs = r.standard_normal((S, m))
    return X, Y, ls, s, etas, cand, ZX, Zs


def test_joint_samples_equal_cholesky_of_the_joint_posterior():
    X, Y, ls, s, eta, cand, ZX, Zs = _problem()
    model = O.fit(X, Y, ls, s, eta)
    F, Ls = O.insample_samples(model, ZX)
    ys = O.candidate_samples(model, cand, ZX, Zs, Ls)
    n = X.shape[0]
    for k in range(2):
        K = _kernel(X, X, ls[k], s[k]) + eta[k] * np.eye(n)
        for c in range(cand.shape[0]):
            U = np.vstack([X, cand[c:c + 1]])
            KU = _kernel(U, U, ls[k], s[k])
            KUX = _kernel(U, X, ls[k], s[k])
            joint = KU - KUX @ np.linalg.solve(K, KUX.T)
            Lj = np.linalg.cholesky(joint)
            for smp in range(ZX.shape[0]):
                z = np.concatenate([ZX[smp, :, k], [Zs[smp, k]]])
                mean = KUX @ np.linalg.solve(K, Y[:, k])
                f = mean + Lj @ z
                np.testing.assert_allclose(F[smp, :, k], f[:n], rtol=1e-9, atol=1e-11)
                assert ys[c, smp, k] == pytest.approx(f[n], rel=1e-8, abs=1e-10)


def test_conditional_equals_noise_free_interpolation():
    # given the latent values at X, y adds nothing: E[f* | f_X] = k*^T K_XX^{-1} f_X
    # and Var[f* | f_X] = s - k*^T K_XX^{-1} k* (the noise-free GP)
    X, Y, ls, s, eta, cand, ZX, Zs = _problem(n=20, M=7, S=6, eta=5e-3, seed=3)
    model = O.fit(X, Y, ls, s, eta)
    F, Ls = O.insample_samples(model, ZX)
    ys = O.candidate_samples(model, cand, ZX, Zs, Ls)
    for k in range(2):
        Kxx = _kernel(X, X, ls[k], s[k])
        Ks = _kernel(cand, X, ls[k], s[k])
        W = np.linalg.solve(Kxx, Ks.T)                      # [n, M]
        tau = np.sqrt(np.maximum(s[k] - np.sum(Ks.T * W, axis=0), 0.0))
        for smp in range(ZX.shape[0]):
            want = W.T @ F[smp, :, k] + tau * Zs[smp, k]
            np.testing.assert_allclose(ys[:, smp, k], want, rtol=1e-7, atol=1e-9)


def test_insample_moments_by_an_independent_route():
    # mu_X = y - eta alpha and Sigma_XX = eta (I - eta K^{-1}) for K = K_XX + eta I
    X, Y, ls, s, eta, *_ = _problem(n=15, eta=2e-2, seed=5)
    model = O.fit(X, Y, ls, s, eta)
    mu, cov = O.insample_posterior(model)
    for k in range(2):
        K = _kernel(X, X, ls[k], s[k]) + eta[k] * np.eye(15)
        Kinv = np.linalg.inv(K)
        np.testing.assert_allclose(mu[:, k], Y[:, k] - eta[k] * (Kinv @ Y[:, k]), rtol=1e-9, atol=1e-11)
        np.testing.assert_allclose(cov[k], eta[k] * (np.eye(15) - eta[k] * Kinv), rtol=1e-8, atol=1e-12)


@pytest.mark.parametrize("lower", [None, "q"])
def test_sample_hvi_equals_exact_hypervolume_difference(lower):
    X, Y, ls, s, eta, cand, ZX, Zs = _problem(n=25, M=6, S=10, eta=5e-2, seed=9)
    model = O.fit(X, Y, ls, s, eta)
    ref = Y.min(axis=0) - 0.1
    low = None if lower is None else np.quantile(Y, 0.3, axis=0)
    got = O.nehvi(model, cand, ref, ZX, Zs, lower=low)["ehvi"]
    F, Ls = O.insample_samples(model, ZX)
    ys = O.candidate_samples(model, cand, ZX, Zs, Ls)
    want = np.zeros(cand.shape[0])
    for smp in range(ZX.shape[0]):
        Fs = F[smp]
        if low is not None:
            Fs = Fs[np.all(Fs >= low, axis=1)]
        front = Fs[front_bruteforce(Fs, ref)]
        base = hv_exact(front, ref)
        for c in range(cand.shape[0]):
            y = ys[c, smp]
            if low is not None and not np.all(y >= low):
                continue
            want[c] += hv_exact(np.vstack([front, y]), ref) - base
    want /= ZX.shape[0]
    np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-12)


def test_small_noise_limit_is_the_plain_ehvi():
    # as eta -> 0 the in-sample samples collapse onto Y and the conditional
    # onto the ordinary posterior: qNEHVI -> EHVI with the same z*
    r = np.random.default_rng(11)
    n, d, M, S = 30, 4, 40, 64
    X = r.random((n, d))
    Y = r.standard_normal((n, 2))
    ls = np.full((2, d), 0.4)
    s = np.ones(2)
    cand = r.random((M, d))
    ZX = r.standard_normal((S, n, 2))
    Zs = r.standard_normal((S, 2))
    ref = Y.min(axis=0) - 0.1
    model = O.fit(X, Y, ls, s, np.full(2, 1e-9))
    got = O.nehvi(model, cand, ref, ZX, Zs)["ehvi"]
    plain = O.score(model, cand[:, None, :], ref, Zs[:, None, :])["ehvi"]
    np.testing.assert_allclose(got, plain, rtol=2e-3, atol=1e-6)
    # and a larger noise moves it measurably (the limit is not trivially met)
    model2 = O.fit(X, Y, ls, s, np.full(2, 0.05))
    got2 = O.nehvi(model2, cand, ref, ZX, Zs)["ehvi"]
    plain2 = O.score(model2, cand[:, None, :], ref, Zs[:, None, :])["ehvi"]
    assert np.max(np.abs(got2 - plain2)) > 1e-3


def test_infeasible_everywhere_gives_zero_and_empty_fronts_give_boxes_from_ref():
    X, Y, ls, s, eta, cand, ZX, Zs = _problem(n=10, M=4, S=5, seed=13)
    model = O.fit(X, Y, ls, s, eta)
    ref = Y.min(axis=0) - 0.1
    high = np.full(2, 50.0)
    assert np.all(O.nehvi(model, cand, ref, ZX, Zs, lower=high)["ehvi"] == 0.0)
    # a reference point above every in-sample value: every front is empty,
    # so each sample's HVI is prod_k (y_k - r_k)_+
    ref_hi = np.full(2, 4.0)
    F, Ls = O.insample_samples(model, ZX)
    assert np.all(F < 4.0)
    ys = O.candidate_samples(model, cand, ZX, Zs, Ls)
    want = np.mean(np.prod(np.maximum(ys - ref_hi, 0.0), axis=-1), axis=1)
    got = O.nehvi(model, cand, ref_hi, ZX, Zs)["ehvi"]
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=0)


def test_planted_transposed_factor_in_the_conditional_is_caught(monkeypatch):
    X, Y, ls, s, eta, cand, ZX, Zs = _problem(n=20, M=7, S=6, eta=5e-3, seed=3)
    model = O.fit(X, Y, ls, s, eta)
    F, Ls = O.insample_samples(model, ZX)
    good = O.candidate_samples(model, cand, ZX, Zs, Ls)
    real = onehvi.solve_triangular
    monkeypatch.setattr(onehvi, "solve_triangular",
                        lambda L, b, lower: real(L.T, b, lower=not lower))
    bad = onehvi.candidate_samples(model, cand, ZX, Zs, Ls)
    k = 0
    Kxx = _kernel(X, X, ls[k], s[k])
    Ks = _kernel(cand, X, ls[k], s[k])
    W = np.linalg.solve(Kxx, Ks.T)
    tau = np.sqrt(np.maximum(s[k] - np.sum(Ks.T * W, axis=0), 0.0))
    want = W.T @ F[0, :, k] + tau * Zs[0, k]
    np.testing.assert_allclose(good[:, 0, k], want, rtol=1e-7, atol=1e-9)
    assert np.max(np.abs(bad[:, 0, k] - want)) > 1e-4


def _problem3(n=14, d=3, M=4, q=2, S=6, eta=2e-2, seed=21):
    r = np.random.default_rng(seed)
    X = r.random((n, d))
    Y = r.standard_normal((n, 3))
    ls = r.uniform(0.3, 0.8, size=(3, d))
    s = r.uniform(0.5, 1.5, size=3)
    cand = r.random((M, q, d))
    ZX = r.standard_normal((S, n, 3))
    Zs = r.standard_normal((S, q, 3))
    return X, Y, ls, s, np.full(3, eta), cand, ZX, Zs


def test_batch_samples_equal_cholesky_of_the_joint_posterior():
    X, Y, ls, s, eta, cand, ZX, Zs = _problem3()
    model = O.fit(X, Y, ls, s, eta)
    F, Ls = O.insample_samples(model, ZX)
    ys = O.batch_samples(model, cand, ZX, Zs, Ls)          # [M, S, q, m]
    n, q = X.shape[0], cand.shape[1]
    for k in range(3):
        K = _kernel(X, X, ls[k], s[k]) + eta[k] * np.eye(n)
        for c in range(cand.shape[0]):
            U = np.vstack([X, cand[c]])
            KU = _kernel(U, U, ls[k], s[k])
            KUX = _kernel(U, X, ls[k], s[k])
            Lj = np.linalg.cholesky(KU - KUX @ np.linalg.solve(K, KUX.T))
            mean = KUX @ np.linalg.solve(K, Y[:, k])
            for smp in range(ZX.shape[0]):
                f = mean + Lj @ np.concatenate([ZX[smp, :, k], Zs[smp, :, k]])
                np.testing.assert_allclose(F[smp, :, k], f[:n], rtol=1e-9, atol=1e-11)
                np.testing.assert_allclose(ys[c, smp, :, k], f[n:], rtol=1e-8, atol=1e-10)


@pytest.mark.parametrize("lower", [None, "q"])
def test_batch_hvi_equals_exact_hypervolume_difference(lower):
    X, Y, ls, s, eta, cand, ZX, Zs = _problem3(n=20, M=5, S=5, eta=5e-2, seed=23)
    model = O.fit(X, Y, ls, s, eta)
    ref = Y.min(axis=0) - 0.1
    low = None if lower is None else np.quantile(Y, 0.3, axis=0)
    got = O.nehvi(model, cand, ref, ZX, Zs, lower=low)["ehvi"]
    F, Ls = O.insample_samples(model, ZX)
    ys = O.batch_samples(model, cand, ZX, Zs, Ls)
    want = np.zeros(cand.shape[0])
    for smp in range(ZX.shape[0]):
        Fs = F[smp]
        if low is not None:
            Fs = Fs[np.all(Fs >= low, axis=1)]
        front = Fs[front_bruteforce(Fs, ref)]
        base = hv_exact(front, ref)
        for c in range(cand.shape[0]):
            mem = ys[c, smp]
            if low is not None:
                mem = mem[np.all(mem >= low, axis=1)]
            want[c] += hv_exact(np.vstack([front, mem]), ref) - base
    want /= ZX.shape[0]
    np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-12)


def test_batch_small_noise_limit_is_the_plain_qehvi():
    r = np.random.default_rng(31)
    n, d, M, S, q = 25, 3, 12, 48, 2
    X = r.random((n, d))
    Y = r.standard_normal((n, 3))
    ls = np.full((3, d), 0.45)
    s = np.ones(3)
    cand = r.random((M, q, d))
    ZX = r.standard_normal((S, n, 3))
    Zs = r.standard_normal((S, q, 3))
    ref = Y.min(axis=0) - 0.1
    model = O.fit(X, Y, ls, s, np.full(3, 1e-9))
    got = O.nehvi(model, cand, ref, ZX, Zs)["ehvi"]
    plain = O.score(model, cand, ref, Zs)["ehvi"]
    np.testing.assert_allclose(got, plain, rtol=2e-3, atol=1e-6)
