"""The seeded workload generator: determinism, shapes, recipe invariants."""
import numpy as np
import pytest

import bo_inputs as bi


@pytest.mark.parametrize("cfg", [0, 1, 2, 4])
def test_shapes_dtypes_and_determinism(cfg):
    a = bi.make_config(cfg, seed=1, M=16)
    b = bi.make_config(cfg, seed=1, M=16)
    c = bi.CONFIGS[cfg]
    assert a.X.shape == (c["n"], c["d"]) and a.X.dtype == np.float32
    assert a.Y.shape == (c["n"], c["m"]) and a.Y.dtype == np.float32
    assert a.cand.shape == (16, c["q"], c["d"]) and a.cand.dtype == np.float32
    assert a.Z.shape == (c["S"], c["q"], c["m"]) and a.Z.dtype == np.float32
    assert a.lengthscale.shape == (c["m"], c["d"])
    for f in ("X", "Y", "cand", "Z", "lengthscale", "ref"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    assert np.all((a.X >= 0) & (a.X <= 1)) and np.all((a.cand >= 0) & (a.cand <= 1))


def test_seeds_differ():
    a = bi.make_config(1, seed=0, M=8)
    b = bi.make_config(1, seed=1, M=8)
    assert not np.array_equal(a.X, b.X)


def test_candidate_prefix_property_and_config3_extends_config2():
    small = bi.make_config(2, seed=0, M=100)
    big = bi.make_config(3, seed=0, M=300)
    np.testing.assert_array_equal(big.cand[:100], small.cand)
    for f in ("X", "Y", "Z", "lengthscale", "ref"):
        np.testing.assert_array_equal(getattr(big, f), getattr(small, f))


def test_standardisation_and_reference_point():
    wl = bi.make_config(1, seed=3, M=4)
    Y = wl.Y.astype(np.float64)
    np.testing.assert_allclose(Y.mean(axis=0), 0.0, atol=1e-6)
    np.testing.assert_allclose(Y.std(axis=0, ddof=1), 1.0, atol=1e-6)
    np.testing.assert_array_equal(wl.ref, (Y.min(axis=0) - 0.1).astype(np.float32))


def test_integer_encoded_dimensions():
    wl = bi.make_config(2, seed=0, M=2000)
    k = wl.cand[:, 0, 4:] * 8.0
    np.testing.assert_array_equal(k, np.round(k))
    assert set(np.unique(k).astype(int)) == set(range(9))
    assert len(np.unique(wl.cand[:, 0, :4])) > 7000


def test_config0_hyperparameters():
    wl = bi.make_config(0, seed=0, M=4)
    assert np.all(wl.lengthscale == np.float32(0.3))
    assert np.all(wl.outputscale == 1.0) and np.all(wl.noise == np.float32(1e-4))
