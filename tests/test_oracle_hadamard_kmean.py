"""Pins for the oracle's rotation and key-mean removal (CPU only)."""

import numpy as np
import pytest
import scipy.linalg

from oracle import hadamard, kmean


@pytest.mark.parametrize("d", [2, 8, 64, 128, 256])
def test_sylvester_orthogonal(d):
    H = hadamard.sylvester(d)
    assert np.array_equal(H @ H.T, d * np.eye(d, dtype=np.int64))
    assert np.array_equal(H, H.T)
    assert np.array_equal(H, scipy.linalg.hadamard(d))


@pytest.mark.parametrize("d", [8, 128])
def test_fwht_matches_matrix(d):
    rng = np.random.default_rng(d)
    xi = rng.integers(-50, 50, size=(7, d))
    assert np.array_equal(hadamard.fwht(xi), xi @ scipy.linalg.hadamard(d).T)
    # twice = d * identity, exactly for small integers
    assert np.array_equal(hadamard.fwht(hadamard.fwht(xi)), d * xi)
    xr = rng.normal(size=(5, d))
    assert np.max(np.abs(hadamard.fwht(xr) - xr @ scipy.linalg.hadamard(d).T)) < 1e-12


def test_fwht_rejects_non_power_of_two():
    with pytest.raises(ValueError):
        hadamard.fwht(np.zeros((2, 12)))


def test_rotation_spreads_outliers():
    # Sec. 4.2 / Fig. 2: a single outlier channel is spread over all channels
    x = np.zeros(128)
    x[5] = 100.0
    y = hadamard.fwht(x)
    assert np.allclose(np.abs(y), 100.0)


def test_window_mean_matches_library():
    rng = np.random.default_rng(3)
    y = rng.normal(size=(2, 3, 128, 16)) * 5 + 1
    mu = kmean.window_mean(y)
    assert np.max(np.abs(mu - y.mean(axis=-2))) < 1e-13


def test_mean_quantization():
    rng = np.random.default_rng(4)
    mu = rng.normal(size=(10, 128)) * 3
    q, s = kmean.quantize_mean(mu)
    assert q.dtype == np.int8 and s.dtype == np.float16
    s64 = s.astype(np.float64)
    assert np.all(np.abs(q.astype(int)) <= 127)
    # the largest channel maps to +-127 and every error is within half a step
    assert np.all(np.abs(q).max(axis=1) >= 126)
    err = np.abs(kmean.dequantize_mean(q, s) - mu)
    assert np.all(err <= 0.5 * s64[:, None] * (1 + 1e-12) + 1e-300)
    # scale is max|mu| / 127 to fp16 precision
    assert np.all(np.abs(s64 - np.abs(mu).max(axis=1) / 127) <= np.abs(mu).max(axis=1) / 127 * 2 ** -11)


def test_mean_quantization_zero():
    q, s = kmean.quantize_mean(np.zeros((2, 8)))
    assert np.all(q == 0) and np.all(s == 0)
