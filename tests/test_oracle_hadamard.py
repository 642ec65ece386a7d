"""Pins of the oracle's fixed normalized Hadamard transform (Sec. 3.1, KVarN).

Checked against scipy's Sylvester Hadamard matrix (a library routine): unit
vectors map to its scaled columns bit for bit, integer vectors map to the
exact integer product scaled once, H H^T = n I, and the normalized
transform is an involution.
"""
import numpy as np
import pytest
import scipy.linalg

import oracle


@pytest.mark.parametrize("n", [64, 128, 256])
def test_unit_vectors_map_to_scaled_hadamard_columns(n):
    Hm = scipy.linalg.hadamard(n)
    c = np.float32(1.0 / np.sqrt(n))
    cols = oracle.fwht_f32(np.eye(n, dtype=np.float32))   # row i = transform of e_i
    assert np.array_equal(cols, (Hm.T * c).astype(np.float32))
    # H H^T = n I on the +-1 matrix recovered from the transform
    Hpm = np.rint(cols.astype(np.float64) / np.float64(c)).astype(np.int64)
    assert np.array_equal(Hpm @ Hpm.T, n * np.eye(n, dtype=np.int64))


@pytest.mark.parametrize("n", [64, 128])
def test_integer_vectors_are_exact(n):
    rng = np.random.default_rng(n)
    Hm = scipy.linalg.hadamard(n).astype(np.int64)
    c = np.float32(1.0 / np.sqrt(n))
    for _ in range(20):
        x = rng.integers(-1000, 1000, n)
        y = oracle.fwht_f32(x.astype(np.float32))
        ref = (Hm @ x).astype(np.float32) * c      # sums < 2^24: exact, then one rounding
        assert np.array_equal(y, ref)


def test_involution_and_norm():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((50, 128)).astype(np.float32)
    y = oracle.fwht_f32(x)
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-5)
    assert np.allclose(oracle.fwht_f32(y), x, rtol=1e-5, atol=1e-6)
    ref = x.astype(np.float64) @ scipy.linalg.hadamard(128).T / np.sqrt(128)
    assert np.allclose(y, ref, rtol=1e-5, atol=1e-5)


def test_normalization_constant_is_nearest_binary32():
    y = oracle.fwht_f32(np.eye(128, dtype=np.float32)[0])
    assert y[0] == np.float32(0.08838834764831845)
