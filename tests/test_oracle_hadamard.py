"""Pins of the oracle's Hadamard rotation (Sec. 2.2, Sec. 3.3, App. A): the orthonormal
Sylvester Walsh-Hadamard matrix of order 128, applied per token along head_dim."""
import numpy as np
import scipy.linalg


def test_equals_sylvester_matrix(orc):
    # scipy builds the Sylvester-ordered matrix independently; H is symmetric.
    H = scipy.linalg.hadamard(128).astype(np.float64) / np.sqrt(128.0)
    x = np.random.default_rng(0).standard_normal((6, 128)) * np.exp(np.random.default_rng(1).standard_normal(128))
    np.testing.assert_allclose(orc.hadamard128(x), x @ H, rtol=0, atol=1e-12 * np.abs(x).max())


def test_involution_and_norm(orc):
    x = np.random.default_rng(2).standard_normal((8, 128)) * 3.0
    y = orc.hadamard128(x)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    np.testing.assert_allclose(orc.hadamard128(y), x, rtol=0, atol=1e-12 * np.abs(x).max())


def test_unit_vectors(orc):
    e0 = np.zeros(128)
    e0[0] = 1.0
    np.testing.assert_allclose(orc.hadamard128(e0), np.full(128, 1 / np.sqrt(128)), rtol=1e-15)
    # row j of H for e_j: entries (-1)^popcount(i & j) / sqrt(128)
    for j in (1, 5, 77, 127):
        ej = np.zeros(128)
        ej[j] = 1.0
        expect = np.array([(-1) ** bin(i & j).count("1") for i in range(128)]) / np.sqrt(128)
        np.testing.assert_allclose(orc.hadamard128(ej), expect, rtol=1e-15)
