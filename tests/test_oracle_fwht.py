"""Pins of the oracle's blockwise Hadamard smoother (Sec. 3.2.2, Sec. 3.3).

Checked against the closed form of the Sylvester matrix
H[i][j] = (-1)^popcount(i & j), exact rational arithmetic, float64 dense
products, and the properties the paper states (H symmetric, orthogonal,
its own inverse, spreading an outlier over the block).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def sylvester(n: int) -> np.ndarray:
    i = np.arange(n)
    pc = np.vectorize(lambda v: bin(int(v)).count("1"))(i[:, None] & i[None, :])
    return np.where(pc % 2 == 0, 1, -1).astype(np.int64)


BLOCKS = [2, 4, 8, 16, 32, 64, 128, 256, 512, 1024]


@pytest.mark.parametrize("n", BLOCKS)
def test_scale_is_nearest_float_to_inverse_sqrt(n):
    c = oracle.hadamard_scale(n)
    # (c^2 n - 1) must be smaller in magnitude than for either float neighbour
    def err(v):
        return abs(Fraction(float(v)) ** 2 * n - 1)
    up = np.nextafter(c, np.float32(1), dtype=np.float32)
    dn = np.nextafter(c, np.float32(0), dtype=np.float32)
    assert err(c) <= err(up) and err(c) <= err(dn)
    if n in (4, 16, 64, 256, 1024):
        assert Fraction(float(c)) ** 2 * n == 1


@pytest.mark.parametrize("n", [2, 4, 8, 16, 32, 64, 128])
def test_unit_vectors_give_scaled_sylvester_columns(n):
    H = sylvester(n)
    assert np.array_equal(H, H.T)
    assert np.array_equal(H @ H.T, n * np.eye(n, dtype=np.int64))
    c = oracle.hadamard_scale(n)
    T = np.stack([oracle.fwht(np.eye(n, dtype=np.float32)[j], n) for j in range(n)], axis=1)
    assert np.array_equal(T, (H * c).astype(np.float32))       # +-c exactly
    assert np.array_equal(T, T.T)                                # H = H^T


@pytest.mark.parametrize("n", BLOCKS)
def test_matches_dense_float64_product(n):
    r = np.random.default_rng(n)
    x = r.standard_normal(4 * n).astype(np.float32)
    y = oracle.fwht(x, n)
    H = sylvester(n).astype(np.float64) / np.sqrt(n)
    want = (x.astype(np.float64).reshape(-1, n) @ H.T).ravel()
    k = np.log2(n)
    assert np.max(np.abs(y - want)) <= (k + 2) * 2.0 ** -23 * np.max(np.abs(x)) * np.sqrt(n)
    assert np.linalg.norm(y - want) <= 1e-6 * np.linalg.norm(want)


@pytest.mark.parametrize("n", [4, 16, 64, 256, 1024])
def test_integer_inputs_are_exact_for_powers_of_four(n):
    r = np.random.default_rng(n + 1)
    xi = r.integers(-1000, 1000, 8 * n)
    y = oracle.fwht(xi.astype(np.float32), n)
    want = (xi.reshape(-1, n) @ sylvester(n).T).ravel()          # integer arithmetic
    s = int(round(np.sqrt(n)))
    assert np.array_equal(y.astype(np.float64) * s, want.astype(np.float64))


@pytest.mark.parametrize("n", BLOCKS)
def test_involution_and_parseval(n):
    r = np.random.default_rng(3 * n)
    x = r.standard_normal(16 * n).astype(np.float32)
    y = oracle.fwht(x, n)
    z = oracle.fwht(y, n)
    tol = 4 * (np.log2(n) + 1) * 2.0 ** -24 * np.sqrt(n)
    assert np.max(np.abs(z - x)) <= tol * np.max(np.abs(x))
    bx = x.reshape(-1, n).astype(np.float64)
    by = y.reshape(-1, n).astype(np.float64)
    assert np.allclose(np.linalg.norm(by, axis=1), np.linalg.norm(bx, axis=1), rtol=1e-6)


@pytest.mark.parametrize("n", [32, 64, 256])
def test_outlier_is_spread_over_the_block(n):
    """Sec. 3.2.2: the transform spreads an outlier over the whole block."""
    x = np.zeros(n, np.float32)
    x[5] = 1000.0
    y = oracle.fwht(x, n)
    mag = np.float32(1000.0) * oracle.hadamard_scale(n)
    assert np.all(np.abs(y) == mag)
    # peak-to-RMS of a gradient-like block with one channel outlier drops
    r = np.random.default_rng(n)
    g = (r.standard_normal(n) * 1e-4).astype(np.float32)
    g[7] = 5e-2
    h = oracle.fwht(g, n)
    par = lambda v: np.max(np.abs(v)) / np.sqrt(np.mean(v.astype(np.float64) ** 2))
    assert par(h) < 0.5 * par(g)


def test_blocks_are_independent_and_contiguous():
    r = np.random.default_rng(11)
    x = r.standard_normal(1024).astype(np.float32)
    y = oracle.fwht(x, 128)
    for b in range(8):
        assert np.array_equal(y[b * 128:(b + 1) * 128], oracle.fwht(x[b * 128:(b + 1) * 128], 128))


def test_hadamard_call_equals_fwht_and_rejects_bad_block():
    x = np.random.default_rng(12).standard_normal(512).astype(np.float32)
    assert np.array_equal(oracle.hadamard(x, 64), oracle.fwht(x, 64))
    with pytest.raises(oracle.OracleError):
        oracle.fwht(x, 48)
    with pytest.raises(oracle.OracleError):
        oracle.fwht(x[:100], 64)
