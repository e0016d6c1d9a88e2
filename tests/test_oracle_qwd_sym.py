"""Pins of the oracle's symmetric qWD codec: Alg. 2's weight difference
quantized with the paper's own symmetric 4-bit quantizer (Sec. 2.2), the
alternative to the asymmetric min-max codec.

Each check is fixed by something other than the oracle: a worked example
small enough to do by hand, exact rational arithmetic on the difference,
the half-step error bound of a round-to-nearest codec, the exact sign
symmetry d(w_prev, w_new) = -d(w_new, w_prev), and lattice-exact inputs
that must reconstruct the new weights bit for bit.  A reversed difference,
a dropped widening of bfloat16 weights, a wrong qmax, an unsigned nibble or
a fused multiply-add in the decode fails at least one of them.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _bf16(x):
    return (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _widen(b):
    return (b.astype(np.uint32) << 16).view(np.float32)


def test_worked_example_by_hand():
    """prev = 1, d = (0.875, -0.25, 0.3 - rounding, 0): s = 0.875, scale = 1/8,
    inv = 8, codes = (7, -2, 2, 0); decode gives 1.875, 0.75, 1.25, 1."""
    prev = np.ones(4, np.float32)
    new = np.array([1.875, 0.75, 1.3, 1.0], np.float32)
    codes, scale, _ = oracle.qwd_encode_sym(new, prev, 4)
    assert scale.tolist() == [0.125]
    assert codes.tolist() == [0x07 | (0xE << 4), 0x02]        # 7, -2 (nibble 0xE), 2, 0
    got = oracle.qwd_decode_sym(codes, scale, prev, 4)
    assert got.tolist() == [1.875, 0.75, 1.25, 1.0]


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("seed", [0, 1])
def test_codes_are_nearest_level_of_the_exact_difference(bf16, seed):
    r = np.random.default_rng(seed)
    n, group = 256, 64
    base = (r.standard_normal(n) * 0.02).astype(np.float32)
    prev = _bf16(base) if bf16 else base
    wide = _widen(prev) if bf16 else prev
    new = (wide + r.standard_normal(n).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
    codes, scale, _ = oracle.qwd_encode_sym(new, prev, group)
    q = oracle.unpack4(codes, n, signed=True)
    for g in range(n // group):
        sl = slice(g * group, (g + 1) * group)
        # d = fl(w_new - widen(w_prev)): one correctly rounded float32 subtraction
        d = [Fraction(float(np.float32(Fraction(float(a)) - Fraction(float(b)))))
             for a, b in zip(new[sl], wide[sl])]
        s = max(abs(v) for v in d)
        assert scale[g] == np.float32(float(s / 7))
        for i, v in enumerate(d):
            exact = v * 7 / s
            frac = exact - (exact.numerator // exact.denominator)
            if abs(frac - Fraction(1, 2)) <= Fraction(1, 1 << 14):
                continue                                          # rounding-order tie zone
            assert q[g * group + i] == max(-7, min(7, round(exact))), (g, i, float(exact))


def test_swapping_new_and_previous_negates_codes():
    r = np.random.default_rng(3)
    a = (r.standard_normal(1024) * 0.02).astype(np.float32)
    b = (a + r.standard_normal(1024).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
    c1, s1, _ = oracle.qwd_encode_sym(b, a, 128)
    c2, s2, _ = oracle.qwd_encode_sym(a, b, 128)
    assert np.array_equal(s1, s2)
    q1, q2 = oracle.unpack4(c1, 1024, signed=True), oracle.unpack4(c2, 1024, signed=True)
    assert np.array_equal(q1.astype(np.int16), -q2.astype(np.int16))
    assert q1.min() >= -7 and q1.max() <= 7


@pytest.mark.parametrize("bf16", [False, True])
def test_decode_is_within_half_a_step_of_the_new_weights(bf16):
    r = np.random.default_rng(4)
    n, group = 4096, 128
    base = (r.standard_normal(n) * 0.02).astype(np.float32)
    prev = _bf16(base) if bf16 else base
    wide = _widen(prev) if bf16 else prev
    new = (wide + (r.standard_t(3, n) * 5e-4).astype(np.float32)).astype(np.float32)
    codes, scale, _ = oracle.qwd_encode_sym(new, prev, group)
    got = oracle.qwd_decode_sym(codes, scale, prev, group)
    got = _widen(got) if bf16 else got
    step = np.repeat(scale.astype(np.float64), group)
    slack = 4 * np.spacing(np.abs(new)).astype(np.float64)
    if bf16:
        slack += np.abs(new).astype(np.float64) * 2.0 ** -8        # half a bfloat16 ulp, rounded up
    err = np.abs(got.astype(np.float64) - new.astype(np.float64))
    assert np.all(err <= step / 2 * (1 + 2 ** -10) + slack)


@pytest.mark.parametrize("bf16", [False, True])
def test_no_change_leaves_weights_bit_identical(bf16):
    r = np.random.default_rng(5)
    base = (r.standard_normal(512) * 0.02).astype(np.float32)
    prev = _bf16(base) if bf16 else base
    new = _widen(prev) if bf16 else prev.copy()
    codes, scale, _ = oracle.qwd_encode_sym(new, prev, 128)
    assert not codes.any() and not scale.any()
    got = oracle.qwd_decode_sym(codes, scale, prev, 128)
    assert np.array_equal(got.view(np.uint8), np.ascontiguousarray(prev).view(np.uint8))


def test_lattice_difference_reconstructs_exactly():
    """d = k * 2^-12 with max |k| = 7 in every group: max|d| / 7 = 2^-12 is
    exact, the codes are k, and w_prev + d is exact in float32."""
    r = np.random.default_rng(6)
    n, group = 1024, 64
    prev = (r.integers(-2 ** 10, 2 ** 10, n) * 2.0 ** -12).astype(np.float32)
    k = r.integers(-7, 8, n)
    k[::group] = 7
    new = (prev.astype(np.float64) + k * 2.0 ** -12).astype(np.float32)
    codes, scale, _ = oracle.qwd_encode_sym(new, prev, group)
    assert np.all(scale == np.float32(2.0 ** -12))
    assert np.array_equal(oracle.unpack4(codes, n, signed=True), k.astype(np.int8))
    assert np.array_equal(oracle.qwd_decode_sym(codes, scale, prev, group), new)


def test_error_feedback_loop_converges():
    """Symmetric qWD as C_w in Alg. 3 on a least-squares problem."""
    r = np.random.default_rng(7)
    n, group = 512, 128
    A = r.standard_normal((64, n)).astype(np.float32) / 8
    b = A @ r.standard_normal(n).astype(np.float32)
    w, wt = np.zeros(n, np.float32), np.zeros(n, np.float32)
    loss0 = np.linalg.norm(A @ wt - b)
    for _ in range(400):
        w = (w - np.float32(0.05) * (A.T @ (A @ wt - b)).astype(np.float32)).astype(np.float32)
        codes, s, _ = oracle.qwd_encode_sym(w, wt, group)
        wt = oracle.qwd_decode_sym(codes, s, wt, group)
        step = np.repeat(s, group)
        assert np.all(np.abs(w - wt) <= step / 2 * (1 + 2 ** -10) + 4 * np.spacing(np.abs(w)))
    assert np.linalg.norm(A @ wt - b) < 1e-3 * loss0


def _f32_exact(f: Fraction) -> np.float32:
    """float32 nearest to f, for an f that float64 holds exactly (one rounding)."""
    d = float(f)
    assert Fraction(d) == f
    return np.float32(d)


def test_decode_rounds_the_product_then_the_sum():
    """value = fl(code * scale), then w <- fl(w + value): two roundings, checked
    in exact rational arithmetic (a fused multiply-add rounds once)."""
    r = np.random.default_rng(8)
    n, group = 512, 64
    prev = (r.standard_normal(n) * 0.02).astype(np.float32)
    new = (prev + r.standard_normal(n).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
    codes, scale, _ = oracle.qwd_encode_sym(new, prev, group)
    q = oracle.unpack4(codes, n, signed=True)
    got = oracle.qwd_decode_sym(codes, scale, prev, group)
    for i in range(n):
        v = _f32_exact(Fraction(int(q[i])) * Fraction(float(scale[i // group])))
        want = _f32_exact(Fraction(float(prev[i])) + Fraction(float(v)))
        assert got[i] == want, i
