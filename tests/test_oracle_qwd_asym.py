"""Pins of the oracle's asymmetric (min-max) qWD codec: Alg. 2's weight
difference quantized to 16 levels over [min, max] of each group (Sec. 3.1),
with float32 or bfloat16 model weights (the mixed-precision setting of
Sec. 5.1).

Each check is fixed by something other than the oracle:
  - a worked example small enough to do by hand, whose fused decode differs
    from a rounded product followed by a rounded sum;
  - exact rational arithmetic: the difference is one correctly rounded
    float32 subtraction of the exactly widened weights, every code is the
    nearest of the 16 levels of that difference, the headers are the float
    minimum and the once-rounded (max - min) / 15;
  - the decode's value is the single rounding of the exact code * scale + min,
    the update is one rounded float32 add, and the bfloat16 narrowing is the
    nearest bfloat16 by exact distance, ties to the even pattern (ties are
    built on purpose, of both parities and signs);
  - lattice-exact differences reconstruct the new weights bit for bit.
A truncating narrowing, a decode as product-then-sum, a dropped widening, a
reversed difference, a wrong range divisor or a wrong minimum fails at least
one of them.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


# ----------------------------------------------------------------------------
# exact-arithmetic helpers (written from the IEEE definitions, not the oracle)
# ----------------------------------------------------------------------------

def _bf16_trunc(x):
    return (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _widen(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def _q(x) -> Fraction:
    return Fraction(float(x))


def _round_f32(f: Fraction) -> np.float32:
    """The float32 nearest to the rational f, ties to an even significand.

    float64 may round f once before float32 rounds again, so the two float32
    neighbours of that first guess are compared by exact distance."""
    c = np.float32(float(f))
    cands = {c, np.nextafter(c, np.float32(np.inf)), np.nextafter(c, np.float32(-np.inf))}
    cands = [v for v in cands if np.isfinite(v)]
    best = min(abs(_q(v) - f) for v in cands)
    near = [v for v in cands if abs(_q(v) - f) == best]
    if len(near) == 1:
        return near[0]
    even = [v for v in near if int(np.array(v, np.float32).view(np.uint32)) & 1 == 0]
    assert len(even) == 1
    return even[0]


def _bf16_nearest(f: Fraction) -> int:
    """The bfloat16 bit pattern nearest to the finite rational f (by exact
    distance, over all finite bfloat16 values of f's sign and the overflow
    threshold), ties to an even last bit."""
    sign = 0x8000 if f < 0 else 0
    a = abs(f)
    # bracket |f| between consecutive non-negative bfloat16 patterns
    lo = int(np.float32(float(a)).view(np.uint32) >> 16) if float(a) < 3.4e38 else 0x7F7F
    while lo > 0 and _q(_widen(np.uint16(lo))) > a:
        lo -= 1
    while lo < 0x7F7F and _q(_widen(np.uint16(lo + 1))) <= a:
        lo += 1
    hi = lo + 1
    vlo = _q(_widen(np.uint16(lo)))
    vhi = _q(_widen(np.uint16(hi))) if hi < 0x7F80 else Fraction(2) ** 128
    dlo, dhi = a - vlo, vhi - a
    pick = lo if dlo < dhi else hi if dhi < dlo else (lo if lo % 2 == 0 else hi)
    return sign | pick


def _levels(d, mn, mx):
    """Nearest of the 16 levels of each exact difference of a group, on the
    exact range [mn, mx], with the near-tie set: values within 2^-14 of a half
    level, where the four float32 roundings of the op order (range, inverse,
    shifted value, product; < 2^-19 of a level in all) may decide."""
    out, ties = [], []
    for v in d:
        exact = (v - mn) * 15 / (mx - mn)
        fl = exact.numerator // exact.denominator
        frac = exact - fl
        ties.append(abs(frac - Fraction(1, 2)) <= Fraction(1, 1 << 14))
        out.append(max(0, min(15, fl + (1 if frac > Fraction(1, 2) else 0))))
    return out, ties


def _is_bf16_midpoint(s: Fraction) -> bool:
    """True when s lies exactly halfway between two consecutive bfloat16
    values of its binade: |s| = (m + 1/2) * 2^(E-7), 2^E <= |s| < 2^(E+1)."""
    a = abs(s)
    if a == 0:
        return False
    E = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** E > a:
        E -= 1
    while Fraction(2) ** (E + 1) <= a:
        E += 1
    t = a * Fraction(2) ** (8 - E)
    return t.denominator == 1 and t.numerator % 2 == 1


def _draw(seed, n, bf16, sigma=1e-3, heavy=False):
    r = np.random.default_rng(seed)
    base = (r.standard_normal(n) * 0.02).astype(np.float32)
    prev = _bf16_trunc(base) if bf16 else base
    wide = _widen(prev) if bf16 else prev
    if heavy:
        diff = (r.standard_t(3, n) * (sigma / np.sqrt(3))).astype(np.float32)
    else:
        diff = (r.standard_normal(n) * sigma).astype(np.float32)
    new = (wide + diff).astype(np.float32)
    return prev, wide, new


# ----------------------------------------------------------------------------
# encode
# ----------------------------------------------------------------------------

def test_worked_example_by_hand():
    """prev = 1, new = (0.5, 1.25, 1, 0.75): d = (-0.5, 0.25, 0, -0.25),
    min = -0.5, max - min = 0.75, inv = 15 / 0.75 = 20, scale = fl(0.05) =
    13421773 * 2^-28; the codes are (0, 15, 10, 5).  Decoding into zero float32
    weights: fmaf(10, scale, -0.5) = 10 * 13421773 * 2^-28 - 2^27 * 2^-28 =
    2^-27 exactly, while a rounded product fl(10 * scale) = 0.5 would give 0."""
    for prev in (np.ones(4, np.float32), _bf16_trunc(np.ones(4, np.float32))):
        new = np.array([0.5, 1.25, 1.0, 0.75], np.float32)
        codes, scale, minv, _ = oracle.qwd_encode(new, prev, 4)
        assert minv.tolist() == [-0.5]
        assert scale.tolist() == [float(np.float32(13421773 * 2.0 ** -28))]
        assert codes.tolist() == [0x00 | (0xF << 4), 0x0A | (0x5 << 4)]
    got = oracle.qwd_decode(codes, scale, minv, np.zeros(4, np.float32), 4)
    assert got.tolist() == [-0.5, 0.25, 2.0 ** -27, -0.25]
    # the same message on bfloat16 ones: 1 + 2^-27 rounds to 1 in float32
    got16 = oracle.qwd_decode(codes, scale, minv, _bf16_trunc(np.ones(4, np.float32)), 4)
    assert _widen(got16).tolist() == [0.5, 1.25, 1.0, 0.75]


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("seed,heavy", [(0, False), (1, True), (2, False)])
def test_codes_and_headers_from_the_exact_difference(bf16, seed, heavy):
    n, group = 512, 64
    prev, wide, new = _draw(seed, n, bf16, sigma=5e-4 if heavy else 1e-3, heavy=heavy)
    codes, scale, minv, _ = oracle.qwd_encode(new, prev, group)
    q = oracle.unpack4(codes, n, signed=False)
    for g in range(n // group):
        sl = slice(g * group, (g + 1) * group)
        # d = fl(w_new - widen(w_prev)): one correctly rounded float32 subtraction
        # of the exact bfloat16 value (its bit pattern shifted into a float32)
        d = [_q(_round_f32(_q(a) - _q(b))) for a, b in zip(new[sl], wide[sl])]
        mn, mx = min(d), max(d)
        assert minv[g] == np.float32(float(mn))
        R = _round_f32(mx - mn)
        assert scale[g] == _round_f32(_q(R) / 15), g
        want, ties = _levels(d, mn, mx)
        for i in range(group):
            if not ties[i]:
                assert q[g * group + i] == want[i], (g, i)
        # the group's extremes take the end levels
        assert q[g * group + d.index(mn)] == 0 and q[g * group + d.index(mx)] == 15


def test_codes_span_the_range_under_a_constant_shift():
    """Adding a constant c (exact on a power-of-two lattice) to every new weight
    shifts min and max by c and leaves the range, the scale and every code
    unchanged; exact when all quantities are multiples of a fine lattice."""
    r = np.random.default_rng(9)
    n, group = 1024, 128
    prev = (r.integers(-2 ** 12, 2 ** 12, n) * 2.0 ** -14).astype(np.float32)
    d = (r.integers(-2 ** 9, 2 ** 9, n) * 2.0 ** -20).astype(np.float32)
    new = (prev + d).astype(np.float32)
    c1, s1, m1, _ = oracle.qwd_encode(new, prev, group)
    shift = np.float32(2.0 ** -16)
    c2, s2, m2, _ = oracle.qwd_encode((new + shift).astype(np.float32), prev, group)
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)
    assert np.array_equal(m2, (m1 + shift).astype(np.float32))


def test_swapping_new_and_previous_mirrors_codes():
    """d -> -d maps min to -max, so on exact lattices code q becomes 15 - q
    (no element sits on a half level: all distances are integer levels)."""
    r = np.random.default_rng(10)
    n, group = 1024, 64
    a = (r.integers(-2 ** 10, 2 ** 10, n) * 2.0 ** -12).astype(np.float32)
    k = r.integers(0, 16, n)
    k[::group] = 0
    k[1::group] = 15
    b = (a + (k - 5) * 2.0 ** -14).astype(np.float32)
    c1, s1, _, _ = oracle.qwd_encode(b, a, group)
    c2, s2, _, _ = oracle.qwd_encode(a, b, group)
    q1, q2 = oracle.unpack4(c1, n, signed=False), oracle.unpack4(c2, n, signed=False)
    assert np.array_equal(s1, s2)
    assert np.array_equal(q1.astype(np.int16), 15 - q2.astype(np.int16))
    assert np.array_equal(q1, k.astype(np.int8))


# ----------------------------------------------------------------------------
# decode
# ----------------------------------------------------------------------------

def _decode_exact(codes, scale, minv, prev, group, bf16):
    """Decode by the definitions: single rounding of q*scale + min, one rounded
    float32 add of the exactly widened weight, nearest-even bfloat16."""
    n = prev.size
    q = oracle.unpack4(codes, n, signed=False)
    out = []
    for i in range(n):
        v = _round_f32(int(q[i]) * _q(scale[i // group]) + _q(minv[i // group]))
        w = _q(_widen(prev[i:i + 1])[0]) if bf16 else _q(prev[i])
        s = _round_f32(w + _q(v))
        out.append(_bf16_nearest(_q(s)) if bf16 else s)
    return np.array(out, np.uint16 if bf16 else np.float32)


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("seed", [3, 4])
def test_decode_is_fused_value_then_sum_then_nearest_even(bf16, seed):
    n, group = 512, 64
    prev, _, new = _draw(seed, n, bf16)
    codes, scale, minv, _ = oracle.qwd_encode(new, prev, group)
    got = oracle.qwd_decode(codes, scale, minv, prev, group)
    want = _decode_exact(codes, scale, minv, prev, group, bf16)
    assert np.array_equal(got.view(np.uint8), want.view(np.uint8))


def test_decode_value_is_one_rounding_into_zero_weights():
    """With zero float32 weights the decoded weight is the dequantized value
    itself: fmaf(q, scale, min) rounded once.  Random full-precision headers
    make the rounded product differ from the exact one for most codes."""
    r = np.random.default_rng(11)
    n, group = 2048, 32
    codes = r.integers(0, 256, n // 2).astype(np.uint8)
    scale = (r.random(n // group) * 1e-3 + 1e-5).astype(np.float32)
    minv = (-(r.random(n // group)) * 8e-3).astype(np.float32)
    got = oracle.qwd_decode(codes, scale, minv, np.zeros(n, np.float32), group)
    want = _decode_exact(codes, scale, minv, np.zeros(n, np.float32), group, False)
    assert np.array_equal(got, want)
    # the pin is sharp: the two-rounding decode differs on a visible share
    q = oracle.unpack4(codes, n, signed=False).astype(np.float32)
    two = (q * np.repeat(scale, group)).astype(np.float32) + np.repeat(minv, group)
    assert np.mean(two.astype(np.float32) != want) > 0.05


def _tie_case(seed, n=512):
    """bfloat16 weights w and messages whose decoded sums land exactly half a
    bfloat16 step from w (or one and a half), both parities and signs."""
    r = np.random.default_rng(seed)
    group = 32
    e = np.repeat(r.integers(-8, 2, n // group), group)    # one exponent per group
    mant = r.integers(128, 256, n)                         # 8 significant bits
    sgn = np.where(r.random(n) < 0.5, -1.0, 1.0)
    w = (sgn * mant * np.ldexp(1.0, e - 7)).astype(np.float32)
    prev = _bf16_trunc(w)
    assert np.array_equal(_widen(prev), w)
    ulp = np.ldexp(1.0, e[::group] - 7)                    # bfloat16 step of the group's binade
    scale = (ulp / 2).astype(np.float32)                   # one code = half a step
    minv = (-ulp * 2).astype(np.float32)                   # code 4 -> 0, code 5 -> +half, 3 -> -half
    codes_u = r.choice([3, 5, 7, 1], size=n)               # half-odd steps: -1/2, 1/2, 3/2, -3/2
    return prev, oracle.pack4(codes_u.astype(np.int8)), scale, minv, group


@pytest.mark.parametrize("seed", [12, 13])
def test_bf16_narrowing_ties_go_to_even(seed):
    prev, codes, scale, minv, group = _tie_case(seed)
    got = oracle.qwd_decode(codes, scale, minv, prev, group)
    want = _decode_exact(codes, scale, minv, prev, group, True)
    assert np.array_equal(got, want)
    # the case is what it claims: many float32 sums are exact bfloat16 midpoints
    n = prev.size
    q = oracle.unpack4(codes, n, signed=False)
    sums = [_q(_widen(prev[i:i + 1])[0]) + int(q[i]) * _q(scale[i // group]) + _q(minv[i // group])
            for i in range(n)]
    assert sum(_is_bf16_midpoint(s) for s in sums) > n // 2
    # ties to even go up and down
    w0, w1 = _widen(prev).astype(np.float64), _widen(got).astype(np.float64)
    assert np.any(w1 > w0) and np.any(w1 < w0)


def test_decode_narrowing_is_not_truncation():
    """Sums three quarters of a step above a bfloat16 value round up to the
    next one; truncating the low half of the float32 would keep the old value.
    Weights 1, -1, 3, -3 plus 3 * 2^-9 = 0.75 * 2^-7 (a bfloat16 step at 1) or
    6 * 2^-9 = 0.75 * 2^-6 (a step at 3): 1 + 2^-7 and 3 + 2^-6; below 1 the
    step halves, so -1 + 0.75 * 2^-7 is the tie -(1 - 1.5 * 2^-8), which goes
    to the even -(1 - 2^-7); -3 + 0.75 * 2^-6 is nearest to -3 + 2^-6."""
    prev = _bf16_trunc(np.array([1.0, -1.0, 3.0, -3.0], np.float32))
    scale = np.array([np.float32(2.0 ** -9)], np.float32)
    minv = np.array([0.0], np.float32)
    codes = oracle.pack4(np.array([3, 3, 6, 6], np.int8))
    got = _widen(oracle.qwd_decode(codes, scale, minv, prev, 4))
    assert got.tolist() == [1.0 + 2.0 ** -7, -1.0 + 2.0 ** -7, 3.0 + 2.0 ** -6, -3.0 + 2.0 ** -6]


# ----------------------------------------------------------------------------
# round trips
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("bf16", [False, True])
def test_lattice_difference_reconstructs_exactly(bf16):
    """d = m*2^-6 + k*2^-6 with k = 0 and k = 15 in every group: the range is
    15*2^-6, scale = 2^-6 and inv = 2^6 are exact, the codes are k, and the
    new weights (at most 8 significant bits) are bfloat16 values."""
    r = np.random.default_rng(14)
    n, group = 1024, 64
    prev = (r.integers(-100, 101, n) * 2.0 ** -6).astype(np.float32)
    m = np.repeat(r.integers(-20, 1, n // group), group)
    k = r.integers(0, 16, n)
    k[::group] = 0
    k[1::group] = 15
    new = (prev + (m + k) * 2.0 ** -6).astype(np.float32)
    p = _bf16_trunc(prev) if bf16 else prev
    assert np.array_equal(_widen(p) if bf16 else p, prev)
    codes, scale, minv, _ = oracle.qwd_encode(new, p, group)
    assert np.all(scale == np.float32(2.0 ** -6))
    assert np.array_equal(minv, (m[::group] * 2.0 ** -6).astype(np.float32))
    assert np.array_equal(oracle.unpack4(codes, n, signed=False), k.astype(np.int8))
    got = oracle.qwd_decode(codes, scale, minv, p, group)
    assert np.array_equal(_widen(got) if bf16 else got, new)


@pytest.mark.parametrize("bf16", [False, True])
def test_no_change_leaves_weights_bit_identical(bf16):
    prev, wide, _ = _draw(15, 512, bf16)
    codes, scale, minv, _ = oracle.qwd_encode(wide.copy(), prev, 128)
    assert not codes.any() and not scale.any() and not minv.any()
    got = oracle.qwd_decode(codes, scale, minv, prev, 128)
    assert np.array_equal(np.ascontiguousarray(got).view(np.uint8), np.ascontiguousarray(prev).view(np.uint8))


@pytest.mark.parametrize("bf16", [False, True])
def test_decode_is_within_half_a_step_of_the_new_weights(bf16):
    n, group = 4096, 128
    prev, _, new = _draw(16, n, bf16, sigma=5e-4, heavy=True)
    codes, scale, minv, _ = oracle.qwd_encode(new, prev, group)
    got = oracle.qwd_decode(codes, scale, minv, prev, group)
    got = _widen(got) if bf16 else got
    step = np.repeat(scale.astype(np.float64), group)
    slack = 4 * np.spacing(np.abs(new)).astype(np.float64)
    if bf16:
        slack += np.abs(new).astype(np.float64) * 2.0 ** -8        # half a bfloat16 step, rounded up
    err = np.abs(got.astype(np.float64) - new.astype(np.float64))
    assert np.all(err <= step / 2 * (1 + 2 ** -10) + slack)
