"""Pins of the oracle's quantizers, packing and bfloat16 narrowing.

These check the oracle against things other than itself: exact rational
arithmetic (brute-force nearest lattice level on 64-element groups), the
error bound any round-to-nearest quantizer must meet, extreme elements,
degenerate groups, exact symmetries, and torch's own float->bfloat16
conversion.  A dropped absolute value, a wrong qmax, a flipped sign or a
truncating round fails at least one of them.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _inputs(seed):
    r = np.random.default_rng(seed)
    yield "normal", r.standard_normal(64).astype(np.float32)
    yield "tiny", (r.standard_normal(64) * 1e-6).astype(np.float32)
    yield "outlier", np.where(np.arange(64) == 17, 80.0, r.standard_normal(64)).astype(np.float32)
    yield "negative", -np.abs(r.standard_normal(64)).astype(np.float32)
    yield "uniform", r.uniform(-3, 5, 64).astype(np.float32)
    yield "heavy", (r.standard_t(3, 64) * 1e-3).astype(np.float32)


def _near_half(num: Fraction, tol: Fraction) -> bool:
    frac = num - (num.numerator // num.denominator)
    return abs(frac - Fraction(1, 2)) <= tol


@pytest.mark.parametrize("bits", [8, 4, 2])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_sym_codes_are_nearest_lattice_level(bits, seed):
    """Sec. 2.2: x_int = round(x / s * (2^(k-1) - 1)), s = max|x| per group."""
    qmax = 2 ** (bits - 1) - 1
    for name, x in _inputs(seed):
        for group in (64, 32):
            q, scale, _ = oracle.quant_sym(x, group, bits)
            for g in range(64 // group):
                xs = x[g * group:(g + 1) * group]
                a = max(Fraction(float(abs(v))) for v in xs)
                # the stored scale is s / qmax rounded to float32
                assert scale[g] == np.float32(float(a / qmax)), (name, g)
                for i, v in enumerate(xs):
                    exact = Fraction(float(v)) * qmax / a          # x / s * qmax, exactly
                    if _near_half(exact, Fraction(1, 1 << 14)):
                        continue                                    # rounding-order tie zone
                    want = round(exact)                             # nearest integer
                    want = max(-qmax, min(qmax, want))
                    assert q[g * group + i] == want, (name, bits, g, i, float(exact))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_asym4_codes_are_nearest_level_in_min_max_range(seed):
    for name, x in _inputs(seed):
        q, scale, minv, _ = oracle.quant_asym4(x, 32)
        for g in range(2):
            xs = x[g * 32:(g + 1) * 32]
            mn = Fraction(float(xs.min()))
            mx = Fraction(float(xs.max()))
            assert minv[g] == xs.min()
            assert scale[g] == np.float32(float(np.float32(float(mx - mn)) / 15))
            for i, v in enumerate(xs):
                exact = (Fraction(float(v)) - mn) * 15 / (mx - mn)
                if _near_half(exact, Fraction(1, 1 << 14)):
                    continue
                assert q[g * 32 + i] == round(exact), (name, g, i, float(exact))
            assert q[g * 32 + int(np.argmin(xs))] == 0
            assert q[g * 32 + int(np.argmax(xs))] == 15


@pytest.mark.parametrize("bits", [8, 4])
def test_sym_round_trip_error_bound(bits):
    r = np.random.default_rng(5)
    x = (r.standard_normal(1 << 14) * np.exp(r.uniform(-8, 8, 1 << 14))).astype(np.float32)
    q, s, _ = oracle.quant_sym(x, 128, bits)
    xh = oracle.dequant_sym(q, s, 128)
    bound = np.repeat(s, 128).astype(np.float64) / 2 * (1 + 2.0 ** -12) + np.spacing(np.abs(x)).astype(np.float64)
    assert np.all(np.abs(xh.astype(np.float64) - x) <= bound)


def test_asym4_round_trip_error_bound():
    r = np.random.default_rng(6)
    x = (r.standard_normal(1 << 14) * 1e-3).astype(np.float32)
    q, s, m, _ = oracle.quant_asym4(x, 128)
    xh = oracle.dequant_asym4(q, s, m, 128)
    bound = np.repeat(s, 128).astype(np.float64) / 2 * (1 + 2.0 ** -12) + 2 * np.spacing(np.abs(x)).astype(np.float64) \
        + np.spacing(np.abs(np.repeat(m, 128))).astype(np.float64)
    assert np.all(np.abs(xh.astype(np.float64) - x) <= bound)


@pytest.mark.parametrize("bits", [8, 4])
def test_sym_extreme_element_gets_qmax(bits):
    qmax = 2 ** (bits - 1) - 1
    r = np.random.default_rng(7)
    x = r.standard_normal(4096).astype(np.float32)
    q, _, _ = oracle.quant_sym(x, 64, bits)
    for g in range(64):
        xs = x[g * 64:(g + 1) * 64]
        j = int(np.argmax(np.abs(xs)))
        assert q[g * 64 + j] == (qmax if xs[j] > 0 else -qmax)


def test_degenerate_groups():
    x = np.zeros(256, np.float32)
    x[64:128] = 0.3
    x[128:192] = -7.25
    q, s, _ = oracle.quant_sym(x, 64, 8)
    assert s[0] == 0 and np.all(q[:64] == 0)                       # zero group: scale 0, codes 0
    xh = oracle.dequant_sym(q, s, 64)
    assert np.all(xh[:64] == 0)
    # a constant group of a symmetric quantizer comes back within one ulp
    assert np.all(np.abs(xh[64:192] - x[64:192]) <= np.spacing(np.abs(x[64:192])))
    qa, sa, ma, _ = oracle.quant_asym4(x, 64)
    xa = oracle.dequant_asym4(qa, sa, ma, 64)
    assert np.array_equal(xa, x)                                    # asymmetric: exact
    assert np.all(sa == 0)


def test_tiny_group_below_float_range_is_zeroed():
    # qmax / s overflows for denormal s: the group is treated as zero
    x = np.full(32, np.float32(1e-45), np.float32)
    q, s, _ = oracle.quant_sym(x, 32, 8)
    assert s[0] == 0 and np.all(q == 0)


@pytest.mark.parametrize("e", [-20, -3, 5, 30])
def test_power_of_two_scaling_invariance(e):
    r = np.random.default_rng(8)
    x = r.standard_normal(1024).astype(np.float32)
    y = (x * np.float32(2.0 ** e)).astype(np.float32)
    for bits in (8, 4):
        qx, sx, _ = oracle.quant_sym(x, 128, bits)
        qy, sy, _ = oracle.quant_sym(y, 128, bits)
        assert np.array_equal(qx, qy)
        assert np.array_equal(sy, (sx * np.float32(2.0 ** e)).astype(np.float32))
    qx, sx, mx, _ = oracle.quant_asym4(x, 128)
    qy, sy, my, _ = oracle.quant_asym4(y, 128)
    assert np.array_equal(qx, qy)
    assert np.array_equal(sy, (sx * np.float32(2.0 ** e)).astype(np.float32))


def test_sym_is_odd():
    r = np.random.default_rng(9)
    x = r.standard_normal(2048).astype(np.float32)
    for bits in (8, 4):
        q1, s1, _ = oracle.quant_sym(x, 128, bits)
        q2, s2, _ = oracle.quant_sym(-x, 128, bits)
        assert np.array_equal(q1, -q2) and np.array_equal(s1, s2)


def test_pack4_layout_and_round_trip():
    # even element in the low nibble, two's-complement nibbles for signed codes
    assert oracle.pack4(np.array([1, 2], np.int8)).tolist() == [0x21]
    assert oracle.pack4(np.array([-1, 7], np.int8)).tolist() == [0x7F]
    assert oracle.pack4(np.array([-7, 0], np.int8)).tolist() == [0x09]
    allb = np.arange(256, dtype=np.uint8)
    for signed in (True, False):
        codes = oracle.unpack4(allb, 512, signed)
        assert np.array_equal(oracle.pack4(codes), allb)
        if signed:
            assert codes.min() == -8 and codes.max() == 7
        else:
            assert codes.min() == 0 and codes.max() == 15


def test_bf16_rne_matches_torch():
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(10)
    vals = [r.standard_normal(3000).astype(np.float32),
            (r.standard_normal(1000) * 1e-40).astype(np.float32),       # denormals
            np.array([1.00390625, 1.01171875, -1.00390625, 3.3961e38, 3.3895e38,
                      -3.39e38, 0.0, -0.0, 1e-45], np.float32)]
    # exact ties: low 16 bits == 0x8000
    ties = (r.integers(0, 2 ** 31, 2000, dtype=np.uint32) & 0x7F7F0000 | 0x8000).view(np.float32)
    vals.append(ties[np.isfinite(ties)])
    x = np.concatenate(vals)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.bf16_rne(x)
    assert np.array_equal(got, want)
    assert np.array_equal(oracle.bf16_to_f32(got),
                          torch.from_numpy(want.view(np.int16)).view(torch.bfloat16).float().numpy())
