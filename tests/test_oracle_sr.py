"""Pins of the oracle's stochastic rounding (the unbiased gradient
compressor the convergence analysis of Sec. 4.2 assumes).

* The generator is Philox4x32-10, checked against its published
  known-answer vectors (tests/golden/philox4x32_10_kat.txt).
* The quantizer rounds each scaled value to one of its two neighbouring
  integers, and is unbiased: averaged over seeds, the dequantized values
  converge to the input (checked against exact rationals and a 6-sigma
  bound).
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

KAT = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def kat_rows():
    for line in open(KAT):
        if line.strip() and not line.startswith("#"):
            w = [int(t, 16) for t in line.split()]
            yield w[0:4], w[4:6], w[6:10]


@pytest.mark.parametrize("row", list(kat_rows()))
def test_philox_known_answers(row):
    ctr, key, want = row
    assert list(oracle.philox4x32_10(ctr, key)) == want


def test_uniform_mapping_and_distribution():
    # element e uses word (e/2)%4 of block e/8: halves of one word are e, e+1
    seed = 0x1234_5678_9ABC_DEF0
    out = oracle.philox4x32_10([3, 0, 0, 0], [seed & 0xFFFFFFFF, seed >> 32])
    for j in range(8):
        w = int(out[j // 2])
        half = (w >> 16) if j % 2 else (w & 0xFFFF)
        assert oracle.sr_uniform(seed, 24 + j) == half / 65536.0
    u = np.array([oracle.sr_uniform(7, e) for e in range(1 << 14)])
    assert u.min() >= 0.0 and u.max() < 1.0
    hist, _ = np.histogram(u, bins=16, range=(0, 1))
    chi2 = np.sum((hist - u.size / 16) ** 2 / (u.size / 16))
    assert chi2 < 45.0          # 15 dof: p ~ 1e-4


@pytest.mark.parametrize("bits", [8, 4])
def test_codes_are_floor_or_ceil(bits):
    qmax = 2 ** (bits - 1) - 1
    r = np.random.default_rng(bits)
    x = r.standard_normal(1024).astype(np.float32)
    q, s, _ = oracle.quant_sym_sr(x, 128, bits, seed=99)
    qd, sd, _ = oracle.quant_sym(x, 128, bits)
    assert np.array_equal(s, sd)                       # same scales as round-to-nearest
    for g in range(8):
        a = max(Fraction(float(abs(v))) for v in x[g * 128:(g + 1) * 128])
        for i in range(128):
            k = g * 128 + i
            exact = Fraction(float(x[k])) * qmax / a
            lo = exact.numerator // exact.denominator
            assert q[k] in (lo, lo + 1) or (abs(exact - round(exact)) < Fraction(1, 1 << 14)), (k, float(exact))
            assert -qmax <= q[k] <= qmax


@pytest.mark.parametrize("bits", [8, 4])
def test_unbiased_over_seeds(bits):
    """E[dequant(Q(x))] = x: the compressor is unbiased (up to 2^-16 of a step)."""
    r = np.random.default_rng(5)
    x = (r.standard_normal(128) * 1e-3).astype(np.float32)
    S = 4096
    acc = np.zeros(128)
    acc2 = np.zeros(128)
    for seed in range(S):
        q, s, _ = oracle.quant_sym_sr(x, 128, bits, seed=seed)
        d = oracle.dequant_sym(q, s, 128).astype(np.float64)
        acc += d
        acc2 += d * d
    mean = acc / S
    std = np.sqrt(np.maximum(acc2 / S - mean ** 2, 0))
    step = float(s[0])
    tol = 6 * np.maximum(std, step * 1e-3) / np.sqrt(S) + step * 2.0 ** -15
    assert np.all(np.abs(mean - x) <= tol)
    # round-to-nearest is biased on the same data
    qd, sd, _ = oracle.quant_sym(x, 128, bits)
    assert np.max(np.abs(oracle.dequant_sym(qd, sd, 128) - x)) > 10 * np.max(tol)


def test_offset_addresses_the_same_stream():
    r = np.random.default_rng(6)
    x = r.standard_normal(4096).astype(np.float32)
    q, s, _ = oracle.quant_sym_sr(x, 128, 8, seed=11)
    q1, _, _ = oracle.quant_sym_sr(x[:2048], 128, 8, seed=11, offset=0)
    q2, _, _ = oracle.quant_sym_sr(x[2048:], 128, 8, seed=11, offset=2048)
    assert np.array_equal(q, np.concatenate([q1, q2]))
    q3, _, _ = oracle.quant_sym_sr(x, 128, 8, seed=12)
    assert not np.array_equal(q, q3)


def test_sr_chain_pieces():
    r = np.random.default_rng(7)
    x = (r.standard_normal(2048) * 1e-2).astype(np.float32)
    c, s, pre = oracle.grad_quant_sr(x, 8, 256, 128, seed=3, offset=64)
    y = oracle.fwht(x, 256)
    q, s2, _ = oracle.quant_sym_sr(y, 128, 8, seed=3, offset=64)
    assert np.array_equal(c, q) and np.array_equal(s, s2)
    c4, s4, _ = oracle.grad_quant_sr(x, 4, 0, 128, seed=3)
    assert np.array_equal(oracle.unpack4(c4, 2048, True), oracle.quant_sym_sr(x, 128, 4, seed=3)[0])
    r2 = oracle.dequant_reduce_sr([c, c], [s, s], 2048, 8, 128, 4, seed=5)
    red = oracle.dequant_reduce([c, c], [s, s], 2048, 8, 128, 4)
    assert np.array_equal(r2["f32"], red["f32"])
    assert np.array_equal(r2["scales"], red["scales"])
    assert np.array_equal(oracle.unpack4(r2["codes"], 2048, True),
                          oracle.quant_sym_sr(red["f32"], 128, 4, seed=5)[0])
    with pytest.raises(oracle.OracleError):
        oracle.grad_quant_sr(x, 8, 0, 128, seed=1, offset=4)   # offset must be a multiple of 8
