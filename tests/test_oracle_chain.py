"""Pins of the oracle's two-level gradient path (Alg. 4, Sec. 3.2-3.3).

* Lattice-exact case: peer gradients are built so that every quantization
  on the path is lossless and every float operation exact.  The path then
  is an exact reduce-scatter, so its output must equal the plain sum of
  all P*Q peer gradients over this GPU's shard, computed here in integer
  arithmetic -- independent of the oracle's own code.
* Sec. 3.3 identity: the simplified path (one transform before the 8-bit
  quantization, one after the last reduction) agrees with the naive one
  (transform around every quantize and dequantize) up to rounding.
* Special cases and exact symmetries.
"""
import numpy as np
import pytest

import oracle

from tests._chain import build_lattice_exact_peers, oracle_chain


@pytest.mark.parametrize("block", [0, 4, 16, 64, 256])
@pytest.mark.parametrize("P,Q", [(4, 4), (8, 2), (2, 8)])
def test_lattice_exact_chain_is_exact_reduce_scatter(block, P, Q):
    group = 128
    grads, want = build_lattice_exact_peers(P, Q, group=group, block=block, m_out=512, seed=P * 10 + Q)
    out = oracle_chain(grads, P, Q, group=group, block=block)
    assert out.dtype == np.float32
    assert np.array_equal(out.astype(np.float64), want), np.max(np.abs(out - want))


def _naive_chain(grads, P, Q, group, block):
    """Alg. 4 with every transform kept: T before each quantize, T after each dequantize."""
    M = grads[0][0].size
    T = (lambda v: oracle.fwht(v, block)) if block else (lambda v: v.copy())
    level2 = []
    for a in range(Q):
        deq = []
        for b in range(P):
            q8, s8, _ = oracle.quant_sym(T(grads[a][b]), group, 8)
            deq.append(T(oracle.dequant_sym(q8, s8, group)))          # inverse after dequantize
        red = oracle.reduce_f32(deq)                                     # back in the plain domain
        q4, s4, _ = oracle.quant_sym(T(red), group, 4)                   # forward before re-quantize
        level2.append((q4, s4))
    m = M // Q
    parts = [T(oracle.dequant_sym(q4[:m], s4[:m // group], group)) for (q4, s4) in level2]
    return oracle.reduce_f32(parts)


@pytest.mark.parametrize("block", [64, 256])
def test_simplified_equals_naive_up_to_rounding(block):
    """Sec. 3.3: H H = I and sum_i H g_i = H sum_i g_i make the extra transforms redundant."""
    import synth
    P, Q, group, M = 4, 4, 128, 8192
    w = synth.scaled(synth.WORKLOADS["c3"], 1 << 20)
    grads = [[synth.gradient(w, 0, M, seed=1, peer=a * P + b) for b in range(P)] for a in range(Q)]
    simp = oracle_chain(grads, P, Q, group=group, block=block)
    naive = _naive_chain(grads, P, Q, group, block)
    # identical up to rounding: most elements agree to ~1e-6 relative; a
    # 4-bit code that lands on the other side of a rounding boundary moves
    # its element by at most one 4-bit step of its group.
    scale = np.max(np.abs(naive))
    close = np.abs(simp - naive) <= 1e-5 * scale
    assert close.mean() > 0.999
    assert np.linalg.norm(simp - naive) <= 1e-2 * np.linalg.norm(naive)


def test_single_peer_without_transform_is_quantize_dequantize():
    r = np.random.default_rng(3)
    x = (r.standard_normal(4096) * 1e-3).astype(np.float32)
    for bits in (8, 4):
        codes, s, _ = oracle.grad_quant(x, bits, 0, 128)
        out = oracle.dequant_reduce([codes], [s], 4096, bits, 128, 0)["f32"]
        q, s2, _ = oracle.quant_sym(x, 128, bits)
        assert np.array_equal(s, s2)
        assert np.array_equal(out, oracle.dequant_sym(q, s2, 128))


@pytest.mark.parametrize("e", [-6, 4])
def test_chain_commutes_with_power_of_two_scaling(e):
    import synth
    P, Q, M = 4, 2, 4096
    w = synth.scaled(synth.WORKLOADS["c1"], 1 << 20)
    grads = [[synth.gradient(w, 0, M, seed=2, peer=a * P + b) for b in range(P)] for a in range(Q)]
    k = np.float32(2.0 ** e)
    scaled = [[(g * k).astype(np.float32) for g in row] for row in grads]
    a = oracle_chain(grads, P, Q, group=128, block=64)
    b = oracle_chain(scaled, P, Q, group=128, block=64)
    assert np.array_equal((a * k).astype(np.float32), b)


def test_out_scale_applies_after_the_inverse_transform():
    r = np.random.default_rng(4)
    x = (r.standard_normal(2048) * 1e-2).astype(np.float32)
    codes, s, _ = oracle.grad_quant(x, 4, 0, 128)
    plain = oracle.dequant_reduce([codes, codes], [s, s], 2048, 4, 128, 0, 256, 1.0)["f32"]
    avg = oracle.dequant_reduce([codes, codes], [s, s], 2048, 4, 128, 0, 256, 0.5)["f32"]
    assert np.array_equal(avg, (plain * np.float32(0.5)).astype(np.float32))


def test_reduce_is_in_peer_order_from_plus_zero():
    # fmaf(q, s, acc) from +0 in peer order: (+1e8) + 1 + (-1e8) != 1 in fp32
    q = [np.full(128, 1, np.int8), np.full(128, 1, np.int8), np.full(128, -1, np.int8)]
    s = [np.array([1e8], np.float32), np.array([1.0], np.float32), np.array([1e8], np.float32)]
    out = oracle.dequant_reduce(q, s, 128, 8, 128, 0)["f32"]
    assert np.all(out == 0.0)
    out2 = oracle.dequant_reduce([q[0], q[2], q[1]], [s[0], s[2], s[1]], 128, 8, 128, 0)["f32"]
    assert np.all(out2 == 1.0)
