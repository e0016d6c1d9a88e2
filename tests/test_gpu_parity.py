"""GPU parity: every entry point of the HIP library against the oracle, on
seeded inputs that span several wave tiles and end in a ragged tail, plus
edge values, the two-level chain, and run-to-run determinism.

All calls go through the C ABI (ctypes binding); the oracle sees the same
host arrays the device received.
"""
import numpy as np
import pytest

import oracle
import synth
from paper_2410_15526_amd import sdp4
from tests._chain import build_lattice_exact_peers, oracle_chain
from tests._gpu import check_codes, check_f32, check_headers, dev, empty, host, say, torch

pytestmark = pytest.mark.gpu

TILE = 2048          # elements per wavefront tile of the kernels


def size_for(lcm: int, target: int = 11000) -> int:
    """A multiple of lcm near `target`: several tiles and, when lcm < TILE, a ragged tail."""
    return lcm * max(1, -(-target // lcm))


def sync():
    torch().cuda.synchronize()


def grad_input(n, seed=0, peer=None, kind="c3"):
    w = synth.scaled(synth.WORKLOADS[kind], max(n, 1 << 20))
    return synth.gradient(w, 0, n, seed=seed, peer=peer)


# ----------------------------------------------------------------------------
# K1: Hadamard + group quantization
# ----------------------------------------------------------------------------

def run_grad_quant(x: np.ndarray, bits, block, group):
    n = x.size
    xd = dev(x)
    codes = empty(n * bits // 8, "u8")
    scale = empty(n // group, "f32")
    sdp4.sdp4_grad_quant(xd, bits, block, group, codes, scale)
    sync()
    return host(codes), host(scale)


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("block", [0, 2, 4, 16, 32, 64, 128, 256, 512, 1024])
@pytest.mark.parametrize("group", [32, 64, 128, 256, 512, 1024, 2048, 4096])
def test_grad_quant(bits, block, group):
    n = size_for(max(group, block))
    say(f"grad_quant bits={bits} block={block} group={group} n={n}")
    x = grad_input(n, seed=bits * 1000 + block + group)
    codes, scale = run_grad_quant(x, bits, block, group)
    rc, rs, pre = oracle.grad_quant(x, bits, block, group)
    check_headers(scale, rs)
    check_codes(codes, rc, pre, n, bits)


def edge_gradient(n):
    r = np.random.default_rng(7)
    x = (r.standard_normal(n) * 1e-3).astype(np.float32)
    g = 128
    x[0:g] = 0.0                                     # zero group
    x[g:2 * g] = -0.0
    x[2 * g:3 * g] = 0.3                             # constant group
    x[3 * g:4 * g] = (r.standard_normal(g) * 1e-41).astype(np.float32)   # denormals
    x[4 * g:5 * g] = (r.standard_normal(g) * 1e37).astype(np.float32)    # huge
    x[5 * g:6 * g] = 0.0
    x[5 * g + 17] = -2.5                             # single outlier in a zero group
    x[6 * g:7 * g] = np.float32(1e-37)               # tiny normal: qmax / s still finite
    x[7 * g:8 * g] = r.choice(np.float32([-1, 1]), g) * np.float32(2.0 ** -20)
    x[8 * g:9 * g] = np.linspace(-127, 127, g).astype(np.float32)         # exact lattice
    x[9 * g:10 * g] = (np.arange(g) - 63.5).astype(np.float32) / 127      # ties at k + 1/2
    return x


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("block", [0, 128, 256])
def test_grad_quant_edge_values(bits, block):
    n = size_for(256, 4096)
    say(f"grad_quant edge bits={bits} block={block}")
    x = edge_gradient(n)
    codes, scale = run_grad_quant(x, bits, block, 128)
    rc, rs, pre = oracle.grad_quant(x, bits, block, 128)
    check_headers(scale, rs)
    check_codes(codes, rc, pre, n, bits)


# ----------------------------------------------------------------------------
# qWD encode / decode
# ----------------------------------------------------------------------------

def qwd_inputs(n, prev_dtype, seed=0):
    w = synth.scaled(synth.WORKLOADS["c4" if prev_dtype == "bf16" else "c2"], max(n, 1 << 20))
    prev = synth.prev_weights(w, 0, n, seed=seed)
    new = synth.new_weights(w, 0, n, seed=seed)
    return new, prev


def run_qwd(new, prev, group):
    n = new.size
    nd, pd = dev(new), dev(prev)
    codes, scale, minv = empty(n // 2, "u8"), empty(n // group, "f32"), empty(n // group, "f32")
    sdp4.sdp4_qwd_encode(nd, pd, group, codes, scale, minv)
    sdp4.sdp4_qwd_decode(codes, scale, minv, group, pd)
    sync()
    return host(codes), host(scale), host(minv), host(pd)


@pytest.mark.parametrize("prev_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("group", [32, 64, 128, 256, 1024, 2048, 4096])
def test_qwd_encode_decode(prev_dtype, group):
    n = size_for(group)
    say(f"qwd prev={prev_dtype} group={group} n={n}")
    new, prev = qwd_inputs(n, prev_dtype, seed=group)
    codes, scale, minv, upd = run_qwd(new, prev, group)
    rc, rs, rm, pre = oracle.qwd_encode(new, prev, group)
    check_headers(minv, rm, "minv")
    check_headers(scale, rs)
    check_codes(codes, rc, pre, n, 4, signed=False)
    want = oracle.qwd_decode(rc, rs, rm, prev, group)
    if prev_dtype == "bf16":
        assert np.array_equal(upd, want)
    else:
        check_f32(upd, want, "updated weights")


def test_qwd_decode_stage_isolated():
    """Decode of the oracle's own message (not the GPU encoder's)."""
    n, group = size_for(128), 128
    for prev_dtype in ("f32", "bf16"):
        say(f"qwd decode isolated prev={prev_dtype}")
        new, prev = qwd_inputs(n, prev_dtype, seed=3)
        rc, rs, rm, _ = oracle.qwd_encode(new, prev, group)
        pd = dev(prev)
        sdp4.sdp4_qwd_decode(dev(rc), dev(rs), dev(rm), group, pd)
        sync()
        want = oracle.qwd_decode(rc, rs, rm, prev, group)
        got = host(pd)
        if prev_dtype == "bf16":
            assert np.array_equal(got, want)
        else:
            check_f32(got, want)


@pytest.mark.parametrize("prev_dtype", ["f32", "bf16"])
def test_qwd_edge_values(prev_dtype):
    n, g = size_for(128, 4096), 128
    say(f"qwd edge prev={prev_dtype}")
    new, prev = qwd_inputs(n, prev_dtype, seed=9)
    base = synth.bf16_bits_to_f32(prev) if prev_dtype == "bf16" else prev
    new = new.copy()
    new[0:g] = base[0:g]                                  # zero difference
    new[g:2 * g] = base[g:2 * g] + np.float32(1e-3)       # (nearly) constant difference
    new[2 * g:3 * g] = base[2 * g:3 * g] + np.float32(1e30) * np.sign(np.arange(g) - 60)
    new[3 * g:4 * g] = base[3 * g:4 * g] + np.float32(1e-42)
    new[4 * g] = base[4 * g] + np.float32(5.0)            # one large update in a group
    codes, scale, minv, upd = run_qwd(new, prev, g)
    rc, rs, rm, pre = oracle.qwd_encode(new, prev, g)
    check_headers(minv, rm, "minv")
    check_headers(scale, rs)
    check_codes(codes, rc, pre, n, 4, signed=False)
    want = oracle.qwd_decode(rc, rs, rm, prev, g)
    if prev_dtype == "bf16":
        assert np.array_equal(upd, want)
    else:
        check_f32(upd, want)


def test_qwd_decode_bf16_rounding_edges():
    """bf16 model weights: the fp32 sum is narrowed with round-to-nearest-even
    at exact ties (both parities, both signs), on denormals and at the top of
    the range (a tie above the largest bf16 goes to infinity).  Scales are 0,
    so each group adds its minimum to every weight."""
    g, ng = 128, 24
    n = g * ng
    rng = np.random.default_rng(5)
    prev_f = np.empty(n, np.float32)
    mn = np.zeros(ng, np.float32)
    ones_to_two = 1.0 + rng.integers(0, 128, n).astype(np.float32) / 128   # bf16-exact values in [1, 2)
    for k in range(ng):
        sl = slice(k * g, (k + 1) * g)
        kind = k % 8
        if kind == 0:                       # ties at half a bf16 step in [1, 2)
            prev_f[sl], mn[k] = ones_to_two[sl], 2.0 ** -8
        elif kind == 1:                     # negative ties
            prev_f[sl], mn[k] = -ones_to_two[sl], -(2.0 ** -8)
        elif kind == 2:                     # 3/2 of a step: ties above the next value
            prev_f[sl], mn[k] = ones_to_two[sl], 3 * 2.0 ** -8
        elif kind == 3:                     # zero weights plus an fp32 denormal
            prev_f[sl], mn[k] = 0.0, np.float32(1e-40) * (k + 1)
        elif kind == 4:                     # bf16 denormal weights plus a denormal
            prev_f[sl] = (rng.integers(-127, 128, g) * 2.0 ** -133).astype(np.float32)
            mn[k] = np.float32(2.0 ** -134 + 2.0 ** -140)
        elif kind == 5:                     # largest bf16 plus half its step: a tie that overflows
            prev_f[sl], mn[k] = np.float32(3.3895313892515355e38), np.float32(2.0 ** 119)
        elif kind == 6:                     # one fp32 step below that tie: stays finite
            prev_f[sl], mn[k] = np.float32(3.3895313892515355e38), np.float32(2.0 ** 119 - 2.0 ** 104)
        else:                               # ordinary values
            prev_f[sl], mn[k] = (rng.standard_normal(g) * 0.02).astype(np.float32), np.float32(1.7e-3)
    prev = oracle.bf16_rne(prev_f)
    codes = np.zeros(n // 2, np.uint8)
    scale = np.zeros(ng, np.float32)
    say("qwd decode bf16 rounding edges")
    pd = dev(prev)
    sdp4.sdp4_qwd_decode(dev(codes), dev(scale), dev(mn), g, pd)
    sync()
    want = oracle.qwd_decode(codes, scale, mn, prev, g)
    got = host(pd)
    assert np.array_equal(got, want), np.nonzero(got != want)[0][:10]
    assert np.all(want[5 * g:6 * g] == 0x7F80) and np.all(want[6 * g:7 * g] == 0x7F7F)


def test_qw_variant_is_encode_from_zero():
    """qW (direct 4-bit weight quantization, Sec. 5.1 baseline) = qWD against zero weights."""
    n, g = size_for(2048), 2048
    say("qW variant")
    w = synth.prev_weights(synth.scaled(synth.WORKLOADS["c2"], 1 << 20), 0, n)
    zero = np.zeros(n, np.float32)
    codes, scale, minv, upd = run_qwd(w, zero, g)
    rc, rs, rm, pre = oracle.qwd_encode(w, zero, g)
    check_codes(codes, rc, pre, n, 4, signed=False)
    check_headers(scale, rs)
    check_f32(upd, oracle.qwd_decode(rc, rs, rm, zero, g))


def run_qwd_sym(new, prev, group):
    n = new.size
    nd, pd = dev(new), dev(prev)
    codes, scale = empty(n // 2, "u8"), empty(n // group, "f32")
    sdp4.sdp4_qwd_encode_sym(nd, pd, group, codes, scale)
    sdp4.sdp4_qwd_decode_sym(codes, scale, group, pd)
    sync()
    return host(codes), host(scale), host(pd)


def check_qwd_sym(new, prev, group, codes, scale, upd):
    rc, rs, pre = oracle.qwd_encode_sym(new, prev, group)
    check_headers(scale, rs)
    check_codes(codes, rc, pre, new.size, 4)
    want = oracle.qwd_decode_sym(rc, rs, prev, group)
    if prev.dtype == np.uint16:
        assert np.array_equal(upd, want)
    else:
        check_f32(upd, want, "updated weights")


@pytest.mark.parametrize("prev_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("group", [32, 64, 128, 256, 1024, 2048, 4096])
def test_qwd_sym_encode_decode(prev_dtype, group):
    """Symmetric 4-bit qWD (the Sec. 2.2 quantizer on the weight difference)."""
    n = size_for(group)
    say(f"qwd sym prev={prev_dtype} group={group} n={n}")
    new, prev = qwd_inputs(n, prev_dtype, seed=group + 1)
    check_qwd_sym(new, prev, group, *run_qwd_sym(new, prev, group))


def test_qwd_sym_decode_stage_isolated():
    """Decode of the oracle's own symmetric message: bit-exact for both dtypes."""
    n, group = size_for(128), 128
    for prev_dtype in ("f32", "bf16"):
        say(f"qwd sym decode isolated prev={prev_dtype}")
        new, prev = qwd_inputs(n, prev_dtype, seed=5)
        rc, rs, _ = oracle.qwd_encode_sym(new, prev, group)
        pd = dev(prev)
        sdp4.sdp4_qwd_decode_sym(dev(rc), dev(rs), group, pd)
        sync()
        want = oracle.qwd_decode_sym(rc, rs, prev, group)
        assert np.array_equal(host(pd).view(np.uint8), np.ascontiguousarray(want).view(np.uint8))


@pytest.mark.parametrize("prev_dtype", ["f32", "bf16"])
def test_qwd_sym_edge_values(prev_dtype):
    n, g = size_for(128, 4096), 128
    say(f"qwd sym edge prev={prev_dtype}")
    new, prev = qwd_inputs(n, prev_dtype, seed=10)
    base = synth.bf16_bits_to_f32(prev) if prev_dtype == "bf16" else prev
    new = new.copy()
    new[0:g] = base[0:g]                                  # zero difference
    new[g:2 * g] = base[g:2 * g] + np.float32(1e-3)       # (nearly) constant difference
    new[2 * g:3 * g] = base[2 * g:3 * g] + np.float32(1e30) * np.sign(np.arange(g) - 60)
    new[3 * g:4 * g] = base[3 * g:4 * g] + np.float32(1e-42)
    new[4 * g] = base[4 * g] - np.float32(5.0)            # one large negative update in a group
    check_qwd_sym(new, prev, g, *run_qwd_sym(new, prev, g))


# ----------------------------------------------------------------------------
# K2 / K3: dequantize + reduce
# ----------------------------------------------------------------------------

def peer_messages(P, n, bits, block, group, seed=0):
    """Oracle-made messages of P synthetic peers (stage-isolated inputs)."""
    out = []
    for p in range(P):
        x = grad_input(n, seed=seed, peer=p)
        c, s, _ = oracle.grad_quant(x, bits, block, group)
        out.append((c, s))
    return out


@pytest.mark.parametrize("P", [1, 2, 3, 4, 5, 8, 16])
@pytest.mark.parametrize("bits_in,bits_out", [(8, 4), (8, 8), (4, 4), (4, 8)])
@pytest.mark.parametrize("group", [32, 128, 4096])
def test_dequant_reduce_requant(P, bits_in, bits_out, group):
    n = size_for(group)
    say(f"dequant_reduce requant P={P} in={bits_in} out={bits_out} group={group} n={n}")
    msgs = peer_messages(P, n, bits_in, 256 if group >= 256 else 0, group, seed=P)
    cd = [dev(c) for c, _ in msgs]
    sd = [dev(s) for _, s in msgs]
    oc, os_, of = empty(n * bits_out // 8, "u8"), empty(n // group, "f32"), empty(n, "f32")
    sdp4.sdp4_dequant_reduce(cd, sd, n, bits_in, group, bits_out, 0, 1.0, oc, os_, of)
    oc2, os2 = empty(n * bits_out // 8, "u8"), empty(n // group, "f32")
    sdp4.sdp4_dequant_reduce(cd, sd, n, bits_in, group, bits_out, 0, 1.0, oc2, os2, None)
    sync()
    ref = oracle.dequant_reduce([c for c, _ in msgs], [s for _, s in msgs], n, bits_in, group, bits_out)
    check_f32(host(of), ref["f32"], "reduced")
    check_headers(host(os_), ref["scales"])
    check_codes(host(oc), ref["codes"], ref["pre"], n, bits_out)
    assert np.array_equal(host(oc2), host(oc)) and np.array_equal(host(os2), host(os_))


@pytest.mark.parametrize("P", [1, 2, 4, 7, 16])
@pytest.mark.parametrize("bits_in", [4, 8])
@pytest.mark.parametrize("block", [0, 2, 64, 128, 256, 1024])
@pytest.mark.parametrize("out_scale", [1.0, 0.125, 1.0 / 3.0])
def test_dequant_reduce_to_f32(P, bits_in, block, out_scale):
    group = 128
    n = size_for(max(group, block))
    say(f"dequant_reduce f32 P={P} in={bits_in} block={block} out_scale={out_scale} n={n}")
    msgs = peer_messages(P, n, bits_in, 0, group, seed=10 + P)
    of = empty(n, "f32")
    sdp4.sdp4_dequant_reduce([dev(c) for c, _ in msgs], [dev(s) for _, s in msgs], n, bits_in, group, 0,
                             block, out_scale, None, None, of)
    sync()
    ref = oracle.dequant_reduce([c for c, _ in msgs], [s for _, s in msgs], n, bits_in, group, 0, block,
                                out_scale)
    check_f32(host(of), ref["f32"])


def test_dequant_reduce_wide_group_to_f32():
    n, group = 3 * 4096, 4096
    say("dequant_reduce f32 group 4096")
    msgs = peer_messages(3, n, 4, 0, group, seed=77)
    of = empty(n, "f32")
    sdp4.sdp4_dequant_reduce([dev(c) for c, _ in msgs], [dev(s) for _, s in msgs], n, 4, group, 0, 1024,
                             0.5, None, None, of)
    sync()
    ref = oracle.dequant_reduce([c for c, _ in msgs], [s for _, s in msgs], n, 4, group, 0, 1024, 0.5)
    check_f32(host(of), ref["f32"])


@pytest.mark.parametrize("bits_in", [4, 8])
@pytest.mark.parametrize("block", [64, 256, 512, 1024])
@pytest.mark.parametrize("out_scale", [1.0, -0.5])
def test_dequant_reduce_to_f32_exact_zeros(bits_in, block, out_scale):
    """Exact zeros out of the inverse transform carry the oracle's sign bit.
    Two peers send equal codes for elements 2j and 2j+1 (one group, power-of-two
    scales, so every product is exact): every odd output of a block is then an
    exact zero, and in every third group the second peer negates the first, so
    whole groups reduce to zero."""
    group = 128
    n = size_for(max(group, block), 16384)
    say(f"dequant_reduce f32 exact zeros in={bits_in} block={block} out_scale={out_scale} n={n}")
    rng = np.random.default_rng(block + bits_in)
    qmax = 127 if bits_in == 8 else 7
    q0 = rng.integers(-qmax, qmax + 1, n // 2).repeat(2)
    q1 = rng.integers(-qmax, qmax + 1, n // 2).repeat(2)
    q1 = np.where((np.arange(n) // group) % 3 == 0, -q0, q1)
    sc = (np.float32(2.0) ** rng.integers(-24, -4, n // group)).astype(np.float32)
    if bits_in == 8:
        codes = [q.astype(np.int8).view(np.uint8) for q in (q0, q1)]
    else:
        codes = [oracle.pack4(q.astype(np.int32)) for q in (q0, q1)]
    of = empty(n, "f32")
    sdp4.sdp4_dequant_reduce([dev(c) for c in codes], [dev(sc), dev(sc)], n, bits_in, group, 0, block,
                             out_scale, None, None, of)
    sync()
    ref = oracle.dequant_reduce(codes, [sc, sc], n, bits_in, group, 0, block, out_scale)
    assert np.count_nonzero(ref["f32"] == 0) >= n // 2
    check_f32(host(of), ref["f32"])


# ----------------------------------------------------------------------------
# standalone pieces of the unfused variant
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("block", [2, 8, 32, 64, 128, 256, 512, 1024])
def test_hadamard(block):
    n = size_for(block)
    say(f"hadamard block={block} n={n}")
    x = grad_input(n, seed=block)
    xd = dev(x)
    y = empty(n, "f32")
    sdp4.sdp4_hadamard(xd, y, block)
    sdp4.sdp4_hadamard(xd, xd, block)          # in place
    sync()
    want = oracle.hadamard(x, block)
    check_f32(host(y), want)
    check_f32(host(xd), want, "in place")


@pytest.mark.parametrize("P", [1, 2, 5, 16])
@pytest.mark.parametrize("n", [4096, 4099, 1 << 20])
def test_reduce_f32_and_copy(P, n):
    say(f"reduce_f32 P={P} n={n}")
    r = np.random.default_rng(P)
    xs = [(r.standard_normal(n) * 10.0 ** r.uniform(-3, 3)).astype(np.float32) for _ in range(P)]
    y = empty(n, "f32")
    sdp4.sdp4_reduce_f32([dev(x) for x in xs], y)
    z = empty(n, "f32")
    x0 = dev(xs[0])
    sdp4.sdp4_copy_f32(x0, z)
    sync()
    check_f32(host(y), oracle.reduce_f32(xs))
    assert np.array_equal(host(z), xs[0])


@pytest.mark.parametrize("n", [4, 4099, 1 << 20, (1 << 22) + 7])
def test_read_and_fill_yardsticks(n):
    """The bandwidth yardsticks touch every element: the read stream's XOR
    checksum (bit patterns of x[i] into word i % 4) and the fill's output."""
    say(f"read/fill yardsticks n={n}")
    t = torch()
    r = np.random.default_rng(n)
    x = r.standard_normal(n).astype(np.float32)
    sink = t.zeros(4, dtype=t.int32, device="cuda")
    sdp4.sdp4_read_f32(dev(x), sink)
    y = empty(n, "f32")
    sdp4.sdp4_fill_f32(y, -2.75)
    sync()
    b = x.view(np.uint32)
    want = np.array([np.bitwise_xor.reduce(b[k::4]) if b[k::4].size else 0 for k in range(4)], np.uint32)
    assert np.array_equal(host(sink).view(np.uint32), want)
    assert np.all(host(y) == np.float32(-2.75))


# ----------------------------------------------------------------------------
# the two-level chain, run the way one GPU runs it
# ----------------------------------------------------------------------------

def gpu_chain(grads, P, Q, group, block, out_scale=1.0):
    """K1 per peer, K2 per node (pointer slices as the all-to-all would deliver), K3."""
    M = grads[0][0].size
    m = M // Q
    level2 = []
    for a in range(Q):
        codes, scales = [], []
        for b in range(P):
            c, s = empty(M, "u8"), empty(M // group, "f32")
            sdp4.sdp4_grad_quant(dev(grads[a][b]), 8, block, group, c, s)
            codes.append(c)
            scales.append(s)
        oc, os_ = empty(M // 2, "u8"), empty(M // group, "f32")
        sdp4.sdp4_dequant_reduce(codes, scales, M, 8, group, 4, 0, 1.0, oc, os_)
        level2.append((oc, os_))
    out = empty(m, "f32")
    sdp4.sdp4_dequant_reduce([oc[:m // 2] for oc, _ in level2], [os_[:m // group] for _, os_ in level2], m, 4,
                             group, 0, block, out_scale, None, None, out)
    sync()
    return host(out)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_chain_matches_oracle(name):
    w = synth.WORKLOADS[name]
    P, Q, group, block = w.P, w.Q, w.group, w.hadamard_block
    M = Q * size_for(max(group, block), 4096)
    say(f"chain {name} P={P} Q={Q} block={block} M={M}")
    ws = synth.scaled(w, 1 << 20)
    grads = [[synth.gradient(ws, 0, M, seed=5, peer=a * P + b) for b in range(P)] for a in range(Q)]
    got = gpu_chain(grads, P, Q, group, block, out_scale=1.0 / (P * Q))
    want = oracle_chain(grads, P, Q, group, block, out_scale=1.0 / (P * Q))
    check_f32(got, want)


@pytest.mark.parametrize("block", [0, 16, 64, 256])
def test_chain_lattice_exact_is_reduce_scatter(block):
    P, Q, group = 8, 4, 128
    say(f"lattice chain block={block}")
    grads, want = build_lattice_exact_peers(P, Q, group=group, block=block, m_out=2048, seed=block + 1)
    got = gpu_chain(grads, P, Q, group, block)
    assert np.array_equal(got.astype(np.float64), want)


def test_unfused_chain_matches_oracle():
    """The 'HS w/o fused' variant: standalone transform, plain (de)quantization
    per chunk, float32 reductions, standalone inverse transform."""
    P, Q, group, block = 4, 2, 128, 256
    M = Q * size_for(256, 4096)
    m = M // Q
    say("unfused chain")
    ws = synth.scaled(synth.WORKLOADS["c3"], 1 << 20)
    grads = [[synth.gradient(ws, 0, M, seed=6, peer=a * P + b) for b in range(P)] for a in range(Q)]
    level2_dev, level2_ref = [], []
    for a in range(Q):
        deq_dev, deq_ref = [], []
        for b in range(P):
            xd = dev(grads[a][b])
            hd = empty(M, "f32")
            sdp4.sdp4_hadamard(xd, hd, block)
            c, s = empty(M, "u8"), empty(M // group, "f32")
            sdp4.sdp4_grad_quant(hd, 8, 0, group, c, s)
            f = empty(M, "f32")
            sdp4.sdp4_dequant_reduce([c], [s], M, 8, group, 0, 0, 1.0, None, None, f)
            deq_dev.append(f)
            rc, rs, _ = oracle.grad_quant(oracle.hadamard(grads[a][b], block), 8, 0, group)
            deq_ref.append(oracle.dequant_reduce([rc], [rs], M, 8, group, 0)["f32"])
        red = empty(M, "f32")
        sdp4.sdp4_reduce_f32(deq_dev, red)
        c4, s4 = empty(M // 2, "u8"), empty(M // group, "f32")
        sdp4.sdp4_grad_quant(red, 4, 0, group, c4, s4)
        level2_dev.append((c4, s4))
        rc4, rs4, _ = oracle.grad_quant(oracle.reduce_f32(deq_ref), 4, 0, group)
        level2_ref.append((rc4, rs4))
    parts_dev, parts_ref = [], []
    for (c4, s4), (rc4, rs4) in zip(level2_dev, level2_ref):
        f = empty(m, "f32")
        sdp4.sdp4_dequant_reduce([c4[:m // 2]], [s4[:m // group]], m, 4, group, 0, 0, 1.0, None, None, f)
        parts_dev.append(f)
        parts_ref.append(oracle.dequant_reduce([rc4[:m // 2]], [rs4[:m // group]], m, 4, group, 0)["f32"])
    red = empty(m, "f32")
    sdp4.sdp4_reduce_f32(parts_dev, red)
    out = empty(m, "f32")
    sdp4.sdp4_hadamard(red, out, block)
    sync()
    want = oracle.hadamard(oracle.reduce_f32(parts_ref), block)
    check_f32(host(out), want)


def test_hotpath_unfused_step_matches_fused_and_its_oracle():
    """HotPath.unfused_gradient_step on a scaled GPT-1.3B shard (P = 8, Q = 4,
    block 256): its output is the oracle's unfused composition bit for bit,
    averaging included, and within the float bar of the fused step."""
    from paper_2410_15526_amd.pipeline import HotPath
    w = synth.scaled(synth.WORKLOADS["c3"], 1 << 22)
    n, g, blk, P, Q = w.n, w.group, w.hadamard_block, w.P, w.Q
    M, m, osc = n // P, n // (P * Q), 1.0 / (P * Q)
    say(f"HotPath unfused vs fused n={n} P={P} Q={Q} block={blk}")
    grad = synth.gradient(w, 0, n, 0)
    hp = HotPath(n, g, blk, P, Q, w.qwd_group, w.prev_dtype)
    hp.grad.copy_(torch().from_numpy(grad))
    hp.grad_quant()
    hp.reduce_intra()
    hp.reduce_inter()
    sync()
    fused = host(hp.out).copy()
    hp.out.fill_(-1.0)
    hp.unfused_gradient_step()
    sync()
    unfused = host(hp.out).copy()

    c8, s8, _ = oracle.grad_quant(grad, 8, blk, g)
    k2 = oracle.dequant_reduce([c8[p * M:(p + 1) * M] for p in range(P)],
                               [s8[p * M // g:(p + 1) * M // g] for p in range(P)], M, 8, g, 4)
    c4, s4 = k2["codes"], k2["scales"]
    want_fused = oracle.dequant_reduce([c4[q * m // 2:(q + 1) * m // 2] for q in range(Q)],
                                       [s4[q * m // g:(q + 1) * m // g] for q in range(Q)], m, 4, g, 0, blk,
                                       osc)["f32"]
    hc8, hs8, _ = oracle.grad_quant(oracle.hadamard(grad, blk), 8, 0, g)
    d = [oracle.dequant_reduce([hc8[p * M:(p + 1) * M]], [hs8[p * M // g:(p + 1) * M // g]], M, 8, g, 0)["f32"]
         for p in range(P)]
    uc4, us4, _ = oracle.grad_quant(oracle.reduce_f32(d), 4, 0, g)
    d2 = [oracle.dequant_reduce([uc4[q * m // 2:(q + 1) * m // 2]], [us4[q * m // g:(q + 1) * m // g]], m, 4, g,
                                0, 0, osc)["f32"] for q in range(Q)]
    want_unfused = oracle.hadamard(oracle.reduce_f32(d2), blk)

    check_f32(fused, want_fused, "fused step")
    check_f32(unfused, want_unfused, "unfused step")
    check_f32(unfused, fused, "unfused vs fused", exact=False)


# ----------------------------------------------------------------------------
# determinism, empty inputs, binding errors
# ----------------------------------------------------------------------------

def test_bitwise_repeatable():
    n, group, block = 1 << 21, 128, 256
    say("repeatability")
    x = dev(grad_input(n, seed=3))
    outs = []
    for _ in range(3):
        c, s = empty(n, "u8"), empty(n // group, "f32")
        sdp4.sdp4_grad_quant(x, 8, block, group, c, s)
        oc, os_ = empty(n // 8, "u8"), empty(n // 4 // group, "f32")
        sdp4.sdp4_dequant_reduce([c[i * n // 4:(i + 1) * n // 4] for i in range(4)],
                                 [s[i * n // 4 // group:(i + 1) * n // 4 // group] for i in range(4)],
                                 n // 4, 8, group, 4, 0, 1.0, oc, os_)
        f = empty(n // 16, "f32")
        sdp4.sdp4_dequant_reduce([oc[i * n // 32:(i + 1) * n // 32] for i in range(2)],
                                 [os_[i * n // 16 // group:(i + 1) * n // 16 // group] for i in range(2)],
                                 n // 16, 4, group, 0, block, 0.125, None, None, f)
        sync()
        outs.append((host(c), host(s), host(oc), host(os_), host(f)))
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_empty_inputs_are_noops():
    say("empty inputs")
    z = empty(16, "f32")
    sentinel = z.clone()
    sdp4.sdp4_grad_quant(z, 8, 256, 128, z[:0], z[:0], n=0)
    sdp4.sdp4_hadamard(z, z, 64, n=0)
    sdp4.sdp4_dequant_reduce([z], [z], 0, 8, 128, 0, 0, 1.0, None, None, z)
    sync()
    assert torch().equal(z, sentinel)


def test_binding_reports_status():
    say("binding errors")
    x = empty(4096 + 4, "f32")
    c, s = empty(4096, "u8"), empty(32, "f32")
    with pytest.raises(sdp4.Sdp4Error) as e:
        sdp4.sdp4_grad_quant(x[1:4097], 8, 256, 128, c, s)          # 4-byte offset: misaligned
    assert e.value.status == sdp4.EALIGN
    with pytest.raises(sdp4.Sdp4Error) as e:
        sdp4.sdp4_grad_quant(x[:4096], 8, 256, 96, c, s)
    assert e.value.status == sdp4.EINVAL


# ----------------------------------------------------------------------------
# stochastic rounding (unbiased gradient compression)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("block,group", [(0, 32), (64, 128), (256, 128), (128, 512), (512, 64), (1024, 256), (16, 1024),
                                         (0, 2048), (1024, 4096)])
@pytest.mark.parametrize("seed,offset", [(0, 0), (0xDEADBEEF12345678, 8 * 12345), (7, 1 << 33)])
def test_grad_quant_sr(bits, block, group, seed, offset):
    n = size_for(max(group, block))
    say(f"grad_quant_sr bits={bits} block={block} group={group} seed={seed} offset={offset} n={n}")
    x = grad_input(n, seed=bits + block + group)
    xd = dev(x)
    codes, scale = empty(n * bits // 8, "u8"), empty(n // group, "f32")
    sdp4.sdp4_grad_quant_sr(xd, bits, block, group, seed, offset, codes, scale)
    sync()
    rc, rs, pre = oracle.grad_quant_sr(x, bits, block, group, seed, offset)
    check_headers(host(scale), rs)
    assert np.array_equal(host(codes).view(np.uint8), rc.view(np.uint8))


@pytest.mark.parametrize("P", [1, 3, 8, 16])
@pytest.mark.parametrize("bits_in,bits_out", [(8, 4), (4, 4), (8, 8)])
def test_dequant_reduce_sr(P, bits_in, bits_out):
    group = 128
    n = size_for(group)
    say(f"dequant_reduce_sr P={P} in={bits_in} out={bits_out}")
    msgs = peer_messages(P, n, bits_in, 0, group, seed=40 + P)
    oc, os_, of = empty(n * bits_out // 8, "u8"), empty(n // group, "f32"), empty(n, "f32")
    sdp4.sdp4_dequant_reduce_sr([dev(c) for c, _ in msgs], [dev(s) for _, s in msgs], n, bits_in, group, bits_out,
                                99, 64, oc, os_, of)
    sync()
    ref = oracle.dequant_reduce_sr([c for c, _ in msgs], [s for _, s in msgs], n, bits_in, group, bits_out, 99, 64)
    check_f32(host(of), ref["f32"])
    check_headers(host(os_), ref["scales"])
    assert np.array_equal(host(oc).view(np.uint8), ref["codes"].view(np.uint8))


def test_sr_pieces_equal_one_call_and_seeds_differ():
    n, group, block = 1 << 16, 128, 256
    say("sr pieces")
    x = dev(grad_input(n, seed=9))
    whole = empty(n, "u8")
    s = empty(n // group, "f32")
    sdp4.sdp4_grad_quant_sr(x, 8, block, group, 5, 0, whole, s)
    parts = empty(n, "u8")
    h = n // 2
    sdp4.sdp4_grad_quant_sr(x[:h], 8, block, group, 5, 0, parts[:h], s[:h // group])
    sdp4.sdp4_grad_quant_sr(x[h:], 8, block, group, 5, h, parts[h:], s[h // group:])
    other = empty(n, "u8")
    sdp4.sdp4_grad_quant_sr(x, 8, block, group, 6, 0, other, s)
    sync()
    assert np.array_equal(host(whole), host(parts))
    assert not np.array_equal(host(whole), host(other))
