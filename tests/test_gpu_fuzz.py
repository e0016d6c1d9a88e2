"""Randomized parity: hypothesis draws shapes (sizes in whole multiples of
max(group, block), from one segment to dozens of wave tiles), bit widths,
Hadamard blocks, groups, peer counts, offsets and value distributions
(normal, heavy-tailed, one-signed, sparse, constant runs, mixed
magnitudes spanning 1e-30..1e30, exact lattice points) and compares every
entry point with the oracle.  Examples are derandomized so every GPU run
draws the same cases."""
import os

import numpy as np
import pytest

hyp = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, given, settings, strategies as st  # noqa: E402

import oracle  # noqa: E402
from paper_2410_15526_amd import sdp4  # noqa: E402
from tests._gpu import check_codes, check_f32, check_headers, dev, empty, host, torch  # noqa: E402

pytestmark = pytest.mark.gpu

# SDP4_FUZZ_EXAMPLES raises the example count for a deeper one-off run (the
# derandomized sequence is extended, so a failure is reproducible).
SETTINGS = settings(max_examples=int(os.environ.get("SDP4_FUZZ_EXAMPLES", "60")), deadline=None, derandomize=True,
                    database=None, suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
DISTS = ["normal", "heavy", "negative", "sparse", "constant_runs", "mixed_magnitude", "lattice"]


def draw_values(kind, n, seed):
    r = np.random.default_rng(seed)
    if kind == "normal":
        x = r.standard_normal(n) * 1e-3
    elif kind == "heavy":
        x = r.standard_t(1.5, n) * 1e-4
    elif kind == "negative":
        x = -np.abs(r.standard_normal(n))
    elif kind == "sparse":
        x = r.standard_normal(n) * (r.random(n) < 0.05)
    elif kind == "constant_runs":
        x = np.repeat(r.standard_normal(max(1, n // 32)), 32)[:n]
        x = np.pad(x, (0, n - x.size))
    elif kind == "mixed_magnitude":
        x = r.standard_normal(n) * np.repeat(10.0 ** r.uniform(-30, 30, -(-n // 64)), 64)[:n]
    else:
        x = r.integers(-127, 128, n).astype(np.float64) * 2.0 ** r.integers(-20, 20)
    return np.ascontiguousarray(x, np.float32)


def sync():
    torch().cuda.synchronize()


@SETTINGS
@given(bits=st.sampled_from([4, 8]), log_group=st.integers(5, 12), log_block=st.sampled_from([0, 1, 2, 4, 6, 7, 8, 10]),
       segments=st.integers(1, 40), kind=st.sampled_from(DISTS), seed=st.integers(0, 2 ** 31 - 1),
       sr=st.booleans(), offset8=st.integers(0, 1 << 20))
def test_grad_quant_random(bits, log_group, log_block, segments, kind, seed, sr, offset8):
    group, block = 1 << log_group, (1 << log_block) if log_block else 0
    n = max(group, block) * segments
    x = draw_values(kind, n, seed)
    codes, scale = empty(n * bits // 8, "u8"), empty(n // group, "f32")
    if sr:
        sdp4.sdp4_grad_quant_sr(dev(x), bits, block, group, seed, 8 * offset8, codes, scale)
        rc, rs, pre = oracle.grad_quant_sr(x, bits, block, group, seed, 8 * offset8)
    else:
        sdp4.sdp4_grad_quant(dev(x), bits, block, group, codes, scale)
        rc, rs, pre = oracle.grad_quant(x, bits, block, group)
    sync()
    check_headers(host(scale), rs)
    if sr:
        assert np.array_equal(host(codes).view(np.uint8), rc.view(np.uint8))
    else:
        check_codes(host(codes), rc, pre, n, bits)


@SETTINGS
@given(P=st.integers(1, 16), bits_in=st.sampled_from([4, 8]), bits_out=st.sampled_from([0, 4, 8]),
       log_group=st.integers(5, 12), log_block=st.sampled_from([0, 1, 3, 5, 8, 10]), segments=st.integers(1, 24),
       seed=st.integers(0, 2 ** 31 - 1), out_scale=st.sampled_from([1.0, 0.5, 0.1]), want_f32=st.booleans())
def test_dequant_reduce_random(P, bits_in, bits_out, log_group, log_block, segments, seed, out_scale, want_f32):
    group = 1 << log_group
    block = ((1 << log_block) if log_block else 0) if bits_out == 0 else 0
    n = max(group, block) * segments
    msgs = []
    for p in range(P):
        x = draw_values(DISTS[(seed + p) % len(DISTS)], n, seed + p)
        c, s, _ = oracle.grad_quant(x, bits_in, 0, group)
        msgs.append((c, s))
    cs, ss = [dev(c) for c, _ in msgs], [dev(s) for _, s in msgs]
    ref = oracle.dequant_reduce([c for c, _ in msgs], [s for _, s in msgs], n, bits_in, group, bits_out, block,
                                out_scale)
    if bits_out == 0:
        of = empty(n, "f32")
        sdp4.sdp4_dequant_reduce(cs, ss, n, bits_in, group, 0, block, out_scale, None, None, of)
        sync()
        check_f32(host(of), ref["f32"])
        return
    oc, os_ = empty(n * bits_out // 8, "u8"), empty(n // group, "f32")
    of = empty(n, "f32") if want_f32 else None
    sdp4.sdp4_dequant_reduce(cs, ss, n, bits_in, group, bits_out, 0, 1.0, oc, os_, of)
    sync()
    check_headers(host(os_), ref["scales"])
    check_codes(host(oc), ref["codes"], ref["pre"], n, bits_out)
    if want_f32:
        check_f32(host(of), ref["f32"])


@SETTINGS
@given(bf16=st.booleans(), log_group=st.integers(5, 12), segments=st.integers(1, 40),
       kind=st.sampled_from(DISTS), seed=st.integers(0, 2 ** 31 - 1), sym=st.booleans())
def test_qwd_random(bf16, log_group, segments, kind, seed, sym):
    group = 1 << log_group
    n = group * segments
    r = np.random.default_rng(seed)
    base = (r.standard_normal(n) * 0.02).astype(np.float32)
    if bf16:
        prev = (base.view(np.uint32) >> 16).astype(np.uint16)
        widened = (prev.astype(np.uint32) << 16).view(np.float32)
    else:
        prev = base
        widened = base
    new = (widened + draw_values(kind, n, seed + 1) * np.float32(1e-3)).astype(np.float32)
    pd = dev(prev)
    if sym:
        codes, scale = empty(n // 2, "u8"), empty(n // group, "f32")
        sdp4.sdp4_qwd_encode_sym(dev(new), pd, group, codes, scale)
        sdp4.sdp4_qwd_decode_sym(codes, scale, group, pd)
        sync()
        rc, rs, pre = oracle.qwd_encode_sym(new, prev, group)
        check_headers(host(scale), rs)
        check_codes(host(codes), rc, pre, n, 4)
        want = oracle.qwd_decode_sym(rc, rs, prev, group)
        assert np.array_equal(host(pd).view(np.uint8), np.ascontiguousarray(want).view(np.uint8))
        return
    codes, scale, minv = empty(n // 2, "u8"), empty(n // group, "f32"), empty(n // group, "f32")
    sdp4.sdp4_qwd_encode(dev(new), pd, group, codes, scale, minv)
    sdp4.sdp4_qwd_decode(codes, scale, minv, group, pd)
    sync()
    rc, rs, rm, pre = oracle.qwd_encode(new, prev, group)
    check_headers(host(minv), rm, "minv")
    check_headers(host(scale), rs)
    check_codes(host(codes), rc, pre, n, 4, signed=False)
    want = oracle.qwd_decode(rc, rs, rm, prev, group)
    got = host(pd)
    assert np.array_equal(got.view(np.uint8), np.ascontiguousarray(want).view(np.uint8))
