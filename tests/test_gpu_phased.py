"""The qWD encoder's phased mode (large launches with bfloat16 model weights:
loads only in the read part of a clock period, outputs buffered in LDS and
written in the rest) against the oracle on every element: groups 64..1024,
both codecs, and a shard whose last wave tile is partial.  Float32 model
weights stream at every size, so their cases check the streaming encoder at
the same size.  The
8-bit K1 and the 4-bit re-quantizing dequantize-reduce (K2: 8- and 4-bit peer
messages, 2..16 peers) are checked at the same size; they stream without
phases."""
import numpy as np
import pytest

import oracle
from paper_2410_15526_amd import sdp4
from tests._gpu import check_codes, check_headers, dev, empty, host, say, torch

pytestmark = pytest.mark.gpu

N = (1 << 26) + 3 * 1024          # above the phased-mode threshold; 3/2 tiles past a whole number


def inputs(bf16, seed):
    r = np.random.default_rng(seed)
    base = (r.standard_normal(N) * 0.02).astype(np.float32)
    if bf16:
        prev = (base.view(np.uint32) >> 16).astype(np.uint16)
        wide = (prev.astype(np.uint32) << 16).view(np.float32)
    else:
        prev, wide = base, base
    new = (wide + (r.standard_t(3, N) * 5e-4).astype(np.float32)).astype(np.float32)
    return new, prev


@pytest.mark.parametrize("bf16,group", [(True, 64), (False, 64), (True, 128), (True, 256), (False, 256), (True, 512),
                                        (True, 1024), (False, 1024)])
def test_phased_asymmetric_encode_matches_oracle(bf16, group):
    say(f"phased qwd encode bf16={bf16} group={group} n={N}")
    new, prev = inputs(bf16, group)
    codes, scale, minv = empty(N // 2, "u8"), empty(N // group, "f32"), empty(N // group, "f32")
    sdp4.sdp4_qwd_encode(dev(new), dev(prev), group, codes, scale, minv)
    torch().cuda.synchronize()
    rc, rs, rm, pre = oracle.qwd_encode(new, prev, group)
    check_headers(host(scale), rs)
    check_headers(host(minv), rm, "minv")
    check_codes(host(codes), rc, pre, N, 4, signed=False)


@pytest.mark.parametrize("bf16,group", [(True, 64), (True, 128), (False, 512)])
def test_phased_symmetric_encode_matches_oracle(bf16, group):
    say(f"phased qwd encode sym bf16={bf16} group={group} n={N}")
    new, prev = inputs(bf16, 7 * group)
    codes, scale = empty(N // 2, "u8"), empty(N // group, "f32")
    sdp4.sdp4_qwd_encode_sym(dev(new), dev(prev), group, codes, scale)
    torch().cuda.synchronize()
    rc, rs, pre = oracle.qwd_encode_sym(new, prev, group)
    check_headers(host(scale), rs)
    check_codes(host(codes), rc, pre, N, 4)


@pytest.mark.parametrize("block,group", [(256, 128), (0, 256), (32, 512), (1024, 1024)])
def test_large_k1_matches_oracle(block, group):
    """8-bit K1 (Hadamard + quantization) on a large shard, every element."""
    say(f"large k1 block={block} group={group} n={N}")
    r = np.random.default_rng(block + group)
    x = (r.standard_normal(N) * 1e-4).astype(np.float32)
    x[r.integers(0, N, N // 1000)] *= 100.0
    codes, scale = empty(N, "u8"), empty(N // group, "f32")
    sdp4.sdp4_grad_quant(dev(x), 8, block, group, codes, scale)
    torch().cuda.synchronize()
    rc, rs, pre = oracle.grad_quant(x, 8, block, group)
    check_headers(host(scale), rs)
    check_codes(host(codes), rc, pre, N, 8)


@pytest.mark.parametrize("P,bits_in,group", [(8, 8, 128), (3, 8, 256), (2, 8, 1024), (4, 4, 128), (16, 4, 512)])
def test_large_requant_matches_oracle(P, bits_in, group):
    """Dequantize-reduce over P peers with 4-bit re-quantization (K2), every element."""
    say(f"large dequant_reduce requant P={P} in={bits_in} group={group} n={N}")
    r = np.random.default_rng(100 * P + bits_in + group)
    qmax = 127 if bits_in == 8 else 7
    codes, scales = [], []
    for _ in range(P):
        q = r.integers(-qmax, qmax + 1, N).astype(np.int8)
        codes.append(q.view(np.uint8) if bits_in == 8 else oracle.pack4(q))
        scales.append((r.random(N // group) * 1e-4).astype(np.float32))
    oc, osc = empty(N // 2, "u8"), empty(N // group, "f32")
    sdp4.sdp4_dequant_reduce([dev(c) for c in codes], [dev(x) for x in scales], N, bits_in, group, 4, 0, 1.0,
                             oc, osc, None)
    torch().cuda.synchronize()
    ref = oracle.dequant_reduce(codes, scales, N, bits_in, group, 4)
    check_headers(host(osc), ref["scales"])
    check_codes(host(oc), ref["codes"], ref["pre"], N, 4)
