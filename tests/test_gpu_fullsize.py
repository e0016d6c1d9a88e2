"""Parity at the full shard sizes of the five workloads, in the launch
configuration the benchmark times (paper_2410_15526_amd.pipeline.HotPath).

The GPU runs one full step on the whole shard.  The oracle then recomputes
segments from regenerated inputs (the generators are addressable by element
range), following the same chunk routing: an output segment of the final
4-bit reduction needs the matching segment of each of the Q 4-bit chunks,
each of which needs the matching segment of each of the P 8-bit chunks.
Sampled segments include the first and the last of every buffer (the ragged
end of the last wave tile) and random ones in between; on c1, c4 and c5
every output element is compared.
"""
import numpy as np
import pytest

import oracle
import synth
from paper_2410_15526_amd import sdp4
from paper_2410_15526_amd.pipeline import HotPath
from tests._gpu import check_codes, check_f32, check_headers, fill, host, say, torch

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def segments(length, seg, count, seed):
    """Start offsets (multiples of seg) of `count` segments inside [0, length)."""
    r = np.random.default_rng(seed)
    k = length // seg
    picks = {0, k - 1} | set(int(v) for v in r.integers(0, k, count))
    return sorted(p * seg for p in picks)


def build(w, seed=0):
    hp = HotPath(w.n, w.group, w.hadamard_block, w.P, w.Q, w.qwd_group, w.prev_dtype)
    say(f"fill {w.describe()}")
    fill(hp.w_prev, lambda s, k: synth.prev_weights(w, s, k, seed), w.n)
    fill(hp.w_new, lambda s, k: synth.new_weights(w, s, k, seed), w.n)
    fill(hp.grad, lambda s, k: synth.gradient(w, s, k, seed), w.n)
    torch().cuda.synchronize()
    return hp


def check_qwd(hp, w, seed, starts, L):
    g = w.qwd_group
    for a in starts:
        new = synth.new_weights(w, a, L, seed)
        prev = synth.prev_weights(w, a, L, seed)
        rc, rs, rm, pre = oracle.qwd_encode(new, prev, g)
        check_codes(host(hp.qcodes[a // 2:(a + L) // 2]), rc, pre, L, 4, signed=False, what=f"qwd@{a}")
        check_headers(host(hp.qscale[a // g:(a + L) // g]), rs, f"qscale@{a}")
        check_headers(host(hp.qmin[a // g:(a + L) // g]), rm, f"qmin@{a}")
        want = oracle.qwd_decode(rc, rs, rm, prev, g)
        got = host(hp.w_prev[a:a + L])
        assert np.array_equal(got.view(np.uint8), np.ascontiguousarray(want).view(np.uint8)), f"decode@{a}"


def k1_ref(w, seed, a, L, bits=8, block=None, sr=None):
    x = synth.gradient(w, a, L, seed)
    block = w.hadamard_block if block is None else block
    if sr is not None:                      # stochastic rounding: element offset = position a
        return oracle.grad_quant_sr(x, bits, block, w.group, sr[0], a)
    return oracle.grad_quant(x, bits, block, w.group)


def k2_ref(w, seed, x, L, bits=8, block=None, sr=None):
    """Oracle K2 output segment [x, x+L) of the intra-node reduction."""
    M, g = w.n // w.P, w.group
    k1 = [k1_ref(w, seed, p * M + x, L, bits, block, sr) for p in range(w.P)]
    if sr is not None:
        return oracle.dequant_reduce_sr([c for c, _, _ in k1], [s for _, s, _ in k1], L, bits, g, 4, sr[1], x,
                                        want_f32=False)
    return oracle.dequant_reduce([c for c, _, _ in k1], [s for _, s, _ in k1], L, bits, g, 4, want_f32=False)


def check_gradient_path(hp, w, seed, starts_k1, starts_k3, L, bits=8, block=None, sr=None):
    block = w.hadamard_block if block is None else block
    g, M, m = w.group, w.n // w.P, w.n // w.P // w.Q
    for a in starts_k1:
        rc, rs, pre = k1_ref(w, seed, a, L, bits, block, sr)
        check_codes(host(hp.c8[a * bits // 8:(a + L) * bits // 8]), rc, pre, L, bits, what=f"k1@{a}")
        check_headers(host(hp.s8[a // g:(a + L) // g]), rs, f"k1 scale@{a}")
    for a in starts_k3:
        parts = []
        for q in range(w.Q):
            r = k2_ref(w, seed, q * m + a, L, bits, block, sr)
            x = q * m + a
            check_codes(host(hp.c4[x // 2:(x + L) // 2]), r["codes"], r["pre"], L, 4, what=f"k2@{x}")
            check_headers(host(hp.s4[x // g:(x + L) // g]), r["scales"], f"k2 scale@{x}")
            parts.append(r)
        want = oracle.dequant_reduce([r["codes"] for r in parts], [r["scales"] for r in parts], L, 4, g, 0,
                                     block, 1.0 / (w.P * w.Q))["f32"]
        check_f32(host(hp.out[a:a + L]), want, f"k3@{a}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_shard_step(name):
    w = synth.WORKLOADS[name]
    seed = 0
    hp = build(w, seed)
    say(f"{name}: one step of the hot path on N={w.n:,}")
    hp.step()
    torch().cuda.synchronize()
    L = 4 * max(w.group, w.hadamard_block, w.qwd_group)
    m = w.n // w.P // w.Q
    check_qwd(hp, w, seed, segments(w.n, L, 12, 1), L)
    check_gradient_path(hp, w, seed, segments(w.n, L, 12, 2), segments(m, L, 6, 3), L)
    say(f"{name}: sampled parity ok")

    if name == "c4":
        # group-size sweep of the gradient quantizer and of qWD at the full size
        for g in (32, 64, 256, 512):
            say(f"c4 grad_quant group {g}")
            c8 = torch().empty(w.n, dtype=torch().uint8, device="cuda")
            s8 = torch().empty(w.n // g, device="cuda")
            sdp4.sdp4_grad_quant(hp.grad, 8, w.hadamard_block, g, c8, s8)
            torch().cuda.synchronize()
            for a in segments(w.n, 4 * max(g, w.hadamard_block), 8, g):
                Lg = 4 * max(g, w.hadamard_block)
                rc, rs, pre = oracle.grad_quant(synth.gradient(w, a, Lg, seed), 8, w.hadamard_block, g)
                check_codes(host(c8[a:a + Lg]), rc, pre, Lg, 8, what=f"k1 g{g}@{a}")
                check_headers(host(s8[a // g:(a + Lg) // g]), rs)
            del c8, s8
        for qg in (64, 256):
            say(f"c4 qWD group {qg}")
            codes = torch().empty(w.n // 2, dtype=torch().uint8, device="cuda")
            sc = torch().empty(w.n // qg, device="cuda")
            mn = torch().empty(w.n // qg, device="cuda")
            fill(hp.w_prev, lambda s, k: synth.prev_weights(w, s, k, seed), w.n)
            sdp4.sdp4_qwd_encode(hp.w_new, hp.w_prev, qg, codes, sc, mn)
            torch().cuda.synchronize()
            for a in segments(w.n, 4 * qg, 8, qg):
                Lq = 4 * qg
                rc, rs, rm, pre = oracle.qwd_encode(synth.new_weights(w, a, Lq, seed),
                                                    synth.prev_weights(w, a, Lq, seed), qg)
                check_codes(host(codes[a // 2:(a + Lq) // 2]), rc, pre, Lq, 4, signed=False)
                check_headers(host(sc[a // qg:(a + Lq) // qg]), rs)
                check_headers(host(mn[a // qg:(a + Lq) // qg]), rm)
        say("c4 symmetric qWD group 128")
        g = 128
        fill(hp.w_prev, lambda s, k: synth.prev_weights(w, s, k, seed), w.n)
        hp.qwd_encode_sym()
        hp.qwd_decode_sym()
        torch().cuda.synchronize()
        for a in segments(w.n, 4 * g, 8, 12):
            Lq = 4 * g
            prev = synth.prev_weights(w, a, Lq, seed)
            rc, rs, pre = oracle.qwd_encode_sym(synth.new_weights(w, a, Lq, seed), prev, g)
            check_codes(host(hp.qcodes[a // 2:(a + Lq) // 2]), rc, pre, Lq, 4, what=f"qwd sym@{a}")
            check_headers(host(hp.qscale[a // g:(a + Lq) // g]), rs)
            want = oracle.qwd_decode_sym(rc, rs, prev, g)
            assert np.array_equal(host(hp.w_prev[a:a + Lq]), want), f"qwd sym decode@{a}"
    if name == "c5":
        # the float32 model-weight variant of qWD at the full size
        say("c5 qWD with float32 model weights")
        prev32 = torch().empty(w.n, device="cuda")
        fill(prev32, lambda s, k: synth.bf16_bits_to_f32(synth.prev_weights(w, s, k, seed)), w.n)
        sdp4.sdp4_qwd_encode(hp.w_new, prev32, w.qwd_group, hp.qcodes, hp.qscale, hp.qmin)
        sdp4.sdp4_qwd_decode(hp.qcodes, hp.qscale, hp.qmin, w.qwd_group, prev32)
        torch().cuda.synchronize()
        g = w.qwd_group
        for a in segments(w.n, 4 * g, 8, 11):
            Lq = 4 * g
            prev = synth.bf16_bits_to_f32(synth.prev_weights(w, a, Lq, seed))
            rc, rs, rm, pre = oracle.qwd_encode(synth.new_weights(w, a, Lq, seed), prev, g)
            check_codes(host(hp.qcodes[a // 2:(a + Lq) // 2]), rc, pre, Lq, 4, signed=False)
            check_f32(host(prev32[a:a + Lq]), oracle.qwd_decode(rc, rs, rm, prev, g))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("variant,bits,block", [("tlq", 8, 0), ("ulq", 4, 0), ("tlq_hs_sr", 8, 256)])
def test_paper_variants_full_shard(variant, bits, block):
    """TLq (no Hadamard) and ULq (4-bit twice, no Hadamard) of Sec. 5.1 / 5.4 on
    the GPT-1.3B shard, through the same launch sequence as the benchmark."""
    w = synth.WORKLOADS["c3"]
    hp = build(w, 0)
    say(f"c3 variant {variant}")
    hp.gradient_variant(variant)
    torch().cuda.synchronize()
    L = 4 * w.group
    check_gradient_path(hp, w, 0, segments(w.n, L, 8, 5), segments(w.n // w.P // w.Q, L, 4, 6), L,
                        bits=bits, block=block, sr=HotPath.SR_SEEDS if variant.endswith("_sr") else None)


def test_tiny_shard_step_every_element():
    """c1 at its full size, every output element of the step compared."""
    w = synth.WORKLOADS["c1"]
    hp = build(w, 0)
    say("c1: one step, full comparison")
    hp.step()
    torch().cuda.synchronize()
    n, g, P, Q, M, m = w.n, w.group, w.P, w.Q, w.n // w.P, w.n // w.P // w.Q
    new, prev = synth.new_weights(w, 0, n), synth.prev_weights(w, 0, n)
    rc, rs, rm, pre = oracle.qwd_encode(new, prev, w.qwd_group)
    check_codes(host(hp.qcodes), rc, pre, n, 4, signed=False)
    check_f32(host(hp.w_prev), oracle.qwd_decode(rc, rs, rm, prev, w.qwd_group))
    k1c, k1s, pre1 = oracle.grad_quant(synth.gradient(w, 0, n), 8, w.hadamard_block, g)
    check_codes(host(hp.c8), k1c, pre1, n, 8)
    check_headers(host(hp.s8), k1s)
    r2 = oracle.dequant_reduce([k1c[p * M:(p + 1) * M] for p in range(P)],
                               [k1s[p * M // g:(p + 1) * M // g] for p in range(P)], M, 8, g, 4)
    check_codes(host(hp.c4), r2["codes"], r2["pre"], M, 4)
    r3 = oracle.dequant_reduce([r2["codes"][q * m // 2:(q + 1) * m // 2] for q in range(Q)],
                               [r2["scales"][q * m // g:(q + 1) * m // g] for q in range(Q)], m, 4, g, 0,
                               w.hadamard_block, 1.0 / (P * Q))
    check_f32(host(hp.out), r3["f32"])


@pytest.mark.timeout(900)
def test_shard_beyond_2_31_elements():
    """64-bit indexing: one step on n = 2^31 + 2^21 elements (the GPT-1.3B
    recipe extended to 43 layers); segments straddling and past element 2^31
    and the last segment are checked against the oracle."""
    w = synth.scaled(synth.WORKLOADS["c3"], (1 << 31) + (1 << 21))
    hp = build(w, 0)
    say(f"n = {w.n:,}: one step")
    hp.step()
    torch().cuda.synchronize()
    L = 1024
    big = [(1 << 31) - L, 1 << 31, (1 << 31) + 7 * L, w.n - L]
    check_qwd(hp, w, 0, big, L)
    check_gradient_path(hp, w, 0, big, segments(w.n // w.P // w.Q, L, 3, 7), L)


def _pool():
    import concurrent.futures as cf
    import os
    return cf.ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0)))))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c4", "c5"])
def test_full_shard_every_element(name):
    """Every output of one step on the GPT-6.7B and GPT-13B shards against the
    oracle: qWD codes, headers and decoded weights over the whole shard, K1
    codes and scales of every element, K2 of every chunk, K3 of every output.
    The oracle runs slice by slice in threads (its C calls release the
    interpreter lock); slices follow the chunk routing of the step."""
    w = synth.WORKLOADS[name]
    seed = 0
    hp = build(w, seed)
    say(f"{name}: one step, every element")
    hp.step()
    torch().cuda.synchronize()
    n, g, qg, P, Q, nb = w.n, w.group, w.qwd_group, w.P, w.Q, w.hadamard_block
    M, m = n // P, n // P // Q
    exempt = 0  # codes that differ at a near-tie (the parity bar's exemption), reported below
    with _pool() as ex:
        # qWD over the whole shard, in batches of B elements cut into slices of S
        B, S = 1 << 27, 1 << 23
        for a in range(0, n, B):
            L = min(B, n - a)
            new, prev = synth.new_weights(w, a, L, seed), synth.prev_weights(w, a, L, seed)
            gc, gs, gm = host(hp.qcodes[a // 2:(a + L) // 2]), host(hp.qscale[a // qg:(a + L) // qg]), \
                host(hp.qmin[a // qg:(a + L) // qg])
            gw = host(hp.w_prev[a:a + L])

            def qwd_slice(o, new=new, prev=prev, gc=gc, gs=gs, gm=gm, gw=gw, a=a, L=L):
                k = min(S, L - o)
                rc, rs, rm, pre = oracle.qwd_encode(new[o:o + k], prev[o:o + k], qg)
                ties = check_codes(gc[o // 2:(o + k) // 2], rc, pre, k, 4, signed=False, what=f"qwd@{a + o}")
                check_headers(gs[o // qg:(o + k) // qg], rs, f"qscale@{a + o}")
                check_headers(gm[o // qg:(o + k) // qg], rm, f"qmin@{a + o}")
                want = oracle.qwd_decode(rc, rs, rm, prev[o:o + k], qg)
                assert np.array_equal(gw[o:o + k].view(np.uint8), np.ascontiguousarray(want).view(np.uint8)), \
                    f"decode@{a + o}"
                return ties
            exempt += sum(ex.map(qwd_slice, range(0, L, S)))
            del new, prev, gc, gs, gm, gw
        say(f"{name}: qWD every element ok")
        # the gradient chain, batch by batch of final outputs [a, a + L)
        c8, s8, c4, s4, out = host(hp.c8), host(hp.s8), host(hp.c4), host(hp.s4), host(hp.out)
        Lb = 1 << 21
        for a in range(0, m, Lb):
            L = min(Lb, m - a)

            def k1(pq, a=a, L=L):
                p, q = pq
                x = p * M + q * m + a                          # input element of peer p's chunk q
                rc, rs, pre = oracle.grad_quant(synth.gradient(w, x, L, seed), 8, nb, g)
                ties = check_codes(c8[x:x + L], rc, pre, L, 8, what=f"k1@{x}")
                check_headers(s8[x // g:(x + L) // g], rs, f"k1 scale@{x}")
                return rc, rs, ties
            r1 = list(ex.map(k1, [(p, q) for q in range(Q) for p in range(P)]))
            exempt += sum(r[2] for r in r1)

            def k2(q, a=a, L=L, r1=r1):
                x = q * m + a
                r = oracle.dequant_reduce([r1[q * P + p][0] for p in range(P)], [r1[q * P + p][1] for p in range(P)],
                                          L, 8, g, 4, want_f32=False)
                r["ties"] = check_codes(c4[x // 2:(x + L) // 2], r["codes"], r["pre"], L, 4, what=f"k2@{x}")
                check_headers(s4[x // g:(x + L) // g], r["scales"], f"k2 scale@{x}")
                return r
            r2 = list(ex.map(k2, range(Q)))
            exempt += sum(r["ties"] for r in r2)
            want = oracle.dequant_reduce([r["codes"] for r in r2], [r["scales"] for r in r2], L, 4, g, 0, nb,
                                         1.0 / (P * Q))["f32"]
            check_f32(out[a:a + L], want, f"k3@{a}")
        say(f"{name}: gradient chain every element ok")
    # every code compared: n qWD codes, n K1 codes, n / P K2 codes
    total = 2 * n + n // P
    say(f"{name}: near-tie exemptions {exempt} of {total:,} codes")
    assert exempt <= 1e-6 * total
