"""One GPU's share of the SDP4Bit hot path: device buffers and launch order.

Per training step a GPU runs (Alg. 2 and Alg. 4 of the paper):

1. ``qwd_encode``   weight difference of its shard -> 4-bit message
2. ``qwd_decode``   gathered 4-bit messages -> model weights, in place
3. ``grad_quant``   local gradient -> Hadamard -> 8-bit message (P chunks)
4. ``reduce_intra`` P received 8-bit chunks -> dequantize, reduce -> 4-bit (Q chunks)
5. ``reduce_inter`` Q received 4-bit chunks -> dequantize, reduce, inverse Hadamard

On one GPU the all-gather and the two all-to-alls are replaced by pointer
slicing: the P chunks of the local 8-bit message stand in for the chunks
received from the P local peers, and the Q chunks of the local 4-bit
message for those received from the Q nodes.  Every kernel therefore reads
and writes exactly the bytes it would in the distributed run, at the real
per-GPU shape.  The collectives themselves are not part of this module.
"""
from __future__ import annotations

from dataclasses import dataclass

from . import sdp4


@dataclass(frozen=True)
class KernelInfo:
    name: str
    alg_bytes: int        # bytes the method must move per launch (reads + writes)
    fp32_in_bytes: int    # 4 x input elements (the "fp32 input processed" yardstick)
    read_bytes: int = 0   # the reads among alg_bytes (the rest are writes)


class HotPath:
    def __init__(self, n: int, group: int, hadamard_block: int, P: int, Q: int, qwd_group: int,
                 prev_dtype: str, device: str = "cuda"):
        import torch
        lcm = max(group, hadamard_block)
        if n % (P * Q * lcm) or n % qwd_group:
            raise ValueError("n must be a multiple of P*Q*max(group, block) and of the qWD group")
        self.n, self.group, self.block, self.P, self.Q = n, group, hadamard_block, P, Q
        self.qwd_group, self.prev_dtype = qwd_group, prev_dtype
        self.M = n // P                   # elements per intra-node chunk
        self.m = self.M // Q              # elements per inter-node chunk = final shard
        f32, u8 = torch.float32, torch.uint8
        e = lambda k, dt: torch.empty(k, dtype=dt, device=device)
        self.w_new = e(n, f32)
        self.w_prev = e(n, torch.bfloat16 if prev_dtype == "bf16" else f32)
        self.qcodes = e(n // 2, u8)
        self.qscale = e(n // qwd_group, f32)
        self.qmin = e(n // qwd_group, f32)
        self.grad = e(n, f32)
        self.c8 = e(n, u8)
        self.s8 = e(n // group, f32)
        self.c4 = e(self.M // 2, u8)
        self.s4 = e(self.M // group, f32)
        self.out = e(self.m, f32)
        self.out_scale = 1.0 / (P * Q)
        self._unfused = None

    def with_groups(self, group: int | None = None, qwd_group: int | None = None) -> "HotPath":
        """The same data buffers with other group sizes (new header arrays
        only), for group-size sweeps on one shard."""
        import copy
        import torch
        h = copy.copy(self)
        e = lambda k: torch.empty(k, dtype=torch.float32, device=self.grad.device)
        if group is not None and group != self.group:
            if self.n % (self.P * self.Q * max(group, self.block)):
                raise ValueError("n must be a multiple of P*Q*max(group, block)")
            h.group = group
            h.s8, h.s4 = e(self.n // group), e(self.M // group)
        if qwd_group is not None and qwd_group != self.qwd_group:
            if self.n % qwd_group:
                raise ValueError("n must be a multiple of the qWD group")
            h.qwd_group = qwd_group
            h.qscale, h.qmin = e(self.n // qwd_group), e(self.n // qwd_group)
        h._unfused = None
        return h

    # -- the five launches ---------------------------------------------------
    def qwd_encode(self, stream=None):
        sdp4.sdp4_qwd_encode(self.w_new, self.w_prev, self.qwd_group, self.qcodes, self.qscale, self.qmin,
                             stream=stream)

    def qwd_decode(self, stream=None):
        sdp4.sdp4_qwd_decode(self.qcodes, self.qscale, self.qmin, self.qwd_group, self.w_prev, stream=stream)

    def qwd_encode_sym(self, stream=None):
        """The symmetric 4-bit codec (scale only) in place of the min-max one."""
        sdp4.sdp4_qwd_encode_sym(self.w_new, self.w_prev, self.qwd_group, self.qcodes, self.qscale, stream=stream)

    def qwd_decode_sym(self, stream=None):
        sdp4.sdp4_qwd_decode_sym(self.qcodes, self.qscale, self.qwd_group, self.w_prev, stream=stream)

    def grad_quant(self, stream=None, bits=8, block=None):
        block = self.block if block is None else block
        sdp4.sdp4_grad_quant(self.grad, bits, block, self.group, self.c8, self.s8, stream=stream)

    def intra_chunks(self, bits=8):
        M, g = self.M, self.group
        cb = M * bits // 8
        return ([self.c8[p * cb:(p + 1) * cb] for p in range(self.P)],
                [self.s8[p * M // g:(p + 1) * M // g] for p in range(self.P)])

    def inter_chunks(self):
        m, g = self.m, self.group
        return ([self.c4[q * m // 2:(q + 1) * m // 2] for q in range(self.Q)],
                [self.s4[q * m // g:(q + 1) * m // g] for q in range(self.Q)])

    def reduce_intra(self, stream=None, bits_in=8):
        c, s = self.intra_chunks(bits_in)
        sdp4.sdp4_dequant_reduce(c, s, self.M, bits_in, self.group, 4, 0, 1.0, self.c4, self.s4, None,
                                 stream=stream)

    def reduce_inter(self, stream=None, block=None):
        block = self.block if block is None else block
        c, s = self.inter_chunks()
        sdp4.sdp4_dequant_reduce(c, s, self.m, 4, self.group, 0, block, self.out_scale, None, None,
                                 self.out, stream=stream)

    # seeds of the stochastically rounded variant (first and second level)
    SR_SEEDS = (0x5D94_0001, 0x5D94_0002)

    def grad_quant_sr(self, stream=None, bits=8, block=None):
        block = self.block if block is None else block
        sdp4.sdp4_grad_quant_sr(self.grad, bits, block, self.group, self.SR_SEEDS[0], 0, self.c8, self.s8,
                                stream=stream)

    def reduce_intra_sr(self, stream=None, bits_in=8):
        c, s = self.intra_chunks(bits_in)
        sdp4.sdp4_dequant_reduce_sr(c, s, self.M, bits_in, self.group, 4, self.SR_SEEDS[1], 0, self.c4, self.s4,
                                    stream=stream)

    def gradient_variant(self, name: str, stream=None):
        """The paper's gradient strategies (Sec. 5.1, Sec. 5.4) on the same kernels:
        TLq-HS (8-bit then 4-bit, Hadamard), TLq (no Hadamard), ULq (4-bit twice,
        no Hadamard), and TLq-HS with stochastic rounding at both levels."""
        if name == "tlq_hs_sr":
            self.grad_quant_sr(stream)
            self.reduce_intra_sr(stream)
            self.reduce_inter(stream)
            return
        bits1, block = {"tlq_hs": (8, self.block), "tlq": (8, 0), "ulq": (4, 0)}[name]
        self.grad_quant(stream, bits=bits1, block=block)
        self.reduce_intra(stream, bits_in=bits1)
        self.reduce_inter(stream, block=block)

    def launches(self):
        return [("qwd_encode", self.qwd_encode), ("qwd_decode", self.qwd_decode),
                ("grad_quant", self.grad_quant), ("reduce_intra", self.reduce_intra),
                ("reduce_inter", self.reduce_inter)]

    def step(self, stream=None, events=None):
        """One pass of the whole path; ``events`` (dict name -> list) collects (start, end) pairs."""
        import torch
        for name, fn in self.launches():
            if events is not None:
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                fn(stream)
                b.record()
                events.setdefault(name, []).append((a, b))
            else:
                fn(stream)

    # -- byte accounting -------------------------------------------------------
    def kernel_info(self):
        n, g, qg, P, Q, M, m = self.n, self.group, self.qwd_group, self.P, self.Q, self.M, self.m
        esz = 2 if self.prev_dtype == "bf16" else 4
        return {
            "qwd_encode": KernelInfo("qwd_encode", 4 * n + esz * n + n // 2 + 8 * (n // qg), 4 * n, 4 * n + esz * n),
            "qwd_decode": KernelInfo("qwd_decode", n // 2 + 8 * (n // qg) + 2 * esz * n, 4 * n,
                                     n // 2 + 8 * (n // qg) + esz * n),
            "grad_quant": KernelInfo("grad_quant", 4 * n + n + 4 * (n // g), 4 * n, 4 * n),
            "reduce_intra": KernelInfo("reduce_intra", P * (M + 4 * (M // g)) + M // 2 + 4 * (M // g), 4 * P * M,
                                       P * (M + 4 * (M // g))),
            "reduce_inter": KernelInfo("reduce_inter", Q * (m // 2 + 4 * (m // g)) + 4 * m, 4 * Q * m,
                                       Q * (m // 2 + 4 * (m // g))),
        }

    # -- the unfused variant ("HS w/o fused") ----------------------------------
    def unfused_gradient_step(self, stream=None):
        """Same gradient path with the transform and the (de)quantization as
        separate launches and float32 intermediates in HBM.

        The averaging factor ``out_scale`` rides on the second-level
        dequantization of each chunk (no extra pass).  For the power-of-two
        1/(P*Q) of every workload here, scaling commutes exactly with the
        float32 sum and the transform that follow (barring subnormals), so
        the result is the fused path's up to the rounding of the separate
        products and sums."""
        import torch
        if self._unfused is None:
            e = lambda k, dt: torch.empty(k, dtype=dt, device=self.grad.device)
            self._unfused = dict(h=e(self.n, torch.float32), d=e(self.n, torch.float32),
                                 r=e(self.M, torch.float32), d2=e(self.M, torch.float32),
                                 r2=e(self.m, torch.float32))
        u = self._unfused
        n, M, m, g, P, Q = self.n, self.M, self.m, self.group, self.P, self.Q
        sdp4.sdp4_hadamard(self.grad, u["h"], self.block, stream=stream)
        sdp4.sdp4_grad_quant(u["h"], 8, 0, g, self.c8, self.s8, stream=stream)
        c, s = self.intra_chunks()
        for p in range(P):
            sdp4.sdp4_dequant_reduce([c[p]], [s[p]], M, 8, g, 0, 0, 1.0, None, None, u["d"][p * M:(p + 1) * M],
                                     stream=stream)
        sdp4.sdp4_reduce_f32([u["d"][p * M:(p + 1) * M] for p in range(P)], u["r"], stream=stream)
        sdp4.sdp4_grad_quant(u["r"], 4, 0, g, self.c4, self.s4, stream=stream)
        c, s = self.inter_chunks()
        for q in range(Q):
            sdp4.sdp4_dequant_reduce([c[q]], [s[q]], m, 4, g, 0, 0, self.out_scale, None, None,
                                     u["d2"][q * m:(q + 1) * m], stream=stream)
        sdp4.sdp4_reduce_f32([u["d2"][q * m:(q + 1) * m] for q in range(Q)], u["r2"], stream=stream)
        sdp4.sdp4_hadamard(u["r2"], self.out, self.block, stream=stream)
