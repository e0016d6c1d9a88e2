"""Benchmark of one GPU's share of the SDP4Bit hot path on MI355X.

A step is one pass of the whole path over the GPT-13B 1/8 shard
(N = 1,625,292,800 elements; bf16 model weights, qWD group 128; Hadamard
block 256, group 128, 8-bit x P=8 then 4-bit x Q=4): qWD encode, qWD
decode, Hadamard + 8-bit quantization, 8-bit dequantize-reduce with 4-bit
re-quantization, 4-bit dequantize-reduce with the inverse Hadamard.  Inputs
are seeded synthetic data resident in HBM before timing starts.

Prints one JSON line.  ``value`` is the fp32-equivalent input throughput of
the step: 4 bytes x (input elements of every kernel) / step time.  Per
kernel the line also carries algorithmic HBM bytes / launch time against the
8 TB/s HBM peak and against a plain copy kernel measured in the same run
(``vs_copy``); ``roofline`` is the peak figure for the kernel that takes the
largest share of the step.  ``cpu_baseline`` is the plain CPU oracle timed
on a bounded sample of the same workload on this host (single thread);
``cpu_baseline_all_cores`` the same oracle over the whole workload split into
one slice per available core (up to 16), each in its own thread.
``ceilings`` holds what HBM gives plain streams at the step's array size
(read-only, write-only and copy yardsticks of the library, the runtime's own
copy and fill); each kernel's ``vs_rw_additive`` compares it with a kernel
that moved its reads at the read-only rate and its writes at the write-only
rate, one after the other.  ``graph_step`` times the same step recorded once
into a HIP graph and replayed (informational).

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 20] [--workload c5]
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "GB/s of fp32 input processed per kernel (quant, dequant-reduce); % of HBM peak"
SLAB = 1 << 26


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def fill(dst, gen, n):
    """Generate host data slab by slab and copy it into the device tensor."""
    import numpy as np
    import torch
    for s in range(0, n, SLAB):
        k = min(SLAB, n - s)
        a = np.ascontiguousarray(gen(s, k))
        t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
        if a.dtype == np.uint16:
            dst[s:s + k].view(torch.int16).copy_(t)
        else:
            dst[s:s + k].copy_(t)


def _code_tokens(text: str) -> str:
    """C/C++ source without its comments, whitespace runs collapsed (the
    kernel sources hold no string literal with a comment marker in it)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_digest() -> str:
    """Digest of the code that decides what the kernels do on the device:
    the kernels and their launch configuration (not the host-side argument
    checks of the C ABI), comments and layout ignored."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2410_15526_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f == "abi.cpp":
            continue
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode() + _code_tokens(fh.read()).encode())
    return h.hexdigest()[:16]


def traffic_for(kernel: str, workload: str = "c5"):
    """HBM traffic per launch from the committed rocprofv3 counter summary,
    or None when that summary is missing, was taken on other kernel sources,
    or on another workload."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except ValueError:
        return None
    if d.get("source_digest") != source_digest() or d.get("workload_key", "c5") != workload:
        return None
    k = d.get("kernels", {}).get(kernel)
    return None if k is None else k.get("bytes_per_launch")


def host_cpu() -> str:
    """Model name of this host's CPU and the cores this process may use."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{name}, {len(os.sched_getaffinity(0))} cores available"


def _oracle_inputs(w, lo: int, n: int, seed: int):
    import synth
    return (synth.prev_weights(w, lo, n, seed), synth.new_weights(w, lo, n, seed), synth.gradient(w, lo, n, seed))


def _oracle_step(w, prev, new, grad):
    """One full step of the oracle on one contiguous slice (its own chain:
    the slice's P chunks are the peers of the 8-bit reduction, and so on)."""
    import oracle
    n = prev.size
    P, Q, g, hb, qg = w.P, w.Q, w.group, w.hadamard_block, w.qwd_group
    M, m = n // P, n // P // Q
    c, s, mn, _ = oracle.qwd_encode(new, prev, qg)
    oracle.qwd_decode(c, s, mn, prev, qg)
    k1c, k1s, _ = oracle.grad_quant(grad, 8, hb, g)
    r = oracle.dequant_reduce([k1c[p * M:(p + 1) * M] for p in range(P)],
                              [k1s[p * M // g:(p + 1) * M // g] for p in range(P)], M, 8, g, 4, want_f32=False)
    oracle.dequant_reduce([r["codes"][q * m // 2:(q + 1) * m // 2] for q in range(Q)],
                          [r["scales"][q * m // g:(q + 1) * m // g] for q in range(Q)], m, 4, g, 0, hb,
                          1.0 / (P * Q))


def _step_fp32_bytes(w, n: int) -> int:
    return 4 * (n + n + n + n + n // w.P)


def _step_desc(w) -> str:
    return (f"one full step (qWD encode+decode, Hadamard+8-bit, 8-bit x{w.P} reduce + 4-bit, 4-bit x{w.Q} "
            f"reduce + inverse Hadamard)")


def cpu_baseline(w, sample_log2: int, seed: int):
    """The oracle on a contiguous sample of the workload: one full step."""
    n = 1 << sample_log2
    prev, new, grad = _oracle_inputs(w, 0, n, seed)
    t0 = time.perf_counter()
    _oracle_step(w, prev, new, grad)
    dt = time.perf_counter() - t0
    return {"value": round(_step_fp32_bytes(w, n) / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "seconds": round(dt, 3), "host_cpu": host_cpu(),
            "sample": f"elements [0, 2^{sample_log2}) of the same workload, {_step_desc(w)}, single-threaded "
                      f"plain C oracle"}


def cpu_baseline_all_cores(w, n_total: int, seed: int, max_threads: int = 16):
    """The same oracle on elements [0, n_total) of the workload, split into one
    contiguous slice per available core (at most max_threads), each slice a
    full step of its own in its own thread (the oracle's C calls release the
    interpreter lock).  Groups and blocks are independent, so every slice
    computes exactly what a single-threaded run computes for those elements.
    The inputs are generated before the clock starts."""
    import concurrent.futures as cf
    import math
    T = max(1, min(len(os.sched_getaffinity(0)), max_threads))
    unit = w.P * w.Q * math.lcm(w.group, w.hadamard_block or 1, w.qwd_group)
    per = n_total // T // unit * unit
    if per == 0:
        T, per = 1, n_total // unit * unit
    slices = [_oracle_inputs(w, i * per, per, seed) for i in range(T)]
    with cf.ThreadPoolExecutor(T) as ex:
        t0 = time.perf_counter()
        list(ex.map(lambda a: _oracle_step(w, *a), slices))
        dt = time.perf_counter() - t0
    whole = "the whole workload" if T * per == w.n else f"elements [0, {T * per}) of the same workload"
    return {"value": round(_step_fp32_bytes(w, per) * T / dt / 1e9, 4), "unit": "GB/s", "cores": T,
            "kind": "oracle", "seconds": round(dt, 3), "host_cpu": host_cpu(),
            "sample": f"{whole} in {T} slices of {per}, {_step_desc(w)} per slice, one thread per slice, "
                      f"plain C oracle"}


def ceilings(n: int, timed):
    """What HBM gives plain streams at the step's own array size (n float32
    elements, 4n bytes each way): the library's read-only, write-only and copy
    yardsticks, and the runtime's own device-to-device copy and fill."""
    import torch
    from paper_2410_15526_amd import sdp4
    x = torch.empty(n, device="cuda")
    y = torch.empty(n, device="cuda")
    sdp4.sdp4_fill_f32(x, 1.0)
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    gb = lambda nbytes, ms: round(nbytes / (ms * 1e-3) / 1e9, 1)
    out = {"array_bytes": 4 * n}
    out["read_GBps"] = gb(4 * n, timed(lambda: sdp4.sdp4_read_f32(x, sink), reps=5))
    out["write_GBps"] = gb(4 * n, timed(lambda: sdp4.sdp4_fill_f32(y, 0.0), reps=5))
    out["copy_GBps"] = gb(8 * n, timed(lambda: sdp4.sdp4_copy_f32(x, y), reps=5))
    out["runtime_copy_GBps"] = gb(8 * n, timed(lambda: y.copy_(x), reps=5))
    out["runtime_fill_GBps"] = gb(4 * n, timed(lambda: y.fill_(0.5), reps=5))
    for k in list(out):
        if k.endswith("_GBps"):
            out[k.replace("_GBps", "_frac")] = round(out[k] / HBM_PEAK_GBPS, 4)
    del x, y, sink
    torch.cuda.empty_cache()
    return out


def rw_additive_GBps(read_bytes: int, write_bytes: int, c: dict) -> float:
    """Rate of a kernel that moved its reads at the read-only ceiling and
    its writes at the write-only ceiling, one after the other (no penalty
    for mixing the two: an upper bound)."""
    t = read_bytes / (c["read_GBps"] * 1e9) + write_bytes / (c["write_GBps"] * 1e9)
    return (read_bytes + write_bytes) / t / 1e9


def workload_from_args(args):
    """The named workload with any shape overrides from the command line."""
    from dataclasses import replace
    import synth
    w = synth.WORKLOADS[args.workload]
    over = {k: v for k, v in (("n", args.n), ("group", args.group), ("hadamard_block", args.hblock), ("P", args.P),
                              ("Q", args.Q), ("qwd_group", args.qwd_group), ("prev_dtype", args.model_weights))
            if v is not None}
    if over:
        w = replace(w, extra_groups=(), extra_qwd_groups=(), **over)
    return w


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c5")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-sample-log2", type=int, default=29)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--no-variants", action="store_true")
    ap.add_argument("--no-table5", action="store_true")
    ap.add_argument("--no-standalone", action="store_true")
    ap.add_argument("--no-group-sweep", action="store_true")
    ap.add_argument("--no-ceilings", action="store_true")
    ap.add_argument("--no-graph", action="store_true")
    # overrides of the workload's shape (the recipe of its data stays that of --workload)
    ap.add_argument("--n", type=int, default=None, help="element count of the shard")
    ap.add_argument("--group", type=int, default=None, help="gradient quantization group")
    ap.add_argument("--hblock", type=int, default=None, help="Hadamard block (0 = none)")
    ap.add_argument("--P", type=int, default=None, help="chunks of the 8-bit dequantize-reduce")
    ap.add_argument("--Q", type=int, default=None, help="chunks of the 4-bit dequantize-reduce")
    ap.add_argument("--qwd-group", type=int, default=None, help="qWD quantization group")
    ap.add_argument("--model-weights", choices=("f32", "bf16"), default=None)
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU's share of the hot path; runs on more than one GPU are not "
              "supported (the collectives between the kernels are not part of this library).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2410_15526_amd import sdp4
    from paper_2410_15526_amd.pipeline import HotPath

    w = workload_from_args(args)
    torch.cuda.set_device(0)
    hp = HotPath(w.n, w.group, w.hadamard_block, w.P, w.Q, w.qwd_group, w.prev_dtype)
    t_fill = time.perf_counter()
    fill(hp.w_prev, lambda s, k: synth.prev_weights(w, s, k, args.seed), w.n)
    fill(hp.w_new, lambda s, k: synth.new_weights(w, s, k, args.seed), w.n)
    fill(hp.grad, lambda s, k: synth.gradient(w, s, k, args.seed), w.n)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.perf_counter() - t_fill:.1f} s: {w.describe()}")

    for _ in range(args.warmup):
        hp.step()
    torch.cuda.synchronize()
    events = {}
    t0 = time.perf_counter()
    for _ in range(args.steps):
        hp.step(events=events)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step")

    # copy-kernel yardstick (2 GiB read + 2 GiB written), after the timed steps so that it runs on a
    # GPU as warm as the one the steps ran on
    cn = 1 << 29
    src = torch.empty(cn, device="cuda")
    dst = torch.empty(cn, device="cuda")
    for _ in range(3):
        sdp4.sdp4_copy_f32(src, dst)
    torch.cuda.synchronize()
    ce = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ce[0].record()
    for _ in range(10):
        sdp4.sdp4_copy_f32(src, dst)
    ce[1].record()
    torch.cuda.synchronize()
    copy_gbps = 2 * 4 * cn * 10 / (ce[0].elapsed_time(ce[1]) * 1e-3) / 1e9
    del src, dst

    # the same step recorded once into a HIP graph and replayed: no per-kernel events and no host
    # launch work inside the timed replays (informational; `value` is the eager step above)
    graph_ms = None
    if not args.no_graph:
        g = torch.cuda.CUDAGraph()
        gs = torch.cuda.Stream()
        gs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(gs):
            with torch.cuda.graph(g, stream=gs):
                hp.step()
        torch.cuda.current_stream().wait_stream(gs)
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        tg = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - tg) * 1e3 / args.steps
        del g
        log(f"{args.steps} graph replays of the step: {graph_ms:.3f} ms/step")

    info = hp.kernel_info()
    kernels = {}
    for name, pairs in events.items():
        per = sorted(a.elapsed_time(b) for a, b in pairs)
        ms = sum(per) / len(per)
        med = per[len(per) // 2] if len(per) % 2 else 0.5 * (per[len(per) // 2 - 1] + per[len(per) // 2])
        std = (sum((x - ms) ** 2 for x in per) / max(len(per) - 1, 1)) ** 0.5
        ki = info[name]
        alg = ki.alg_bytes / (ms * 1e-3) / 1e9
        kernels[name] = {"ms": round(ms, 4), "ms_median": round(med, 4), "ms_std": round(std, 4),
                         "alg_bytes": ki.alg_bytes, "alg_GBps": round(alg, 1),
                         "hbm_frac": round(alg / HBM_PEAK_GBPS, 4),
                         "vs_copy": round(alg / copy_gbps, 4),
                         "fp32_in_GBps": round(ki.fp32_in_bytes / (ms * 1e-3) / 1e9, 1),
                         "elems_per_s": round(ki.fp32_in_bytes / 4 / (ms * 1e-3), 1)}
    dom = max(kernels, key=lambda k: kernels[k]["ms"])
    dk = kernels[dom]
    fp32_total = sum(k.fp32_in_bytes for k in info.values())
    value = fp32_total / (ms_step * 1e-3) / 1e9

    unfused = None
    if not args.no_unfused:
        for _ in range(2):
            hp.unfused_gradient_step()
        torch.cuda.synchronize()
        ue = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ue[0].record()
        for _ in range(5):
            hp.grad_quant(); hp.reduce_intra(); hp.reduce_inter()
        ue[1].record()
        ue[2].record()
        for _ in range(5):
            hp.unfused_gradient_step()
        ue[3].record()
        torch.cuda.synchronize()
        unfused = {"fused_gradient_ms": round(ue[0].elapsed_time(ue[1]) / 5, 4),
                   "unfused_gradient_ms": round(ue[2].elapsed_time(ue[3]) / 5, 4)}

    # Isolated timings (the paper's ablation variants on the same kernels and shard, the group sweep,
    # Table 5): a short kernel runs faster than the host can
    # issue it through the binding, so a ~2 ms spin kernel goes first and keeps the GPU busy while the
    # timed launches are enqueued; the events then see back-to-back launches only.
    sa, sb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    sa.record()
    torch.cuda._sleep(1 << 20)
    sb.record()
    torch.cuda.synchronize()
    spin_cycles = int((1 << 20) * 2.0 / max(sa.elapsed_time(sb), 1e-3))

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(spin_cycles)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return round(a.elapsed_time(b) / reps, 4)

    # each step kernel alone over back-to-back launches (no event pair per launch, whose ~5 us of
    # dispatch and event processing is a visible share of the short kernels)
    for name, fn in hp.launches():
        ms = timed(lambda: fn(None), reps=10)
        gbps = info[name].alg_bytes / (ms * 1e-3) / 1e9
        kernels[name]["ms_isolated"] = ms
        kernels[name]["hbm_frac_isolated"] = round(gbps / HBM_PEAK_GBPS, 4)

    # read-only / write-only / copy ceilings at the step's array size, and each kernel against the
    # bound its own mix of reads and writes would have at those rates
    ceil = None
    if not args.no_ceilings:
        ceil = ceilings(w.n, timed)
        for name, k in kernels.items():
            ki = info[name]
            bound = rw_additive_GBps(ki.read_bytes, ki.alg_bytes - ki.read_bytes, ceil)
            k["read_share"] = round(ki.read_bytes / ki.alg_bytes, 4)
            k["rw_additive_GBps"] = round(bound, 1)
            k["vs_rw_additive"] = round(k["alg_GBps"] / bound, 4)

    variants = {}
    if not args.no_variants:
        for v in ("tlq_hs", "tlq", "ulq", "tlq_hs_sr"):
            variants[f"{v}_gradient_ms"] = timed(lambda: hp.gradient_variant(v))
        g2 = 2048
        codes = torch.empty(w.n // 2, dtype=torch.uint8, device="cuda")
        sc = torch.empty(w.n // g2, device="cuda")
        mn = torch.empty(w.n // g2, device="cuda")
        variants["qwd_g2048_encode_ms"] = timed(lambda: sdp4.sdp4_qwd_encode(hp.w_new, hp.w_prev, g2, codes, sc, mn))
        variants["qwd_g2048_decode_ms"] = timed(lambda: sdp4.sdp4_qwd_decode(codes, sc, mn, g2, hp.w_prev))
        zero = torch.zeros(w.n, dtype=hp.w_prev.dtype, device="cuda")
        variants["qw_g2048_encode_ms"] = timed(lambda: sdp4.sdp4_qwd_encode(hp.w_new, zero, g2, codes, sc, mn))
        del codes, sc, mn, zero
        variants["qwd_sym_encode_ms"] = timed(hp.qwd_encode_sym)
        variants["qwd_sym_decode_ms"] = timed(hp.qwd_decode_sym)
        if w.prev_dtype == "bf16":
            # the same shard with float32 model weights: 8.5 bytes per element + 8 per group, each way
            wf = hp.w_prev.float()
            qg = w.qwd_group
            ms_e = timed(lambda: sdp4.sdp4_qwd_encode(hp.w_new, wf, qg, hp.qcodes, hp.qscale, hp.qmin))
            ms_d = timed(lambda: sdp4.sdp4_qwd_decode(hp.qcodes, hp.qscale, hp.qmin, qg, wf))
            alg = w.n * 17 // 2 + 8 * (w.n // qg)
            variants["qwd_f32_encode_ms"], variants["qwd_f32_decode_ms"] = ms_e, ms_d
            variants["qwd_f32_hbm_frac"] = {"encode": round(alg / (ms_e * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                                            "decode": round(alg / (ms_d * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)}
            del wf

    # group-size sweep of the workload (the GPT-6.7B shard sweeps the gradient group 32..512 and
    # the qWD group 64..256): the same data, new header arrays; each kernel timed on its own
    group_sweep = {}
    if not args.no_group_sweep and (w.extra_groups or w.extra_qwd_groups):
        def sweep_row(h, names):
            ki = h.kernel_info()
            row = {}
            for name in names:
                ms = timed(getattr(h, name), reps=10)
                gbps = ki[name].alg_bytes / (ms * 1e-3) / 1e9
                row[name] = {"ms": ms, "alg_GBps": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4)}
            return row
        for g in sorted(set(w.extra_groups) | {w.group}):
            group_sweep[f"group_{g}"] = sweep_row(hp.with_groups(group=g), ("grad_quant", "reduce_intra",
                                                                           "reduce_inter"))
        if w.extra_qwd_groups:
            for qg in sorted(set(w.extra_qwd_groups) | {w.qwd_group}):
                group_sweep[f"qwd_group_{qg}"] = sweep_row(hp.with_groups(qwd_group=qg), ("qwd_encode", "qwd_decode"))
        torch.cuda.empty_cache()

    # the shape of the paper's Table 5 (one GPU, 8 MB .. 2048 MB of fp32 data): 8-bit group
    # quantization and single-chunk dequantization to fp32, without and with a fused 32 x 32
    # Hadamard transform (the size the paper uses), group 128; GB/s of fp32 input / output
    table5 = {}
    if not args.no_table5:
        hp = None  # the step's buffers are no longer needed
        torch.cuda.empty_cache()
        for mb in (8, 16, 64, 512, 1024, 2048):
            n = mb * (1 << 20) // 4
            x = torch.randn(n, device="cuda")
            c = torch.empty(n, dtype=torch.uint8, device="cuda")
            s = torch.empty(n // 128, device="cuda")
            y = torch.empty(n, device="cuda")
            row = {}
            for blk in (0, 32):
                t_q = timed(lambda: sdp4.sdp4_grad_quant(x, 8, blk, 128, c, s), reps=20)
                t_d = timed(lambda: sdp4.sdp4_dequant_reduce([c], [s], n, 8, 128, 0, blk, 1.0, None, None, y),
                            reps=20)
                tag = "had" if blk else "no_had"
                row[f"quant_{tag}_GBps"] = round(4 * n / (t_q * 1e-3) / 1e9, 1)
                row[f"dequant_{tag}_GBps"] = round(4 * n / (t_d * 1e-3) / 1e9, 1)
            table5[f"{mb}MB"] = row
            del x, c, s, y

    # K3 standalone on N_in = N (the workload's element count) 4-bit inputs: Q chunks of N/Q
    # elements reduced into N/Q fp32 outputs with the inverse Hadamard transform, its rate away from
    # the ramp-up and the last partial round of a launch (in the chain it gets N/P inputs)
    standalone = {}
    if not args.no_standalone:
        hp = None  # the step's buffers are no longer needed
        torch.cuda.empty_cache()
        m, g, Q = w.n // w.Q, w.group, w.Q
        gen = torch.Generator(device="cuda").manual_seed(args.seed)
        c4 = torch.randint(0, 256, (Q * m // 2,), dtype=torch.uint8, device="cuda", generator=gen)
        s4 = torch.rand(Q * m // g, device="cuda", generator=gen) * 1e-3
        out = torch.empty(m, device="cuda")
        cl = [c4[q * m // 2:(q + 1) * m // 2] for q in range(Q)]
        sl = [s4[q * m // g:(q + 1) * m // g] for q in range(Q)]
        ms = timed(lambda: sdp4.sdp4_dequant_reduce(cl, sl, m, 4, g, 0, w.hadamard_block, 1.0 / (w.P * Q), None,
                                                    None, out), reps=20)
        alg = Q * (m // 2 + 4 * (m // g)) + 4 * m
        gbps = alg / (ms * 1e-3) / 1e9
        standalone["reduce_inter"] = {"n_in": Q * m, "ms": ms, "alg_bytes": alg, "alg_GBps": round(gbps, 1),
                                      "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4)}
        if ceil:
            rd = Q * (m // 2 + 4 * (m // g))
            standalone["reduce_inter"]["vs_rw_additive"] = round(gbps / rw_additive_GBps(rd, alg - rd, ceil), 4)
        del c4, s4, out, cl, sl

    # the recorded counters hold for the named workload's own shape only
    traffic = traffic_for(dom, args.workload if w is synth.WORKLOADS[args.workload] else "custom shape")
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.describe(), "n": w.n, "hadamard_block": w.hadamard_block,
                   "group": w.group, "P": w.P, "Q": w.Q, "qwd_group": w.qwd_group,
                   "model_weights": w.prev_dtype, "gradient_bits": [8, 4]},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": dk["alg_GBps"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(dk["alg_GBps"] / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
        "kernels": kernels,
        "copy_GBps": round(copy_gbps, 1),
        "step_alg_GBps": round(sum(k.alg_bytes for k in info.values()) / (ms_step * 1e-3) / 1e9, 1),
    }
    if graph_ms is not None:
        line["graph_step"] = {"ms_per_step": round(graph_ms, 4),
                              "value": round(fp32_total / (graph_ms * 1e-3) / 1e9, 1),
                              "note": "the same step recorded once into a HIP graph and replayed, without "
                                      "per-kernel events; informational, value above is the eager step"}
    if unfused:
        line["hadamard_fusion"] = unfused
    if variants:
        line["variants"] = variants
    if table5:
        line["table5_sweep"] = table5
    if standalone:
        line["standalone"] = standalone
    if ceil:
        line["ceilings"] = ceil
    if group_sweep:
        line["group_sweep"] = group_sweep
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample ...")
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_sample_log2, args.seed)
        log("timing the CPU oracle on all cores over the whole workload ...")
        line["cpu_baseline_all_cores"] = cpu_baseline_all_cores(w, w.n, args.seed)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
