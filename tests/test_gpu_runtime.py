"""The library inside a real runtime: launches recorded into a HIP graph and
replayed, and independent work on concurrent streams.

Each graph replay is compared with the eager result, with eager work and
synchronizations between replays.  The kernels use no memset and keep no
device state, so every replay must reproduce the eager bytes exactly.
"""
import numpy as np
import pytest

import synth
from paper_2410_15526_amd import sdp4
from paper_2410_15526_amd.pipeline import HotPath
from tests._gpu import fill, host, say, torch

pytestmark = pytest.mark.gpu


def make_path(name="c1", n=None, seed=0):
    w = synth.WORKLOADS[name] if n is None else synth.scaled(synth.WORKLOADS[name], n)
    hp = HotPath(w.n, w.group, w.hadamard_block, w.P, w.Q, w.qwd_group, w.prev_dtype)
    fill(hp.w_prev, lambda s, k: synth.prev_weights(w, s, k, seed), w.n)
    fill(hp.w_new, lambda s, k: synth.new_weights(w, s, k, seed), w.n)
    fill(hp.grad, lambda s, k: synth.gradient(w, s, k, seed), w.n)
    torch().cuda.synchronize()
    return hp


def outputs(hp):
    return [host(t).copy() for t in (hp.qcodes, hp.qscale, hp.qmin, hp.w_prev, hp.c8, hp.s8, hp.c4, hp.s4, hp.out)]


@pytest.mark.parametrize("name,n", [("c1", None), ("c5", 1 << 26)])
def test_step_replayed_from_a_hip_graph(name, n):
    """c1: the tiny shard (streaming kernels).  c5 scaled to 2^26 elements:
    bfloat16 model weights and groups of 128, so the encoder runs in its
    clock-phased mode (launches of at least 2^26 elements), whose period the
    host computes from the device's wall-clock rate at capture time."""
    t = torch()
    say(f"graph capture of one step: {name} n={n}")
    hp = make_path(name, n)
    prev0 = hp.w_prev.clone()
    hp.step()                                   # eager step (also warms the launch caches)
    t.cuda.synchronize()
    want = outputs(hp)

    g = t.cuda.CUDAGraph()
    s = t.cuda.Stream()
    s.wait_stream(t.cuda.current_stream())
    with t.cuda.stream(s):
        hp.w_prev.copy_(prev0)
        with t.cuda.graph(g, stream=s):
            hp.step()
    t.cuda.current_stream().wait_stream(s)
    t.cuda.synchronize()
    junk = t.randn(1 << 20, device="cuda")
    for r in range(4):
        hp.w_prev.copy_(prev0)                  # decode updates the model weights in place
        for buf in (hp.qcodes, hp.c8, hp.c4):
            buf.fill_(0xA5)
        for buf in (hp.qscale, hp.qmin, hp.s8, hp.s4, hp.out):
            buf.fill_(-1.0)
        t.cuda.synchronize()
        g.replay()
        junk.mul_(1.0001)                       # eager work between replays
        t.cuda.synchronize()
        got = outputs(hp)
        for a, b in zip(got, want):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"replay {r}"


def test_concurrent_streams_do_not_interfere():
    t = torch()
    say("two streams")
    n, group, block = 1 << 22, 128, 256
    xs = [t.randn(n, device="cuda") * (10.0 ** -k) for k in range(2)]
    ref = []
    for x in xs:
        c, s = t.empty(n, dtype=t.uint8, device="cuda"), t.empty(n // group, device="cuda")
        sdp4.sdp4_grad_quant(x, 8, block, group, c, s)
        ref.append((c, s))
    t.cuda.synchronize()
    streams = [t.cuda.Stream(), t.cuda.Stream()]
    outs = [(t.empty(n, dtype=t.uint8, device="cuda"), t.empty(n // group, device="cuda")) for _ in xs]
    for _ in range(3):
        for x, st, (c, s) in zip(xs, streams, outs):
            st.wait_stream(t.cuda.current_stream())
            with t.cuda.stream(st):
                sdp4.sdp4_grad_quant(x, 8, block, group, c, s, stream=st)
        for st in streams:
            t.cuda.current_stream().wait_stream(st)
    t.cuda.synchronize()
    for (c, s), (rc, rs) in zip(outs, ref):
        assert t.equal(c, rc) and t.equal(s, rs)
