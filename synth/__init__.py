"""Seeded synthetic inputs shaped like the paper's GPT-scale workloads.

This module only draws random numbers and lays them out. It holds none of
the compression method's arithmetic (no quantizer, no transform, no
reduction), so that the CPU oracle and the HIP path can both be fed from it
without sharing any of the computation they are checked on.

Reproducibility model
---------------------
Every random stream is cut into fixed chunks of ``CHUNK`` elements.  Chunk
``c`` of stream ``s`` of workload ``w`` under seed ``seed`` is drawn from
``numpy.random.Generator(PCG64(SeedSequence([seed, w, s, c])))`` and always
draws the whole chunk, so the value at element ``i`` never depends on which
range was requested.  Any sample of a multi-GB shard can therefore be
regenerated on the host from its element range alone.

Stream ids: 0 previous/model weights, 1 weight difference, 2 local
gradient, 3 per-layer layout (sigma and outlier channels), 4 outlier
positions for the uniform-outlier recipe, 100+p gradient of synthetic peer p.

Workloads (sizes and hidden widths follow the paper's GPT model table in
Appendix C; distributions stand in for the Pile-trained weights and
gradients the paper measures on, which are not available):

* ``c1`` tiny shard: 1,048,576 elements.
* ``c2`` 125M-parameter GPT shard: 125,829,120 elements.
* ``c3`` GPT-1.3B, one GPU's 1/8 shard: 167,772,160 elements (h = 2048).
* ``c4`` GPT-6.7B, one GPU's 1/8 shard: 838,860,800 elements (h = 4096).
* ``c5`` GPT-13B, one GPU's 1/8 shard: 1,625,292,800 elements (h = 5120).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

CHUNK = 1 << 20

STREAM_PREV = 0
STREAM_DIFF = 1
STREAM_GRAD = 2
STREAM_LAYOUT = 3
STREAM_OUTLIER_POS = 4
STREAM_PEER0 = 100


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _rng(seed: int, wid: int, stream: int, chunk: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wid, stream, chunk])))


def _chunked(fill_chunk, start: int, count: int, dtype) -> np.ndarray:
    """Evaluate ``fill_chunk(c) -> array[CHUNK]`` over the chunks covering a range."""
    out = np.empty(count, dtype=dtype)
    if count == 0:
        return out
    c_lo = start // CHUNK
    c_hi = (start + count - 1) // CHUNK

    def work(c: int) -> None:
        vals = fill_chunk(c)
        lo = max(start, c * CHUNK)
        hi = min(start + count, (c + 1) * CHUNK)
        out[lo - start:hi - start] = vals[lo - c * CHUNK:hi - c * CHUNK]

    chunks = range(c_lo, c_hi + 1)
    if len(chunks) == 1:
        work(c_lo)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, chunks))
    return out


def standard_normal(seed: int, wid: int, stream: int, start: int, count: int) -> np.ndarray:
    """float32 N(0, 1) draws for elements ``[start, start + count)`` of a stream."""
    return _chunked(lambda c: _rng(seed, wid, stream, c).standard_normal(CHUNK, dtype=np.float32),
                    start, count, np.float32)


def student_t3_unit(seed: int, wid: int, stream: int, start: int, count: int) -> np.ndarray:
    """float32 Student-t draws with 3 degrees of freedom, rescaled to unit variance.

    t3 = Z / sqrt(V / 3) with V ~ chi^2(3) = 2 Gamma(3/2); t3 has variance 3,
    so t3 / sqrt(3) = Z / sqrt(2 Gamma(3/2)).
    """
    def chunk(c: int) -> np.ndarray:
        r = _rng(seed, wid, stream, c)
        z = r.standard_normal(CHUNK, dtype=np.float32)
        g = r.standard_gamma(1.5, CHUNK, dtype=np.float32)
        np.maximum(g, np.float32(1e-30), out=g)
        return z / np.sqrt(np.float32(2.0) * g)
    return _chunked(chunk, start, count, np.float32)


def bf16_bits_toward_zero(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns obtained by dropping the low 16 bits of float32 ``x``.

    Used only to *draw* bfloat16 model weights with a given distribution; the
    method's own float->bfloat16 narrowing (round to nearest even) is not
    this operation and lives in the oracle and the kernels separately.
    """
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact float32 value of bfloat16 bit patterns (a bit shift, no rounding)."""
    return (np.ascontiguousarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Workload:
    """One synthetic shard recipe.

    ``grad_kind`` is ``"uniform_outliers"`` (N(0, grad_sigma^2) with a
    fraction ``outlier_frac`` of positions, chosen uniformly per chunk,
    multiplied by ``outlier_mult``) or ``"layered"`` (consecutive layers of
    12 h^2 elements, per-layer sigma log-uniform in [1e-6, 1e-3], and in each
    layer round(0.005 h) hidden channels whose elements are multiplied by
    ``outlier_mult``).
    """
    wid: int
    name: str
    n: int
    hidden: int
    grad_kind: str
    hadamard_block: int
    group: int
    P: int
    Q: int
    qwd_group: int
    prev_dtype: str  # "f32" or "bf16"
    diff_kind: str  # "normal" or "t3"
    diff_sigma: float
    weight_sigma: float = 0.02
    grad_sigma: float = 1e-4
    outlier_frac: float = 1e-3
    outlier_mult: float = 100.0
    extra_groups: tuple = field(default=())
    extra_qwd_groups: tuple = field(default=())

    @property
    def layer_elems(self) -> int:
        return 12 * self.hidden * self.hidden

    def describe(self) -> str:
        return (f"{self.name}: N={self.n:,} elements, Hadamard block {self.hadamard_block}, group "
                f"{self.group}, 8-bit x P={self.P} then 4-bit x Q={self.Q}; qWD group "
                f"{self.qwd_group}, {self.prev_dtype} model weights")


WORKLOADS = {
    "c1": Workload(1, "tiny shard", 1 << 20, 768, "uniform_outliers", 64, 128, 4, 4, 128,
                   "f32", "normal", 1e-3),
    "c2": Workload(2, "GPT-125M shard", 125_829_120, 768, "uniform_outliers", 128, 128, 8, 2, 128,
                   "f32", "t3", 5e-4),
    "c3": Workload(3, "GPT-1.3B 1/8 shard", 167_772_160, 2048, "layered", 256, 128, 8, 4, 128,
                   "f32", "t3", 5e-4, outlier_mult=50.0, extra_groups=(256,)),
    "c4": Workload(4, "GPT-6.7B 1/8 shard", 838_860_800, 4096, "layered", 128, 128, 8, 4, 128,
                   "bf16", "t3", 5e-4, outlier_mult=50.0,
                   extra_groups=(32, 64, 256, 512), extra_qwd_groups=(64, 256)),
    "c5": Workload(5, "GPT-13B 1/8 shard", 1_625_292_800, 5120, "layered", 256, 128, 8, 4, 128,
                   "bf16", "t3", 5e-4, outlier_mult=50.0),
}


def scaled(w: Workload, n: int) -> Workload:
    """The same recipe at a smaller element count (for tests that must run fast)."""
    from dataclasses import replace
    return replace(w, n=n)


# ----------------------------------------------------------------------------
# weights (qWD inputs)
# ----------------------------------------------------------------------------

def _prev_chunk(w: Workload, seed: int, c: int) -> np.ndarray:
    x = _rng(seed, w.wid, STREAM_PREV, c).standard_normal(CHUNK, dtype=np.float32)
    x *= np.float32(w.weight_sigma)
    return bf16_bits_toward_zero(x) if w.prev_dtype == "bf16" else x


def _diff_chunk(w: Workload, seed: int, c: int) -> np.ndarray:
    r = _rng(seed, w.wid, STREAM_DIFF, c)
    z = r.standard_normal(CHUNK, dtype=np.float32)
    if w.diff_kind != "normal":
        # Student-t(3) rescaled to unit variance: Z / sqrt(2 Gamma(3/2))
        g = r.standard_gamma(1.5, CHUNK, dtype=np.float32)
        np.maximum(g, np.float32(1e-30), out=g)
        g *= np.float32(2.0)
        np.sqrt(g, out=g)
        z /= g
    z *= np.float32(w.diff_sigma)
    return z


def prev_weights(w: Workload, start: int, count: int, seed: int = 0) -> np.ndarray:
    """Previously communicated model weights: float32, or bfloat16 bits (uint16)."""
    dt = np.uint16 if w.prev_dtype == "bf16" else np.float32
    return _chunked(lambda c: _prev_chunk(w, seed, c), start, count, dt)


def weight_diff(w: Workload, start: int, count: int, seed: int = 0) -> np.ndarray:
    return _chunked(lambda c: _diff_chunk(w, seed, c), start, count, np.float32)


def new_weights(w: Workload, start: int, count: int, seed: int = 0, prev: np.ndarray | None = None) -> np.ndarray:
    """fp32 main weights = previous weights (widened) + a synthetic update."""
    def chunk(c: int) -> np.ndarray:
        p = _prev_chunk(w, seed, c)
        base = bf16_bits_to_f32(p) if w.prev_dtype == "bf16" else p
        return base + _diff_chunk(w, seed, c)
    return _chunked(chunk, start, count, np.float32)


# ----------------------------------------------------------------------------
# gradients (two-level path inputs)
# ----------------------------------------------------------------------------

_LAYOUT_CACHE: dict = {}


def _layer_layout(w: Workload, seed: int):
    """Per-layer sigma and outlier channel ids, drawn once per workload."""
    key = (w.wid, w.n, w.hidden, seed)
    if key not in _LAYOUT_CACHE:
        n_layers = -(-w.n // w.layer_elems)
        r = _rng(seed, w.wid, STREAM_LAYOUT, 0)
        sig = np.power(10.0, r.uniform(-6.0, -3.0, size=n_layers)).astype(np.float32)
        k = int(round(0.005 * w.hidden))
        chans = [np.sort(r.choice(w.hidden, size=k, replace=False)) for _ in range(n_layers)]
        _LAYOUT_CACHE[key] = (sig, chans)
    return _LAYOUT_CACHE[key]


def _gradient_chunk(w: Workload, seed: int, stream: int, c: int) -> np.ndarray:
    z = _rng(seed, w.wid, stream, c).standard_normal(CHUNK, dtype=np.float32)
    if w.grad_kind == "uniform_outliers":
        z *= np.float32(w.grad_sigma)
        k = int(round(w.outlier_frac * CHUNK))
        pos = _rng(seed, w.wid, STREAM_OUTLIER_POS, c).choice(CHUNK, size=k, replace=False)
        z[pos] *= np.float32(w.outlier_mult)
        return z
    sig, chans = _layer_layout(w, seed)
    n_layers = len(sig)
    lo = c * CHUNK
    while lo < (c + 1) * CHUNK:                      # a chunk spans at most a few layers
        layer = min(lo // w.layer_elems, n_layers - 1)
        end = min((c + 1) * CHUNK, (layer + 1) * w.layer_elems if layer < n_layers - 1 else (c + 1) * CHUNK)
        seg = z[lo - c * CHUNK:end - c * CHUNK]
        seg *= sig[layer]
        mask = np.zeros(w.hidden, dtype=bool)
        mask[chans[layer]] = True
        off = (lo - layer * w.layer_elems) % w.hidden
        seg[np.resize(np.roll(mask, -off), seg.size)] *= np.float32(w.outlier_mult)
        lo = end
    return z


def gradient(w: Workload, start: int, count: int, seed: int = 0, peer: int | None = None) -> np.ndarray:
    """fp32 gradient values of the local GPU (peer=None) or of synthetic peer ``peer``.

    Peers share the per-element structure (layer sigmas, outlier channels or
    outlier positions) and differ only in the underlying normal draws.
    """
    stream = STREAM_GRAD if peer is None else STREAM_PEER0 + peer
    return _chunked(lambda c: _gradient_chunk(w, seed, stream, c), start, count, np.float32)
