"""Device-buffer helpers and the parity rules for the GPU tests.

Parity bar (from the build's target): packed codes bit-exact, except
elements whose oracle pre-round value lies within one ulp of a rounding
boundary (k + 1/2), and those may be at most 1e-6 of the elements; headers
within 1e-6 relative; float32 results within 1e-5 relative L2.  The kernels
are designed to follow the oracle's operation order exactly, so the helpers
additionally require bit-exact headers and float results (``exact=True``),
which is stricter than the bar.
"""
from __future__ import annotations

import sys

import numpy as np

import oracle


def torch():
    import torch as _t
    return _t


def dev(a: np.ndarray):
    """numpy -> device tensor (uint16 arrays are bfloat16 bit patterns)."""
    t = torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return t.from_numpy(a.view(np.int16)).cuda().view(t.bfloat16)
    return t.from_numpy(a).cuda()


def host(t) -> np.ndarray:
    tt = torch()
    if t.dtype == tt.bfloat16:
        return t.view(tt.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def empty(n: int, dtype: str):
    t = torch()
    dt = {"u8": t.uint8, "i8": t.int8, "f32": t.float32, "bf16": t.bfloat16}[dtype]
    return t.empty(max(n, 0), dtype=dt, device="cuda")


def say(*a):
    """Name the case on stdout (flushed) before GPU work, so a failing run says which."""
    print(*a, flush=True)
    sys.stdout.flush()


def _unpack(b: np.ndarray, n: int, bits: int, signed: bool) -> np.ndarray:
    if bits == 8:
        return np.ascontiguousarray(b).view(np.int8).astype(np.int32)
    return oracle.unpack4(b, n, signed).astype(np.int32)


def check_codes(got, want, pre, n: int, bits: int, signed: bool = True, what: str = "codes"):
    """Bit-exact packed codes, with the near-tie exemption of the parity bar."""
    g = np.ascontiguousarray(got).view(np.uint8)
    w = np.ascontiguousarray(want).view(np.uint8)
    assert g.shape == w.shape, (what, g.shape, w.shape)
    if np.array_equal(g, w):
        return 0
    gu, wu = _unpack(g, n, bits, signed), _unpack(w, n, bits, signed)
    bad = np.nonzero(gu != wu)[0]
    v = pre[bad].astype(np.float32)
    frac = np.abs(v - (np.floor(v) + np.float32(0.5)))
    near = frac <= np.spacing(np.abs(v)).astype(np.float32)
    assert np.all(np.abs(gu[bad] - wu[bad]) == 1), (what, "codes differ by more than one level", bad[:10])
    assert np.all(near), (what, "mismatch away from a rounding boundary", bad[~near][:10], v[~near][:10])
    assert bad.size <= 1e-6 * n, (what, "too many boundary mismatches", bad.size, n)
    return int(bad.size)


def check_headers(got, want, what: str = "scales", exact: bool = True):
    got = np.asarray(got, np.float32)
    want = np.asarray(want, np.float32)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    rel = np.abs(got.astype(np.float64) - want) / np.maximum(np.abs(want.astype(np.float64)), 1e-300)
    assert np.all((got == want) | (rel <= 1e-6)), (what, np.nonzero(rel > 1e-6)[0][:10])
    if exact:
        bad = np.nonzero(got != want)[0]                   # +0 == -0 here: headers compare numerically
        assert bad.size == 0, (what, "not bit-exact", bad[:10], got[bad[:10]], want[bad[:10]])


def check_f32(got, want, what: str = "f32", exact: bool = True):
    got = np.asarray(got, np.float32)
    want = np.asarray(want, np.float32)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.all(np.isfinite(got)), (what, "non-finite output")
    den = np.linalg.norm(want.astype(np.float64))
    err = np.linalg.norm(got.astype(np.float64) - want)
    assert err <= 1e-5 * den or err == 0, (what, "relative L2", err / max(den, 1e-300))
    if exact:
        bad = np.nonzero(got.view(np.uint32) != want.view(np.uint32))[0]
        assert bad.size == 0, (what, "not bit-exact", bad[:10], got[bad[:10]], want[bad[:10]])


def fill(dst, gen, n, slab=1 << 26):
    """Generate host data slab by slab (gen(start, count)) and copy it into a device tensor."""
    t = torch()
    for s in range(0, n, slab):
        k = min(slab, n - s)
        a = np.ascontiguousarray(gen(s, k))
        if a.dtype == np.uint16:
            dst[s:s + k].view(t.int16).copy_(t.from_numpy(a.view(np.int16)))
        else:
            dst[s:s + k].copy_(t.from_numpy(a))
