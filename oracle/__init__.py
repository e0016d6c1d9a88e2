"""CPU oracle of the SDP4Bit compression hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
CPU-baseline leg may import this package.  The product path (the HIP
library and its binding) never imports it, and the two share no code.

The arithmetic lives in ``sdp4_oracle.c`` (plain scalar C, float32 ops in
written order, ``-ffp-contract=off``); this module only compiles it with gcc
and marshals numpy arrays.  Every function returns fresh numpy arrays.

Codes are returned *unpacked* (one int8/uint8 per element) by the
``quant_*`` helpers and *packed* (the wire format) by the composite calls
``qwd_encode``, ``grad_quant`` and ``dequant_reduce``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sdp4_oracle.c")
_LIB = os.path.join(_HERE, "_sdp4_oracle.so")
_CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
           "-Wall", "-Wextra"]
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/_sdp4_oracle.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", *_CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def lib() -> C.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            L = C.CDLL(_LIB)
            vp, i64, i32, f32 = C.c_void_p, C.c_int64, C.c_int, C.c_float
            sig = {
                "sdp4ref_bf16_to_f32": (f32, [C.c_uint16]),
                "sdp4ref_f32_to_bf16_rne": (C.c_uint16, [f32]),
                "sdp4ref_hadamard_scale": (f32, [i32]),
                "sdp4ref_fwht": (i32, [vp, i64, i32]),
                "sdp4ref_quant_sym": (i32, [vp, i64, i32, i32, vp, vp, vp]),
                "sdp4ref_dequant_sym": (i32, [vp, vp, i64, i32, vp]),
                "sdp4ref_quant_asym4": (i32, [vp, i64, i32, vp, vp, vp, vp]),
                "sdp4ref_dequant_asym4": (i32, [vp, vp, vp, i64, i32, vp]),
                "sdp4ref_pack4": (i32, [vp, i64, vp]),
                "sdp4ref_unpack4": (i32, [vp, i64, i32, vp]),
                "sdp4ref_qwd_encode": (i32, [vp, vp, i32, i64, i32, vp, vp, vp, vp]),
                "sdp4ref_qwd_decode": (i32, [vp, vp, vp, i64, i32, vp, i32]),
                "sdp4ref_qwd_encode_sym": (i32, [vp, vp, i32, i64, i32, vp, vp, vp]),
                "sdp4ref_qwd_decode_sym": (i32, [vp, vp, i64, i32, vp, i32]),
                "sdp4ref_grad_quant": (i32, [vp, i64, i32, i32, i32, vp, vp, vp]),
                "sdp4ref_dequant_reduce": (i32, [i32, vp, vp, i64, i32, i32, i32, i32, f32,
                                                 vp, vp, vp, vp]),
                "sdp4ref_hadamard": (i32, [vp, vp, i64, i32]),
                "sdp4ref_reduce_f32": (i32, [i32, vp, vp, i64]),
                "sdp4ref_version": (C.c_char_p, []),
                "sdp4ref_philox4x32_10": (None, [vp, vp, vp]),
                "sdp4ref_sr_uniform": (f32, [C.c_uint64, C.c_uint64]),
                "sdp4ref_quant_sym_sr": (i32, [vp, i64, i32, i32, C.c_uint64, C.c_uint64, vp, vp, vp]),
                "sdp4ref_grad_quant_sr": (i32, [vp, i64, i32, i32, i32, C.c_uint64, C.c_uint64, vp, vp, vp]),
                "sdp4ref_dequant_reduce_sr": (i32, [i32, vp, vp, i64, i32, i32, i32, C.c_uint64, C.c_uint64,
                                                    vp, vp, vp, vp]),
            }
            for name, (res, args) in sig.items():
                fn = getattr(L, name)
                fn.restype, fn.argtypes = res, args
            _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _ck(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what}: oracle status {rc}")


def _f32(x) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float32)


def _p(a: np.ndarray | None):
    return None if a is None else a.ctypes.data


# --------------------------------------------------------------------------
# scalar helpers
# --------------------------------------------------------------------------

def hadamard_scale(block: int) -> np.float32:
    return np.float32(lib().sdp4ref_hadamard_scale(block))


def bf16_rne(x) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (element by element)."""
    f = lib().sdp4ref_f32_to_bf16_rne
    x = _f32(x).ravel()
    return np.fromiter((f(float(v)) for v in x), dtype=np.uint16, count=x.size)


def bf16_to_f32(b) -> np.ndarray:
    f = lib().sdp4ref_bf16_to_f32
    b = np.ascontiguousarray(b, np.uint16).ravel()
    return np.fromiter((f(int(v)) for v in b), dtype=np.float32, count=b.size)


# --------------------------------------------------------------------------
# building blocks
# --------------------------------------------------------------------------

def fwht(x, block: int) -> np.ndarray:
    y = _f32(x).copy()
    _ck(lib().sdp4ref_fwht(_p(y), y.size, block), "fwht")
    return y


def quant_sym(x, group: int, bits: int):
    """-> (codes int8[n], scale f32[n/group], pre f32[n])"""
    x = _f32(x)
    q = np.empty(x.size, np.int8)
    s = np.empty(x.size // group, np.float32)
    pre = np.empty(x.size, np.float32)
    _ck(lib().sdp4ref_quant_sym(_p(x), x.size, group, bits, _p(q), _p(s), _p(pre)), "quant_sym")
    return q, s, pre


def dequant_sym(q, scale, group: int) -> np.ndarray:
    q = np.ascontiguousarray(q, np.int8)
    s = _f32(scale)
    out = np.empty(q.size, np.float32)
    _ck(lib().sdp4ref_dequant_sym(_p(q), _p(s), q.size, group, _p(out)), "dequant_sym")
    return out


def quant_asym4(x, group: int):
    """-> (codes uint8[n] in 0..15, scale f32[n/group], minv f32[n/group], pre f32[n])"""
    x = _f32(x)
    q = np.empty(x.size, np.uint8)
    s = np.empty(x.size // group, np.float32)
    m = np.empty(x.size // group, np.float32)
    pre = np.empty(x.size, np.float32)
    _ck(lib().sdp4ref_quant_asym4(_p(x), x.size, group, _p(q), _p(s), _p(m), _p(pre)), "quant_asym4")
    return q, s, m, pre


def dequant_asym4(q, scale, minv, group: int) -> np.ndarray:
    q = np.ascontiguousarray(q, np.uint8)
    s, m = _f32(scale), _f32(minv)
    out = np.empty(q.size, np.float32)
    _ck(lib().sdp4ref_dequant_asym4(_p(q), _p(s), _p(m), q.size, group, _p(out)), "dequant_asym4")
    return out


def pack4(codes) -> np.ndarray:
    c = np.ascontiguousarray(codes).view(np.int8) if np.asarray(codes).dtype.itemsize == 1 else \
        np.ascontiguousarray(codes, np.int8)
    out = np.empty(c.size // 2, np.uint8)
    _ck(lib().sdp4ref_pack4(_p(c), c.size, _p(out)), "pack4")
    return out


def unpack4(packed, n: int, signed: bool) -> np.ndarray:
    b = np.ascontiguousarray(packed, np.uint8)
    out = np.empty(n, np.int8)
    _ck(lib().sdp4ref_unpack4(_p(b), n, int(signed), _p(out)), "unpack4")
    return out


# --------------------------------------------------------------------------
# the hot-path operations (same meaning as the C ABI of the HIP library)
# --------------------------------------------------------------------------

def qwd_encode(w_new, w_prev, group: int):
    """-> (codes u8[n/2], scale f32[n/g], minv f32[n/g], pre f32[n]).

    ``w_prev`` is float32, or uint16 holding bfloat16 bit patterns.
    """
    w_new = _f32(w_new)
    w_prev = np.ascontiguousarray(w_prev)
    is_bf16 = int(w_prev.dtype == np.uint16)
    if not is_bf16:
        w_prev = _f32(w_prev)
    n = w_new.size
    codes = np.empty(n // 2, np.uint8)
    s = np.empty(n // group, np.float32)
    m = np.empty(n // group, np.float32)
    pre = np.empty(n, np.float32)
    _ck(lib().sdp4ref_qwd_encode(_p(w_new), _p(w_prev), is_bf16, n, group, _p(codes), _p(s), _p(m),
                                 _p(pre)), "qwd_encode")
    return codes, s, m, pre


def qwd_decode(codes, scale, minv, w_prev, group: int) -> np.ndarray:
    """Returns the updated model weights (same dtype as ``w_prev``)."""
    w = np.array(w_prev, copy=True)
    is_bf16 = int(w.dtype == np.uint16)
    if not is_bf16:
        w = _f32(w).copy()
    codes = np.ascontiguousarray(codes, np.uint8)
    s, m = _f32(scale), _f32(minv)
    _ck(lib().sdp4ref_qwd_decode(_p(codes), _p(s), _p(m), w.size, group, _p(w), is_bf16),
        "qwd_decode")
    return w


def qwd_encode_sym(w_new, w_prev, group: int):
    """Symmetric 4-bit qWD -> (codes u8[n/2] signed nibbles, scale f32[n/g], pre f32[n])."""
    w_new = _f32(w_new)
    w_prev = np.ascontiguousarray(w_prev)
    is_bf16 = int(w_prev.dtype == np.uint16)
    if not is_bf16:
        w_prev = _f32(w_prev)
    n = w_new.size
    codes = np.empty(n // 2, np.uint8)
    s = np.empty(n // group, np.float32)
    pre = np.empty(n, np.float32)
    _ck(lib().sdp4ref_qwd_encode_sym(_p(w_new), _p(w_prev), is_bf16, n, group, _p(codes), _p(s), _p(pre)),
        "qwd_encode_sym")
    return codes, s, pre


def qwd_decode_sym(codes, scale, w_prev, group: int) -> np.ndarray:
    """Returns the updated model weights (same dtype as ``w_prev``)."""
    w = np.array(w_prev, copy=True)
    is_bf16 = int(w.dtype == np.uint16)
    if not is_bf16:
        w = _f32(w).copy()
    codes = np.ascontiguousarray(codes, np.uint8)
    s = _f32(scale)
    _ck(lib().sdp4ref_qwd_decode_sym(_p(codes), _p(s), w.size, group, _p(w), is_bf16), "qwd_decode_sym")
    return w


def grad_quant(x, bits: int, hadamard_block: int, group: int):
    """-> (codes: int8[n] for 8 bits or u8[n/2] packed for 4, scale f32[n/g], pre f32[n])"""
    x = _f32(x)
    n = x.size
    codes = np.empty(n, np.int8) if bits == 8 else np.empty(n // 2, np.uint8)
    s = np.empty(n // group, np.float32)
    pre = np.empty(n, np.float32)
    _ck(lib().sdp4ref_grad_quant(_p(x), n, bits, hadamard_block, group, _p(codes), _p(s), _p(pre)),
        "grad_quant")
    return codes, s, pre


def dequant_reduce(codes_list, scales_list, n_chunk: int, bits_in: int, group: int, bits_out: int,
                   hadamard_block: int = 0, out_scale: float = 1.0, want_f32: bool = True):
    """-> dict(codes, scales, f32, pre) with the entries this mode produces."""
    P = len(codes_list)
    cl = [np.ascontiguousarray(c) for c in codes_list]
    sl = [_f32(s) for s in scales_list]
    cptr = (C.c_void_p * P)(*[c.ctypes.data for c in cl])
    sptr = (C.c_void_p * P)(*[s.ctypes.data for s in sl])
    out = {}
    oc = os_ = pre = None
    if bits_out:
        oc = np.empty(n_chunk, np.int8) if bits_out == 8 else np.empty(n_chunk // 2, np.uint8)
        os_ = np.empty(n_chunk // group, np.float32)
        pre = np.empty(n_chunk, np.float32)
    f = np.empty(n_chunk, np.float32) if (want_f32 or not bits_out) else None
    _ck(lib().sdp4ref_dequant_reduce(P, C.cast(cptr, C.c_void_p), C.cast(sptr, C.c_void_p), n_chunk,
                                     bits_in, group, bits_out, hadamard_block, float(out_scale),
                                     _p(oc), _p(os_), _p(f), _p(pre)), "dequant_reduce")
    out.update(codes=oc, scales=os_, f32=f, pre=pre)
    return out


def hadamard(x, block: int) -> np.ndarray:
    x = _f32(x)
    y = np.empty_like(x)
    _ck(lib().sdp4ref_hadamard(_p(x), _p(y), x.size, block), "hadamard")
    return y


def reduce_f32(xs) -> np.ndarray:
    xs = [_f32(x) for x in xs]
    n = xs[0].size
    ptr = (C.c_void_p * len(xs))(*[x.ctypes.data for x in xs])
    y = np.empty(n, np.float32)
    _ck(lib().sdp4ref_reduce_f32(len(xs), C.cast(ptr, C.c_void_p), _p(y), n), "reduce_f32")
    return y


# --------------------------------------------------------------------------
# stochastic rounding (counter-based Philox4x32-10 random numbers)
# --------------------------------------------------------------------------

def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    out = np.empty(4, np.uint32)
    lib().sdp4ref_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def sr_uniform(seed: int, e: int) -> float:
    return float(lib().sdp4ref_sr_uniform(seed, e))


def quant_sym_sr(x, group: int, bits: int, seed: int, offset: int = 0):
    x = _f32(x)
    q = np.empty(x.size, np.int8)
    s = np.empty(x.size // group, np.float32)
    pre = np.empty(x.size, np.float32)
    _ck(lib().sdp4ref_quant_sym_sr(_p(x), x.size, group, bits, seed, offset, _p(q), _p(s), _p(pre)),
        "quant_sym_sr")
    return q, s, pre


def grad_quant_sr(x, bits: int, hadamard_block: int, group: int, seed: int, offset: int = 0):
    x = _f32(x)
    n = x.size
    codes = np.empty(n, np.int8) if bits == 8 else np.empty(n // 2, np.uint8)
    s = np.empty(n // group, np.float32)
    pre = np.empty(n, np.float32)
    _ck(lib().sdp4ref_grad_quant_sr(_p(x), n, bits, hadamard_block, group, seed, offset, _p(codes), _p(s),
                                    _p(pre)), "grad_quant_sr")
    return codes, s, pre


def dequant_reduce_sr(codes_list, scales_list, n_chunk: int, bits_in: int, group: int, bits_out: int,
                      seed: int, offset: int = 0, want_f32: bool = True):
    P = len(codes_list)
    cl = [np.ascontiguousarray(c) for c in codes_list]
    sl = [_f32(s) for s in scales_list]
    cptr = (C.c_void_p * P)(*[c.ctypes.data for c in cl])
    sptr = (C.c_void_p * P)(*[s.ctypes.data for s in sl])
    oc = np.empty(n_chunk, np.int8) if bits_out == 8 else np.empty(n_chunk // 2, np.uint8)
    os_ = np.empty(n_chunk // group, np.float32)
    pre = np.empty(n_chunk, np.float32)
    f = np.empty(n_chunk, np.float32) if want_f32 else None
    _ck(lib().sdp4ref_dequant_reduce_sr(P, C.cast(cptr, C.c_void_p), C.cast(sptr, C.c_void_p), n_chunk, bits_in,
                                        group, bits_out, seed, offset, _p(oc), _p(os_), _p(f), _p(pre)),
        "dequant_reduce_sr")
    return dict(codes=oc, scales=os_, f32=f, pre=pre)
