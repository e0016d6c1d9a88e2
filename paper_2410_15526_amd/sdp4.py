"""ctypes binding of ``libsdp4.so`` -- argument marshalling only.

Each function has the name and argument order of the C entry point it
wraps, takes torch tensors (device memory) or raw integer device pointers
for the arrays, derives element counts and dtypes from tensors where the C
call needs them, passes torch's current HIP stream unless one is given, and
raises :class:`Sdp4Error` on a non-zero status.  No computation happens
here, and there is no fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsdp4.so")
_lock = threading.Lock()
_lib = None

OK, EINVAL, EALIGN, ERANGE, EHIP = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
MIN_GROUP, MAX_GROUP, MAX_HADAMARD, MAX_PEERS = 32, 4096, 1024, 16


class Sdp4Error(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = lib().sdp4_status_string(status).decode()
        if status == EHIP:
            msg += f" (hip error {lib().sdp4_last_hip_error()})"
        super().__init__(f"{fn}: status {status}: {msg}")


def lib() -> C.CDLL:
    """The loaded HIP library (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                raise ImportError(f"{_LIB_PATH} is missing: build it with "
                                  "`python -c 'import __graft_entry__ as g; g.build()'`")
            L = C.CDLL(_LIB_PATH)
            vp, i64, i32, f32 = C.c_void_p, C.c_int64, C.c_int, C.c_float
            sig = {
                "sdp4_qwd_encode": (i32, [vp, vp, i32, i64, i32, vp, vp, vp, vp]),
                "sdp4_qwd_decode": (i32, [vp, vp, vp, i64, i32, vp, i32, vp]),
                "sdp4_qwd_encode_sym": (i32, [vp, vp, i32, i64, i32, vp, vp, vp]),
                "sdp4_qwd_decode_sym": (i32, [vp, vp, i64, i32, vp, i32, vp]),
                "sdp4_grad_quant": (i32, [vp, i64, i32, i32, i32, vp, vp, vp]),
                "sdp4_dequant_reduce": (i32, [i32, vp, vp, i64, i32, i32, i32, i32, f32, vp, vp, vp, vp]),
                "sdp4_grad_quant_sr": (i32, [vp, i64, i32, i32, i32, C.c_uint64, C.c_uint64, vp, vp, vp]),
                "sdp4_dequant_reduce_sr": (i32, [i32, vp, vp, i64, i32, i32, i32, C.c_uint64, C.c_uint64, vp, vp,
                                                 vp, vp]),
                "sdp4_hadamard": (i32, [vp, vp, i64, i32, vp]),
                "sdp4_reduce_f32": (i32, [i32, vp, vp, i64, vp]),
                "sdp4_copy_f32": (i32, [vp, vp, i64, vp]),
                "sdp4_read_f32": (i32, [vp, i64, vp, vp]),
                "sdp4_fill_f32": (i32, [vp, i64, f32, vp]),
                "sdp4_codes_bytes": (i64, [i64, i32]),
                "sdp4_num_groups": (i64, [i64, i32]),
                "sdp4_status_string": (C.c_char_p, [i32]),
                "sdp4_version": (C.c_char_p, []),
                "sdp4_last_hip_error": (i32, []),
            }
            for name, (res, args) in sig.items():
                fn = getattr(L, name)
                fn.restype, fn.argtypes = res, args
            _lib = L
    return _lib


def _ptr(x):
    """Device address of a tensor (must live on a GPU), an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError("sdp4: arrays must be device tensors")
    if not x.is_contiguous():
        raise ValueError("sdp4: arrays must be contiguous")
    return x.data_ptr()


def _need(x, nbytes: int, what: str) -> None:
    """A tensor argument must hold every byte the call reads or writes
    through it: the library sees only its address, so a short tensor would
    be overrun on the device.  Integer addresses are the caller's to size."""
    if x is None or isinstance(x, int):
        return
    have = x.numel() * x.element_size()
    if have < nbytes:
        raise ValueError(f"sdp4: {what} holds {have} bytes; the call touches {nbytes}")


def _ng(n: int, group: int) -> int:
    """Groups in n elements; 0 for a group the library will reject itself."""
    ok = isinstance(group, int) and group > 0 and group & (group - 1) == 0
    return n // group if ok else 0


def _prev_bytes(w_prev, n: int) -> int:
    import torch
    return (4 if w_prev.dtype == torch.float32 else 2) * n


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _prev_dtype(w_prev) -> int:
    import torch
    if w_prev.dtype == torch.float32:
        return F32
    if w_prev.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return BF16
    raise ValueError(f"sdp4: model weights must be float32 or bfloat16, not {w_prev.dtype}")


def _ck(name: str, rc: int) -> None:
    if rc != OK:
        raise Sdp4Error(name, rc)


def sdp4_qwd_encode(w_new, w_prev, group, codes, scale, minv, n=None, stream=None):
    """codes/scale/minv <- 4-bit quantized (w_new - w_prev); see include/sdp4.h."""
    n = w_new.numel() if n is None else n
    _need(w_new, 4 * n, "w_new"); _need(w_prev, _prev_bytes(w_prev, n), "w_prev"); _need(codes, n // 2, "codes")
    _need(scale, 4 * _ng(n, group), "scale"); _need(minv, 4 * _ng(n, group), "minv")
    _ck("sdp4_qwd_encode", lib().sdp4_qwd_encode(_ptr(w_new), _ptr(w_prev), _prev_dtype(w_prev), n, group,
                                                 _ptr(codes), _ptr(scale), _ptr(minv), _stream(stream)))


def sdp4_qwd_decode(codes, scale, minv, group, w_prev, n=None, stream=None):
    """w_prev <- w_prev + dequantized message, in place."""
    n = w_prev.numel() if n is None else n
    _need(codes, n // 2, "codes"); _need(scale, 4 * _ng(n, group), "scale"); _need(minv, 4 * _ng(n, group), "minv")
    _need(w_prev, _prev_bytes(w_prev, n), "w_prev")
    _ck("sdp4_qwd_decode", lib().sdp4_qwd_decode(_ptr(codes), _ptr(scale), _ptr(minv), n, group,
                                                 _ptr(w_prev), _prev_dtype(w_prev), _stream(stream)))


def sdp4_qwd_encode_sym(w_new, w_prev, group, codes, scale, n=None, stream=None):
    """codes/scale <- symmetric 4-bit quantized (w_new - w_prev); see include/sdp4.h."""
    n = w_new.numel() if n is None else n
    _need(w_new, 4 * n, "w_new"); _need(w_prev, _prev_bytes(w_prev, n), "w_prev"); _need(codes, n // 2, "codes")
    _need(scale, 4 * _ng(n, group), "scale")
    _ck("sdp4_qwd_encode_sym", lib().sdp4_qwd_encode_sym(_ptr(w_new), _ptr(w_prev), _prev_dtype(w_prev), n, group,
                                                         _ptr(codes), _ptr(scale), _stream(stream)))


def sdp4_qwd_decode_sym(codes, scale, group, w_prev, n=None, stream=None):
    """w_prev <- w_prev + dequantized symmetric message, in place."""
    n = w_prev.numel() if n is None else n
    _need(codes, n // 2, "codes"); _need(scale, 4 * _ng(n, group), "scale"); _need(w_prev, _prev_bytes(w_prev, n), "w_prev")
    _ck("sdp4_qwd_decode_sym", lib().sdp4_qwd_decode_sym(_ptr(codes), _ptr(scale), n, group, _ptr(w_prev),
                                                         _prev_dtype(w_prev), _stream(stream)))


def sdp4_grad_quant(x, bits, hadamard_block, group, codes, scale, n=None, stream=None):
    n = x.numel() if n is None else n
    _need(x, 4 * n, "x"); _need(codes, n * bits // 8, "codes"); _need(scale, 4 * _ng(n, group), "scale")
    _ck("sdp4_grad_quant", lib().sdp4_grad_quant(_ptr(x), n, bits, hadamard_block, group, _ptr(codes),
                                                 _ptr(scale), _stream(stream)))


def _need_reduce(codes, scales, n_chunk, bits_in, group, bits_out, out_codes, out_scales, out_f32):
    for p, (c, sc) in enumerate(zip(codes, scales)):
        _need(c, n_chunk * bits_in // 8, f"codes[{p}]")
        _need(sc, 4 * _ng(n_chunk, group), f"scales[{p}]")
    if bits_out:
        _need(out_codes, n_chunk * bits_out // 8, "out_codes")
        _need(out_scales, 4 * _ng(n_chunk, group), "out_scales")
    _need(out_f32, 4 * n_chunk, "out_f32")


def sdp4_dequant_reduce(codes, scales, n_chunk, bits_in, group, bits_out, hadamard_block=0,
                        out_scale=1.0, out_codes=None, out_scales=None, out_f32=None, stream=None):
    """``codes``/``scales``: sequences of P chunk tensors (or addresses)."""
    P = len(codes)
    if len(scales) != P:
        raise ValueError("sdp4_dequant_reduce: codes and scales differ in length")
    _need_reduce(codes, scales, n_chunk, bits_in, group, bits_out, out_codes, out_scales, out_f32)
    cp = (C.c_void_p * max(P, 1))(*[_ptr(c) for c in codes])
    sp = (C.c_void_p * max(P, 1))(*[_ptr(s) for s in scales])
    _ck("sdp4_dequant_reduce", lib().sdp4_dequant_reduce(
        P, C.cast(cp, C.c_void_p), C.cast(sp, C.c_void_p), n_chunk, bits_in, group, bits_out,
        hadamard_block, float(out_scale), _ptr(out_codes), _ptr(out_scales), _ptr(out_f32),
        _stream(stream)))


def sdp4_grad_quant_sr(x, bits, hadamard_block, group, seed, offset, codes, scale, n=None, stream=None):
    """Stochastically rounded sdp4_grad_quant (unbiased; see include/sdp4.h)."""
    n = x.numel() if n is None else n
    _need(x, 4 * n, "x"); _need(codes, n * bits // 8, "codes"); _need(scale, 4 * _ng(n, group), "scale")
    _ck("sdp4_grad_quant_sr", lib().sdp4_grad_quant_sr(_ptr(x), n, bits, hadamard_block, group, seed, offset,
                                                       _ptr(codes), _ptr(scale), _stream(stream)))


def sdp4_dequant_reduce_sr(codes, scales, n_chunk, bits_in, group, bits_out, seed, offset, out_codes, out_scales,
                           out_f32=None, stream=None):
    P = len(codes)
    if len(scales) != P:
        raise ValueError("sdp4_dequant_reduce_sr: codes and scales differ in length")
    _need_reduce(codes, scales, n_chunk, bits_in, group, bits_out, out_codes, out_scales, out_f32)
    cp = (C.c_void_p * max(P, 1))(*[_ptr(c) for c in codes])
    sp = (C.c_void_p * max(P, 1))(*[_ptr(s) for s in scales])
    _ck("sdp4_dequant_reduce_sr", lib().sdp4_dequant_reduce_sr(
        P, C.cast(cp, C.c_void_p), C.cast(sp, C.c_void_p), n_chunk, bits_in, group, bits_out, seed, offset,
        _ptr(out_codes), _ptr(out_scales), _ptr(out_f32), _stream(stream)))


def sdp4_hadamard(x, y, block, n=None, stream=None):
    n = x.numel() if n is None else n
    _need(x, 4 * n, "x"); _need(y, 4 * n, "y")
    _ck("sdp4_hadamard", lib().sdp4_hadamard(_ptr(x), _ptr(y), n, block, _stream(stream)))


def sdp4_reduce_f32(xs, y, n=None, stream=None):
    n = y.numel() if n is None else n
    for i, x in enumerate(xs):
        _need(x, 4 * n, f"xs[{i}]")
    _need(y, 4 * n, "y")
    xp = (C.c_void_p * max(len(xs), 1))(*[_ptr(x) for x in xs])
    _ck("sdp4_reduce_f32", lib().sdp4_reduce_f32(len(xs), C.cast(xp, C.c_void_p), _ptr(y), n,
                                                 _stream(stream)))


def sdp4_copy_f32(x, y, n=None, stream=None):
    n = x.numel() if n is None else n
    _need(x, 4 * n, "x"); _need(y, 4 * n, "y")
    _ck("sdp4_copy_f32", lib().sdp4_copy_f32(_ptr(x), _ptr(y), n, _stream(stream)))


def sdp4_read_f32(x, sink, n=None, stream=None):
    """Read-only stream over x; XORs the bit patterns of x[i] into sink[i % 4]
    (sink: 4 int32 or uint32 words on the device, cleared by the caller)."""
    n = x.numel() if n is None else n
    _need(x, 4 * n, "x"); _need(sink, 16, "sink")
    _ck("sdp4_read_f32", lib().sdp4_read_f32(_ptr(x), n, _ptr(sink), _stream(stream)))


def sdp4_fill_f32(y, value, n=None, stream=None):
    n = y.numel() if n is None else n
    _need(y, 4 * n, "y")
    _ck("sdp4_fill_f32", lib().sdp4_fill_f32(_ptr(y), n, float(value), _stream(stream)))


def sdp4_codes_bytes(n, bits):
    return lib().sdp4_codes_bytes(n, bits)


def sdp4_num_groups(n, group):
    return lib().sdp4_num_groups(n, group)


def sdp4_version() -> str:
    return lib().sdp4_version().decode()
