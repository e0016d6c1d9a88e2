"""The C ABI library on a host without a GPU: it loads, exports every entry
point the public header declares, and rejects invalid arguments on the
host with the documented status before anything reaches the device (these
calls never launch a kernel).

Tests that hand the library made-up device addresses carry the ``cpu_only``
marker and are skipped where a GPU is visible: there a lapse in the
library's checks would launch a kernel on unmapped memory."""
import ctypes as C
import math
import os
import re
import subprocess

import pytest

from paper_2410_15526_amd import sdp4

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sdp4.h")

OK, EINVAL, EALIGN, ERANGE = 0, 1, 2, 3
A = 0x7F0000000000          # fake, 256-byte-aligned device addresses (never dereferenced)
B = A + (1 << 32)
CC = A + (2 << 32)
D = A + (3 << 32)


def declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(sdp4_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared()
    assert "sdp4_qwd_encode" in names and "sdp4_dequant_reduce" in names
    L = sdp4.lib()
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", sdp4._LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (sdp4_\w+)", out))
    assert set(names) <= exported, set(names) - exported


def test_helpers():
    L = sdp4.lib()
    assert L.sdp4_codes_bytes(1000, 4) == 500 and L.sdp4_codes_bytes(1000, 8) == 1000
    assert L.sdp4_codes_bytes(1000, 3) == -1
    assert L.sdp4_num_groups(4096, 128) == 32 and L.sdp4_num_groups(4096, 48) == -1
    assert L.sdp4_num_groups(4096, 16) == -1 and L.sdp4_num_groups(4096, 8192) == -1
    for s in range(5):
        assert L.sdp4_status_string(s)
    assert b"gfx950" in L.sdp4_version()
    assert L.sdp4_last_hip_error() == 0


def gq(x=A, n=4096, bits=8, block=256, group=128, codes=B, scale=CC):
    return sdp4.lib().sdp4_grad_quant(x, n, bits, block, group, codes, scale, None)


@pytest.mark.cpu_only
@pytest.mark.parametrize("kw,want", [
    (dict(bits=3), EINVAL), (dict(bits=2), EINVAL), (dict(group=48), EINVAL), (dict(group=16), EINVAL),
    (dict(group=8192), EINVAL), (dict(block=3), EINVAL), (dict(block=2048), EINVAL), (dict(block=1), EINVAL),
    (dict(n=-128), EINVAL), (dict(n=100), EALIGN), (dict(n=128, block=256), EALIGN),
    (dict(n=4096 + 128, group=256, block=0), EALIGN),
    (dict(x=None), EINVAL), (dict(codes=None), EINVAL), (dict(scale=None), EINVAL),
    (dict(x=A + 4), EALIGN), (dict(codes=B + 8), EALIGN), (dict(scale=CC + 2), EALIGN),
    (dict(codes=A + 1024), EINVAL),                       # codes overlap the input
    (dict(scale=B + 100 * 16), EINVAL),                   # scales overlap the codes
    (dict(n=0), OK), (dict(n=0, x=None, codes=None, scale=None), OK),
])
def test_grad_quant_validation(kw, want):
    assert gq(**kw) == want


def enc(w_new=A, w_prev=B, dt=0, n=4096, group=128, codes=CC, scale=D, minv=D + 4096):
    return sdp4.lib().sdp4_qwd_encode(w_new, w_prev, dt, n, group, codes, scale, minv, None)


def dec(codes=A, scale=B, minv=B + 4096, n=4096, group=128, w=CC, dt=0):
    return sdp4.lib().sdp4_qwd_decode(codes, scale, minv, n, group, w, dt, None)


@pytest.mark.cpu_only
@pytest.mark.parametrize("kw,want", [
    (dict(dt=2), EINVAL), (dict(dt=-1), EINVAL), (dict(group=100), EINVAL), (dict(n=4000), EALIGN),
    (dict(w_new=None), EINVAL), (dict(minv=None), EINVAL), (dict(w_prev=B + 2), EALIGN),
    (dict(codes=CC + 4), EALIGN), (dict(minv=D + 1), EALIGN),
    (dict(codes=A + 16), EINVAL), (dict(minv=D + 16), EINVAL), (dict(scale=B + 4 * 100), EINVAL),
    (dict(n=0), OK),
])
def test_qwd_encode_validation(kw, want):
    assert enc(**kw) == want


@pytest.mark.cpu_only
@pytest.mark.parametrize("kw,want", [
    (dict(dt=7), EINVAL), (dict(group=64 + 32), EINVAL), (dict(n=4096 + 64), EALIGN), (dict(w=None), EINVAL),
    (dict(w=CC + 8), EALIGN), (dict(codes=A + 8), EALIGN), (dict(w=A + 512), EINVAL),
    (dict(scale=CC + 100, w=CC), EINVAL), (dict(n=0), OK),
])
def test_qwd_decode_validation(kw, want):
    assert dec(**kw) == want


def enc_sym(w_new=A, w_prev=B, dt=0, n=4096, group=128, codes=CC, scale=D):
    return sdp4.lib().sdp4_qwd_encode_sym(w_new, w_prev, dt, n, group, codes, scale, None)


def dec_sym(codes=A, scale=B, n=4096, group=128, w=CC, dt=0):
    return sdp4.lib().sdp4_qwd_decode_sym(codes, scale, n, group, w, dt, None)


@pytest.mark.cpu_only
@pytest.mark.parametrize("kw,want", [
    (dict(dt=2), EINVAL), (dict(group=100), EINVAL), (dict(group=8192), EINVAL), (dict(n=4000), EALIGN),
    (dict(n=-128), EINVAL), (dict(w_new=None), EINVAL), (dict(w_prev=None), EINVAL), (dict(codes=None), EINVAL),
    (dict(scale=None), EINVAL), (dict(w_prev=B + 2), EALIGN), (dict(codes=CC + 4), EALIGN),
    (dict(scale=D + 1), EALIGN), (dict(codes=A + 16), EINVAL), (dict(scale=CC + 100 * 16), EINVAL),
    (dict(scale=B + 4 * 100, dt=1), EINVAL), (dict(n=0), OK), (dict(n=0, w_new=None, codes=None), OK),
])
def test_qwd_encode_sym_validation(kw, want):
    assert enc_sym(**kw) == want


@pytest.mark.cpu_only
@pytest.mark.parametrize("kw,want", [
    (dict(dt=7), EINVAL), (dict(group=96), EINVAL), (dict(n=4096 + 64), EALIGN), (dict(w=None), EINVAL),
    (dict(codes=None), EINVAL), (dict(scale=None), EINVAL), (dict(w=CC + 8), EALIGN),
    (dict(codes=A + 8), EALIGN), (dict(scale=B + 2), EALIGN), (dict(w=A + 512), EINVAL),
    (dict(scale=CC + 100), EINVAL), (dict(n=0), OK),
])
def test_qwd_decode_sym_validation(kw, want):
    assert dec_sym(**kw) == want


def dr(P=4, codes=None, scales=None, n=4096, bits_in=8, group=128, bits_out=4, block=0, out_scale=1.0,
       oc=D, os_=D + (1 << 24), of=None, table_null=False):
    if codes is None:
        codes = [A + p * (1 << 20) for p in range(P)]
    if scales is None:
        scales = [B + p * (1 << 20) for p in range(P)]
    cp = (C.c_void_p * max(len(codes), 1))(*codes)
    sp = (C.c_void_p * max(len(scales), 1))(*scales)
    ct = None if table_null else C.cast(cp, C.c_void_p)
    st = None if table_null else C.cast(sp, C.c_void_p)
    return sdp4.lib().sdp4_dequant_reduce(P, ct, st, n, bits_in, group, bits_out, block, out_scale, oc, os_,
                                          of, None)


@pytest.mark.cpu_only
@pytest.mark.parametrize("kw,want", [
    (dict(P=0), ERANGE), (dict(P=17, codes=[A] * 17, scales=[B] * 17), ERANGE), (dict(P=-3), ERANGE),
    (dict(bits_in=2), EINVAL), (dict(bits_out=2), EINVAL), (dict(bits_out=4, block=64), EINVAL),
    (dict(out_scale=math.inf), EINVAL), (dict(out_scale=math.nan), EINVAL),
    (dict(table_null=True), EINVAL), (dict(codes=[A, 0, A + 2 * (1 << 20), A + 3 * (1 << 20)]), EINVAL),
    (dict(codes=[A, A + 8, A + 2 * (1 << 20), A + 3 * (1 << 20)]), EALIGN),
    (dict(scales=[B, B + 2, B + 8, B + 12]), EALIGN),
    (dict(oc=None), EINVAL), (dict(os_=None), EINVAL), (dict(bits_out=0, block=64, of=None), EINVAL),
    (dict(n=4096 + 64), EALIGN), (dict(bits_out=0, block=256, n=128 * 3, of=D), EALIGN),
    (dict(oc=A + 1024), EINVAL),                          # output codes overlap peer 0's codes
    (dict(os_=B + 3 * (1 << 20) + 8), EINVAL),            # output scales overlap peer 3's scales
    (dict(of=D + 256), EINVAL),                           # f32 output overlaps output codes
    (dict(of=D + 8), EALIGN),
    (dict(n=0), OK),
])
def test_dequant_reduce_validation(kw, want):
    assert dr(**kw) == want


@pytest.mark.cpu_only
def test_hadamard_reduce_copy_validation():
    L = sdp4.lib()
    assert L.sdp4_hadamard(A, B, 4096, 0, None) == EINVAL
    assert L.sdp4_hadamard(A, B, 4096, 96, None) == EINVAL
    assert L.sdp4_hadamard(A, B, 4000, 64, None) == EALIGN
    assert L.sdp4_hadamard(A, A + 64, 4096, 64, None) == EINVAL      # partial overlap
    assert L.sdp4_hadamard(A + 4, B, 4096, 64, None) == EALIGN
    assert L.sdp4_hadamard(A, B, 0, 64, None) == OK
    xs = (C.c_void_p * 2)(A, B)
    assert L.sdp4_reduce_f32(0, C.cast(xs, C.c_void_p), CC, 1024, None) == ERANGE
    assert L.sdp4_reduce_f32(17, C.cast(xs, C.c_void_p), CC, 1024, None) == ERANGE
    assert L.sdp4_reduce_f32(2, C.cast(xs, C.c_void_p), A + 16, 1024, None) == EINVAL
    assert L.sdp4_reduce_f32(2, C.cast(xs, C.c_void_p), CC + 4, 1024, None) == EALIGN
    assert L.sdp4_reduce_f32(2, None, CC, 1024, None) == EINVAL
    assert L.sdp4_copy_f32(A, A + 16, 1024, None) == EINVAL
    assert L.sdp4_copy_f32(A, None, 1024, None) == EINVAL
    assert L.sdp4_copy_f32(A, B, -1, None) == EINVAL
    assert L.sdp4_copy_f32(A, B, 0, None) == OK


@pytest.mark.cpu_only
def test_yardstick_validation():
    L = sdp4.lib()
    assert L.sdp4_read_f32(None, 4096, B, None) == EINVAL
    assert L.sdp4_read_f32(A, 4096, None, None) == EINVAL
    assert L.sdp4_read_f32(A + 4, 4096, B, None) == EALIGN
    assert L.sdp4_read_f32(A, 4096, B + 2, None) == EALIGN
    assert L.sdp4_read_f32(A, 4096, A + 64, None) == EINVAL                   # sink inside x
    assert L.sdp4_read_f32(A, -1, B, None) == EINVAL
    assert L.sdp4_read_f32(A, 0, B, None) == OK
    assert L.sdp4_fill_f32(None, 4096, 1.0, None) == EINVAL
    assert L.sdp4_fill_f32(A + 8, 4096, 1.0, None) == EALIGN
    assert L.sdp4_fill_f32(A, -5, 1.0, None) == EINVAL
    assert L.sdp4_fill_f32(A, 0, 1.0, None) == OK


@pytest.mark.cpu_only
def test_element_counts_beyond_the_limit_are_rejected():
    big = (1 << 48) + 4096
    L = sdp4.lib()
    assert gq(n=big) == EINVAL and gq(n=1 << 62) == EINVAL
    assert enc(n=big) == EINVAL and dec(n=big) == EINVAL
    assert enc_sym(n=big) == EINVAL and dec_sym(n=big) == EINVAL
    assert dr(n=big) == EINVAL
    assert L.sdp4_grad_quant_sr(A, big, 8, 256, 128, 1, 0, B, CC, None) == EINVAL
    assert L.sdp4_hadamard(A, B, big, 256, None) == EINVAL
    assert L.sdp4_copy_f32(A, B, big, None) == EINVAL
    assert L.sdp4_read_f32(A, big, B, None) == EINVAL and L.sdp4_fill_f32(A, big, 0.0, None) == EINVAL
    assert L.sdp4_codes_bytes(big, 8) == -1 and L.sdp4_num_groups(big, 128) == -1
    assert L.sdp4_codes_bytes(1 << 48, 8) == 1 << 48


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(4096)
    with pytest.raises(ValueError):
        sdp4.sdp4_grad_quant(x, 8, 256, 128, x, x)


@pytest.mark.cpu_only
def test_stochastic_rounding_entry_points_validation():
    L = sdp4.lib()
    args = lambda **k: dict(dict(x=A, n=4096, bits=8, block=256, group=128, seed=1, offset=0, codes=B, scale=CC), **k)
    call = lambda a: L.sdp4_grad_quant_sr(a["x"], a["n"], a["bits"], a["block"], a["group"], a["seed"], a["offset"],
                                          a["codes"], a["scale"], None)
    assert call(args(offset=4)) == EALIGN
    assert call(args(offset=12)) == EALIGN
    assert call(args(bits=2)) == EINVAL
    assert call(args(block=96)) == EINVAL
    assert call(args(n=0)) == OK
    assert call(args(x=None)) == EINVAL
    assert call(args(codes=A + 64)) == EINVAL
    cp = (C.c_void_p * 2)(A, A + (1 << 20))
    sp = (C.c_void_p * 2)(B, B + (1 << 20))
    dr = lambda P=2, bits_out=4, offset=0, oc=D, os_=D + (1 << 24), n=4096: L.sdp4_dequant_reduce_sr(
        P, C.cast(cp, C.c_void_p), C.cast(sp, C.c_void_p), n, 8, 128, bits_out, 7, offset, oc, os_, None, None)
    assert dr(P=0) == ERANGE and dr(P=17) == ERANGE
    assert dr(bits_out=0) == EINVAL and dr(bits_out=2) == EINVAL
    assert dr(offset=6) == EALIGN
    assert dr(oc=None) == EINVAL
    assert dr(oc=A + 32) == EINVAL
    assert dr(n=0) == OK


@pytest.mark.cpu_only
def test_header_is_c99_and_a_c_program_links(tmp_path):
    """The boundary is a C ABI: the header compiles as strict C99 and a C
    program links against the library and gets the documented statuses."""
    import shutil
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = tmp_path / "client"
    libdir = os.path.dirname(sdp4._LIB_PATH)
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "abi_c_client.c"), "-L", libdir, "-lsdp4", f"-Wl,-rpath,{libdir}",
           "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True)
    env = dict(os.environ, HIP_VISIBLE_DEVICES="", ROCR_VISIBLE_DEVICES="")   # no device to launch on
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, env=env).stdout.split("\n")
    assert out[:10] == ["1", "2", "0", "3", "1", "2", "2048", "32", "peer count out of range", "0"]


class _DevTensor:
    """Stands in for a device tensor on a machine without a GPU: an address
    and a size, nothing the library could dereference here."""
    def __init__(self, nbytes, itemsize=1, f32=False):
        import torch
        self._n, self._item = nbytes // itemsize, itemsize
        self.dtype = torch.float32 if f32 else torch.bfloat16
        self.is_cuda = True

    def numel(self):
        return self._n

    def element_size(self):
        return self._item

    def is_contiguous(self):
        return True

    def data_ptr(self):
        return 1 << 40


def _binding_calls(monkeypatch):
    """Replace the library with a recorder: a call that gets through the
    binding's checks is recorded instead of launched."""
    calls = []

    class Rec:
        def __getattr__(self, name):
            return lambda *a: calls.append(name) or 0
    monkeypatch.setattr(sdp4, "lib", lambda: Rec())
    monkeypatch.setattr(sdp4, "_stream", lambda s: None)
    return calls


def test_binding_refuses_tensors_too_small_for_the_call(monkeypatch):
    """The library sees only addresses: the binding checks that every tensor
    holds the bytes the call touches, before anything reaches the device."""
    pytest.importorskip("torch")
    calls = _binding_calls(monkeypatch)
    n, g = 1 << 12, 128
    T = _DevTensor
    ok = dict(w_new=T(4 * n, 4, True), w_prev=T(2 * n, 2), group=g, codes=T(n // 2), scale=T(4 * n // g, 4),
              minv=T(4 * n // g, 4))
    sdp4.sdp4_qwd_encode(**ok)
    for key, short in (("w_new", T(4 * n - 4, 4, True)), ("w_prev", T(2 * n - 2, 2)), ("codes", T(n // 2 - 1)),
                       ("scale", T(4 * n // g - 4, 4)), ("minv", T(4 * n // g - 4, 4))):
        with pytest.raises(ValueError, match=key):
            sdp4.sdp4_qwd_encode(**{**ok, key: short}, n=n)
    with pytest.raises(ValueError, match="w_prev"):             # float32 weights take 4 bytes each
        sdp4.sdp4_qwd_decode(T(n // 2), T(4 * n // g, 4), T(4 * n // g, 4), g, T(2 * n, 4, True), n=n)
    sdp4.sdp4_grad_quant(T(4 * n, 4, True), 8, 256, g, T(n), T(4 * n // g, 4))
    with pytest.raises(ValueError, match="codes"):
        sdp4.sdp4_grad_quant(T(4 * n, 4, True), 8, 256, g, T(n // 2), T(4 * n // g, 4))
    P, m = 4, n // 4
    cs, ss = [T(m) for _ in range(P)], [T(4 * m // g, 4) for _ in range(P)]
    sdp4.sdp4_dequant_reduce(cs, ss, m, 8, g, 4, 0, 1.0, T(m // 2), T(4 * m // g, 4), None)
    with pytest.raises(ValueError, match=r"codes\[2\]"):
        sdp4.sdp4_dequant_reduce(cs[:2] + [T(m // 2)] + cs[3:], ss, m, 8, g, 4, 0, 1.0, T(m // 2), T(4 * m // g, 4))
    with pytest.raises(ValueError, match="out_f32"):
        sdp4.sdp4_dequant_reduce(cs, ss, m, 8, g, 0, 256, 1.0, None, None, T(4 * m - 4, 4, True))
    with pytest.raises(ValueError, match="y"):
        sdp4.sdp4_copy_f32(T(4 * n, 4, True), T(2 * n, 4, True))
    with pytest.raises(ValueError, match=r"xs\[1\]"):
        sdp4.sdp4_reduce_f32([T(4 * n, 4, True), T(4 * n - 4, 4, True)], T(4 * n, 4, True))
    assert calls == ["sdp4_qwd_encode", "sdp4_grad_quant", "sdp4_dequant_reduce"]


def test_readme_c_example_compiles(tmp_path):
    """The C example in README.md uses the header's entry points with their
    documented signatures: it compiles against include/sdp4.h."""
    import re
    import shutil
    hip_inc = "/opt/rocm/include"
    if not shutil.which("g++") or not os.path.isdir(os.path.join(hip_inc, "hip")):
        pytest.skip("g++ or the HIP headers not available")
    text = open(os.path.join(ROOT, "README.md")).read()
    m = re.search(r"```c\n(.*?)```", text, re.S)
    assert m, "README.md has no C example"
    src = tmp_path / "readme_example.cpp"
    src.write_text(m.group(1))
    subprocess.run(["g++", "-std=c++17", "-fsyntax-only", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", hip_inc,
                    "-I", os.path.join(ROOT, "include"), str(src)], check=True, capture_output=True)
