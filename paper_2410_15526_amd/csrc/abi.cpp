// abi.cpp -- the C ABI declared in include/sdp4.h: host-side argument
// checks, then one kernel launch per call on the caller's stream.
//
// Every check runs before any HIP call, so invalid arguments are reported
// without touching the device (and without a device being present).
#include "sdp4.h"
#include "launch.hpp"

#include <cmath>
#include <cstddef>
#include <cstdint>

namespace sdp4 {

namespace {
thread_local int t_last_hip_error = 0;
}

int set_hip_error(hipError_t err)
{
    t_last_hip_error = static_cast<int>(err);
    return SDP4_EHIP;
}

} // namespace sdp4

namespace {

using sdp4::F32Table;
using sdp4::PeerTable;

bool pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
bool valid_group(int g) { return pow2(g) && g >= SDP4_MIN_GROUP && g <= SDP4_MAX_GROUP; }
bool valid_block(int b) { return b == 0 || (pow2(b) && b >= 2 && b <= SDP4_MAX_HADAMARD); }
bool valid_bits(int b) { return b == 4 || b == 8; }
bool valid_n(int64_t n) { return n >= 0 && n <= SDP4_MAX_ELEMENTS; } // keeps byte counts far from overflow
bool aligned(const void *p, std::uintptr_t a) { return reinterpret_cast<std::uintptr_t>(p) % a == 0; }

// [a, a+na) and [b, b+nb) share a byte
bool overlap(const void *a, int64_t na, const void *b, int64_t nb)
{
    if (na <= 0 || nb <= 0)
        return false;
    const auto a0 = reinterpret_cast<std::uintptr_t>(a);
    const auto b0 = reinterpret_cast<std::uintptr_t>(b);
    return a0 < b0 + static_cast<std::uintptr_t>(nb) && b0 < a0 + static_cast<std::uintptr_t>(na);
}

int64_t lcm_pow2(int a, int b) { return a > b ? a : b; }

// The float nearest to 1/sqrt(n) for n a power of two (the double result is
// far from any float rounding boundary for these n).
float hadamard_scale(int n) { return n > 1 ? static_cast<float>(1.0 / std::sqrt(static_cast<double>(n))) : 1.0f; }

hipStream_t as_stream(void *s) { return static_cast<hipStream_t>(s); }

// Pointer checks shared by the dequantize-reduce entry points: non-null,
// aligned, outputs overlapping neither an input chunk nor each other.
int check_reduce_args(int P, const void *const *codes, const float *const *scales, int64_t n_chunk, int bits_in,
                      int group, int bits_out, void *out_codes, float *out_scales, float *out_f32,
                      PeerTable &peers)
{
    if (!codes || !scales)
        return SDP4_EINVAL;
    if (bits_out ? (!out_codes || !out_scales) : !out_f32)
        return SDP4_EINVAL;
    const int64_t ng = n_chunk / group;
    const int64_t in_cb = n_chunk * bits_in / 8;
    const int64_t out_cb = n_chunk * bits_out / 8;
    for (int p = 0; p < P; ++p) {
        if (!codes[p] || !scales[p])
            return SDP4_EINVAL;
        if (!aligned(codes[p], 16) || !aligned(scales[p], 4))
            return SDP4_EALIGN;
        peers.codes[p] = codes[p];
        peers.scales[p] = scales[p];
    }
    if ((out_codes && !aligned(out_codes, 16)) || (out_scales && !aligned(out_scales, 4)) ||
        (out_f32 && !aligned(out_f32, 16)))
        return SDP4_EALIGN;
    const void *outs[3] = {bits_out ? out_codes : nullptr, bits_out ? out_scales : nullptr, out_f32};
    const int64_t outn[3] = {bits_out ? out_cb : 0, bits_out ? 4 * ng : 0, out_f32 ? 4 * n_chunk : 0};
    for (int i = 0; i < 3; ++i) {
        if (!outs[i])
            continue;
        for (int p = 0; p < P; ++p)
            if (overlap(outs[i], outn[i], codes[p], in_cb) || overlap(outs[i], outn[i], scales[p], 4 * ng))
                return SDP4_EINVAL;
        for (int j = 0; j < i; ++j)
            if (outs[j] && overlap(outs[i], outn[i], outs[j], outn[j]))
                return SDP4_EINVAL;
    }
    return SDP4_OK;
}

// qWD encode / decode with either codec; minv is used (and checked) only by
// the asymmetric one, the symmetric entry points pass null.
int qwd_encode(const float *w_new, const void *w_prev, int prev_dtype, int64_t n, int group,
               uint8_t *codes, float *scale, float *minv, bool sym, void *stream)
{
    if (!valid_n(n) || !valid_group(group) || (prev_dtype != SDP4_F32 && prev_dtype != SDP4_BF16))
        return SDP4_EINVAL;
    if (n % group)
        return SDP4_EALIGN;
    if (n == 0)
        return SDP4_OK;
    if (!w_new || !w_prev || !codes || !scale || (!sym && !minv))
        return SDP4_EINVAL;
    if (!aligned(w_new, 16) || !aligned(w_prev, 16) || !aligned(codes, 16) || !aligned(scale, 4) ||
        (minv && !aligned(minv, 4)))
        return SDP4_EALIGN;
    const int64_t esz = prev_dtype == SDP4_BF16 ? 2 : 4;
    const int64_t ng = n / group;
    const void *outs[3] = {codes, scale, minv};
    const int64_t outn[3] = {n / 2, 4 * ng, 4 * ng};
    for (int i = 0; i < 3; ++i) {
        if (!outs[i])
            continue;
        if (overlap(outs[i], outn[i], w_new, 4 * n) || overlap(outs[i], outn[i], w_prev, esz * n))
            return SDP4_EINVAL;
        for (int j = 0; j < i; ++j)
            if (overlap(outs[i], outn[i], outs[j], outn[j]))
                return SDP4_EINVAL;
    }
    return sdp4::launch_qwd_encode(w_new, w_prev, prev_dtype == SDP4_BF16, sym, n, group, codes, scale,
                                   minv, as_stream(stream));
}

int qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n, int group,
               void *w_prev, int prev_dtype, bool sym, void *stream)
{
    if (!valid_n(n) || !valid_group(group) || (prev_dtype != SDP4_F32 && prev_dtype != SDP4_BF16))
        return SDP4_EINVAL;
    if (n % group)
        return SDP4_EALIGN;
    if (n == 0)
        return SDP4_OK;
    if (!codes || !scale || !w_prev || (!sym && !minv))
        return SDP4_EINVAL;
    if (!aligned(codes, 16) || !aligned(w_prev, 16) || !aligned(scale, 4) || (minv && !aligned(minv, 4)))
        return SDP4_EALIGN;
    const int64_t esz = prev_dtype == SDP4_BF16 ? 2 : 4;
    const int64_t ng = n / group;
    if (overlap(w_prev, esz * n, codes, n / 2) || overlap(w_prev, esz * n, scale, 4 * ng) ||
        (minv && overlap(w_prev, esz * n, minv, 4 * ng)))
        return SDP4_EINVAL;
    return sdp4::launch_qwd_decode(codes, scale, minv, n, group, w_prev, prev_dtype == SDP4_BF16, sym,
                                   as_stream(stream));
}

} // namespace

extern "C" {

int sdp4_qwd_encode(const float *w_new, const void *w_prev, int prev_dtype, int64_t n, int group,
                    uint8_t *codes, float *scale, float *minv, void *stream)
{
    return qwd_encode(w_new, w_prev, prev_dtype, n, group, codes, scale, minv, false, stream);
}

int sdp4_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                    int group, void *w_prev, int prev_dtype, void *stream)
{
    return qwd_decode(codes, scale, minv, n, group, w_prev, prev_dtype, false, stream);
}

int sdp4_qwd_encode_sym(const float *w_new, const void *w_prev, int prev_dtype, int64_t n, int group,
                        uint8_t *codes, float *scale, void *stream)
{
    return qwd_encode(w_new, w_prev, prev_dtype, n, group, codes, scale, nullptr, true, stream);
}

int sdp4_qwd_decode_sym(const uint8_t *codes, const float *scale, int64_t n, int group, void *w_prev,
                        int prev_dtype, void *stream)
{
    return qwd_decode(codes, scale, nullptr, n, group, w_prev, prev_dtype, true, stream);
}

int sdp4_grad_quant(const float *x, int64_t n, int bits, int hadamard_block, int group, void *codes,
                    float *scale, void *stream)
{
    if (!valid_n(n) || !valid_bits(bits) || !valid_block(hadamard_block) || !valid_group(group))
        return SDP4_EINVAL;
    if (n % lcm_pow2(group, hadamard_block))
        return SDP4_EALIGN;
    if (n == 0)
        return SDP4_OK;
    if (!x || !codes || !scale)
        return SDP4_EINVAL;
    if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scale, 4))
        return SDP4_EALIGN;
    const int64_t cb = n * bits / 8, sb = 4 * (n / group);
    if (overlap(codes, cb, x, 4 * n) || overlap(scale, sb, x, 4 * n) || overlap(codes, cb, scale, sb))
        return SDP4_EINVAL;
    return sdp4::launch_grad_quant(x, n, bits, hadamard_block, group, hadamard_scale(hadamard_block),
                                   static_cast<uint8_t *>(codes), scale, as_stream(stream));
}

int sdp4_grad_quant_sr(const float *x, int64_t n, int bits, int hadamard_block, int group, uint64_t seed,
                       uint64_t offset, void *codes, float *scale, void *stream)
{
    if (!valid_n(n) || !valid_bits(bits) || !valid_block(hadamard_block) || !valid_group(group))
        return SDP4_EINVAL;
    if (n % lcm_pow2(group, hadamard_block) || offset % 8)
        return SDP4_EALIGN;
    if (n == 0)
        return SDP4_OK;
    if (!x || !codes || !scale)
        return SDP4_EINVAL;
    if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scale, 4))
        return SDP4_EALIGN;
    const int64_t cb = n * bits / 8, sb = 4 * (n / group);
    if (overlap(codes, cb, x, 4 * n) || overlap(scale, sb, x, 4 * n) || overlap(codes, cb, scale, sb))
        return SDP4_EINVAL;
    return sdp4::launch_grad_quant_sr(x, n, bits, hadamard_block, group, hadamard_scale(hadamard_block), seed,
                                      offset, static_cast<uint8_t *>(codes), scale, as_stream(stream));
}

int sdp4_dequant_reduce_sr(int P, const void *const *codes, const float *const *scales, int64_t n_chunk,
                           int bits_in, int group, int bits_out, uint64_t seed, uint64_t offset,
                           void *out_codes, float *out_scales, float *out_f32, void *stream)
{
    if (P < 1 || P > SDP4_MAX_PEERS)
        return SDP4_ERANGE;
    if (!valid_n(n_chunk) || !valid_bits(bits_in) || !valid_group(group) || !valid_bits(bits_out))
        return SDP4_EINVAL;
    if (n_chunk % group || offset % 8)
        return SDP4_EALIGN;
    if (n_chunk == 0)
        return SDP4_OK;
    PeerTable peers{};
    const int rc = check_reduce_args(P, codes, scales, n_chunk, bits_in, group, bits_out, out_codes, out_scales,
                                     out_f32, peers);
    if (rc != SDP4_OK)
        return rc;
    return sdp4::launch_dequant_reduce_sr(peers, P, n_chunk, bits_in, group, bits_out, seed, offset,
                                          static_cast<uint8_t *>(out_codes), out_scales, out_f32,
                                          as_stream(stream));
}

int sdp4_dequant_reduce(int P, const void *const *codes, const float *const *scales,
                        int64_t n_chunk, int bits_in, int group, int bits_out, int hadamard_block,
                        float out_scale, void *out_codes, float *out_scales, float *out_f32,
                        void *stream)
{
    if (P < 1 || P > SDP4_MAX_PEERS)
        return SDP4_ERANGE;
    if (!valid_n(n_chunk) || !valid_bits(bits_in) || !valid_group(group) || !valid_block(hadamard_block) ||
        !(bits_out == 0 || valid_bits(bits_out)) || !std::isfinite(out_scale))
        return SDP4_EINVAL;
    if (bits_out != 0 && hadamard_block != 0)
        return SDP4_EINVAL;
    if (n_chunk % lcm_pow2(group, hadamard_block))
        return SDP4_EALIGN;
    if (n_chunk == 0)
        return SDP4_OK;
    PeerTable peers{};
    const int rc = check_reduce_args(P, codes, scales, n_chunk, bits_in, group, bits_out, out_codes, out_scales,
                                     out_f32, peers);
    if (rc != SDP4_OK)
        return rc;
    return sdp4::launch_dequant_reduce(peers, P, n_chunk, bits_in, group, bits_out, hadamard_block,
                                       hadamard_scale(hadamard_block), out_scale,
                                       static_cast<uint8_t *>(bits_out ? out_codes : nullptr),
                                       bits_out ? out_scales : nullptr, out_f32, as_stream(stream));
}

int sdp4_hadamard(const float *x, float *y, int64_t n, int block, void *stream)
{
    if (!valid_n(n) || block == 0 || !valid_block(block))
        return SDP4_EINVAL;
    if (n % block)
        return SDP4_EALIGN;
    if (n == 0)
        return SDP4_OK;
    if (!x || !y)
        return SDP4_EINVAL;
    if (!aligned(x, 16) || !aligned(y, 16))
        return SDP4_EALIGN;
    if (x != y && overlap(x, 4 * n, y, 4 * n))
        return SDP4_EINVAL;
    return sdp4::launch_hadamard(x, y, n, block, hadamard_scale(block), as_stream(stream));
}

int sdp4_reduce_f32(int P, const float *const *xs, float *y, int64_t n, void *stream)
{
    if (P < 1 || P > SDP4_MAX_PEERS)
        return SDP4_ERANGE;
    if (!valid_n(n))
        return SDP4_EINVAL;
    if (n == 0)
        return SDP4_OK;
    if (!xs || !y)
        return SDP4_EINVAL;
    if (!aligned(y, 16))
        return SDP4_EALIGN;
    F32Table t{};
    for (int p = 0; p < P; ++p) {
        if (!xs[p])
            return SDP4_EINVAL;
        if (!aligned(xs[p], 16))
            return SDP4_EALIGN;
        if (overlap(y, 4 * n, xs[p], 4 * n))
            return SDP4_EINVAL;
        t.p[p] = xs[p];
    }
    return sdp4::launch_reduce_f32(t, P, n, y, as_stream(stream));
}

int sdp4_copy_f32(const float *x, float *y, int64_t n, void *stream)
{
    if (!valid_n(n))
        return SDP4_EINVAL;
    if (n == 0)
        return SDP4_OK;
    if (!x || !y)
        return SDP4_EINVAL;
    if (!aligned(x, 16) || !aligned(y, 16))
        return SDP4_EALIGN;
    if (overlap(x, 4 * n, y, 4 * n))
        return SDP4_EINVAL;
    return sdp4::launch_copy_f32(x, y, n, as_stream(stream));
}

int sdp4_read_f32(const float *x, int64_t n, uint32_t *sink, void *stream)
{
    if (!valid_n(n))
        return SDP4_EINVAL;
    if (n == 0)
        return SDP4_OK;
    if (!x || !sink)
        return SDP4_EINVAL;
    if (!aligned(x, 16) || !aligned(sink, 4))
        return SDP4_EALIGN;
    if (overlap(x, 4 * n, sink, 16))
        return SDP4_EINVAL;
    return sdp4::launch_read_f32(x, n, sink, as_stream(stream));
}

int sdp4_fill_f32(float *y, int64_t n, float value, void *stream)
{
    if (!valid_n(n))
        return SDP4_EINVAL;
    if (n == 0)
        return SDP4_OK;
    if (!y)
        return SDP4_EINVAL;
    if (!aligned(y, 16))
        return SDP4_EALIGN;
    return sdp4::launch_fill_f32(y, n, value, as_stream(stream));
}

int64_t sdp4_codes_bytes(int64_t n, int bits)
{
    if (!valid_n(n) || !valid_bits(bits))
        return -1;
    return n * bits / 8;
}

int64_t sdp4_num_groups(int64_t n, int group)
{
    if (!valid_n(n) || !valid_group(group))
        return -1;
    return n / group;
}

const char *sdp4_status_string(int status)
{
    switch (status) {
    case SDP4_OK: return "ok";
    case SDP4_EINVAL: return "invalid argument";
    case SDP4_EALIGN: return "size or pointer alignment";
    case SDP4_ERANGE: return "peer count out of range";
    case SDP4_EHIP: return "HIP launch failed";
    default: return "unknown status";
    }
}

const char *sdp4_version(void) { return "sdp4-mi355x 0.1 (gfx950)"; }

int sdp4_last_hip_error(void) { return sdp4::t_last_hip_error; }

} // extern "C"
