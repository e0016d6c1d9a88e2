// k_reduce.hip -- launchers of the dequantize-reduce kernel with 4- or
// 8-bit re-quantization (K2), and of the float32 reduction and the copy.
#include "kernels.hpp"

#ifndef SDP4_COPY_BPC
#define SDP4_COPY_BPC -64 // block cap of the copy yardstick (one block per 4 KiB chunk)
#endif
#ifndef SDP4_COPY_U
#define SDP4_COPY_U 1 // 16-byte chunks per lane and block-iteration of the copy yardstick
#endif
#ifndef SDP4_REDF_BPC
#define SDP4_REDF_BPC -64 // ... of the standalone float32 reduction
#endif
#ifndef SDP4_STREAM_BPC
#define SDP4_STREAM_BPC 1 // ... of the read-only yardstick (persistent: one atomic per wave at the end)
#endif
#ifndef SDP4_FILL_BPC
#define SDP4_FILL_BPC -64 // ... of the write-only yardstick (one block per 4 KiB)
#endif

namespace sdp4 {

// ---------------------------------------------------------------------------
// standalone float32 reduction and plain copy (16 bytes per lane per step)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlockThreads) void k_reduce_f32(F32Table xs, int P, int64_t n,
                                                               float *__restrict__ y)
{
    const int64_t n4 = n / 4;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f, a3 = 0.0f;
        for (int p = 0; p < P; ++p) {
            const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(xs.p[p]) + i);
            a0 = a0 + __uint_as_float(v.x);
            a1 = a1 + __uint_as_float(v.y);
            a2 = a2 + __uint_as_float(v.z);
            a3 = a3 + __uint_as_float(v.w);
        }
        __builtin_nontemporal_store(u32x4{__float_as_uint(a0), __float_as_uint(a1), __float_as_uint(a2),
                                          __float_as_uint(a3)},
                                    reinterpret_cast<u32x4 *>(y) + i);
    }
    for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float a = 0.0f;
        for (int p = 0; p < P; ++p)
            a = a + xs.p[p][i];
        y[i] = a;
    }
}

// Block-contiguous copy: each block moves U * 4 KiB per iteration with U
// 16-byte loads per lane in flight.
constexpr int kCopyU = SDP4_COPY_U;
__global__ __launch_bounds__(kBlockThreads) void k_copy_f32(const float *__restrict__ x,
                                                             float *__restrict__ y, int64_t n)
{
    constexpr int U = kCopyU;
    const int64_t n4 = n / 4;
    const int64_t chunk = (int64_t)kBlockThreads * U;
    const int64_t nchunks = n4 / chunk;
    const u32x4 *xv = reinterpret_cast<const u32x4 *>(x);
    u32x4 *yv = reinterpret_cast<u32x4 *>(y);
    for (int64_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            v[u] = __builtin_nontemporal_load(xv + c * chunk + u * kBlockThreads + threadIdx.x);
#pragma unroll
        for (int u = 0; u < U; ++u)
            __builtin_nontemporal_store(v[u], yv + c * chunk + u * kBlockThreads + threadIdx.x);
    }
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = nchunks * chunk * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        y[i] = x[i];
}

// ---------------------------------------------------------------------------
// read-only and write-only streams (bandwidth yardsticks), each in the access
// pattern that streamed fastest on MI355X in compute-free sweeps: one block
// of four waves per compute unit; reads in tiles of 8 KiB per wave (eight
// 1-KiB instructions), writes 1 KiB per wave and iteration, the grid's waves
// interleaved so that the whole grid sweeps memory front to back.
// ---------------------------------------------------------------------------
constexpr int kStreamWaves = 4;

// sink[k] ^= XOR of the bit patterns of x[i] over every i = k (mod 4).
__global__ __launch_bounds__(kWave * kStreamWaves) void k_read_f32(const float *__restrict__ x, int64_t n,
                                                                   uint32_t *__restrict__ sink)
{
    constexpr int U = 8;
    const int lane = lane_id();
    const int64_t S = (int64_t)gridDim.x * kStreamWaves;
    const int64_t w = (int64_t)blockIdx.x * kStreamWaves + threadIdx.x / kWave;
    const u32x4 *xv = reinterpret_cast<const u32x4 *>(x);
    const int64_t tiles = n / (4 * kWave * U);
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int64_t t = w; t < tiles; t += S) {
        u32x4 v[U];
#pragma unroll
        for (int i = 0; i < U; ++i)
            v[i] = __builtin_nontemporal_load(xv + (t * U + i) * kWave + lane);
#pragma unroll
        for (int i = 0; i < U; ++i)
            acc ^= v[i];
    }
    // the rest: whole 16-byte chunks, then single elements
    const int64_t gt = w * kWave + lane, G = S * kWave;
    for (int64_t c = tiles * U * kWave + gt; c < n / 4; c += G)
        acc ^= xv[c];
    for (int64_t i = n / 4 * 4 + gt; i < n; i += G) {
        const uint32_t b = __float_as_uint(x[i]);
        acc[i & 3] ^= b;
    }
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        acc.x ^= (uint32_t)__shfl_xor((int)acc.x, d);
        acc.y ^= (uint32_t)__shfl_xor((int)acc.y, d);
        acc.z ^= (uint32_t)__shfl_xor((int)acc.z, d);
        acc.w ^= (uint32_t)__shfl_xor((int)acc.w, d);
    }
    if (lane == 0) {
        atomicXor(sink + 0, acc.x);
        atomicXor(sink + 1, acc.y);
        atomicXor(sink + 2, acc.z);
        atomicXor(sink + 3, acc.w);
    }
}

// y[i] = value.
__global__ __launch_bounds__(kWave * kStreamWaves) void k_fill_f32(float *__restrict__ y, int64_t n, float value)
{
    const int64_t G = (int64_t)gridDim.x * kWave * kStreamWaves;
    const int64_t gt = ((int64_t)blockIdx.x * kStreamWaves + threadIdx.x / kWave) * kWave + lane_id();
    const uint32_t b = __float_as_uint(value);
    const u32x4 v = {b, b, b, b};
    u32x4 *yv = reinterpret_cast<u32x4 *>(y);
    for (int64_t c = gt; c < n / 4; c += G)
        __builtin_nontemporal_store(v, yv + c);
    for (int64_t i = n / 4 * 4 + gt; i < n; i += G)
        y[i] = value;
}

int launch_dequant_reduce(const PeerTable &peers, int P, int64_t n, int bits_in, int group,
                          int bits_out, int nblk, float cn, float out_scale, uint8_t *out_codes,
                          float *out_scales, float *out_f32, hipStream_t s)
{
    if (bits_out == 0)
        return bits_in == 8
                   ? launch_dequant_reduce_f32_in8(peers, P, n, group, nblk, cn, out_scale, out_f32, s)
                   : launch_dequant_reduce_f32_in4(peers, P, n, group, nblk, cn, out_scale, out_f32, s);
    const bool wide = use_wide_lanes(group, SDP4_E_RED);
    if (bits_in == 8 && SDP4_E_RQ8 == 16 && group <= kWave * 16) { // a group must fit one wavefront
        if (bits_out == 4)
            return dr_launch<8, 4, 16, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s);
        return dr_launch<8, 8, 16, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s);
    }
    if (bits_in == 8) {
        if (bits_out == 4)
            return wide ? dr_launch<8, 4, 64, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s)
                        : dr_launch<8, 4, 32, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s);
        return wide ? dr_launch<8, 8, 64, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s)
                    : dr_launch<8, 8, 32, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s);
    }
    if (bits_out == 4)
        return wide ? dr_launch<4, 4, 64, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s)
                    : dr_launch<4, 4, 32, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s);
    return wide ? dr_launch<4, 8, 64, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s)
                : dr_launch<4, 8, 32, 0>(peers, P, n, group, cn, 1.0f, out_codes, out_scales, out_f32, s);
}

int launch_reduce_f32(const F32Table &xs, int P, int64_t n, float *y, hipStream_t s)
{
    const int64_t blocks = (n / 4 + kBlockThreads - 1) / kBlockThreads;
    return launch<kWavesPerBlock>(k_reduce_f32, blocks > 0 ? blocks : 1, SDP4_REDF_BPC, s, xs, P, n, y);
}

int launch_read_f32(const float *x, int64_t n, uint32_t *sink, hipStream_t s)
{
    const int64_t tiles = n / (4 * kWave * 8);
    return launch<kStreamWaves>(k_read_f32, tiles > 0 ? tiles : 1, SDP4_STREAM_BPC, s, x, n, sink);
}

int launch_fill_f32(float *y, int64_t n, float value, hipStream_t s)
{
    const int64_t blocks = n / 4 / (kWave * kStreamWaves);
    return launch<kStreamWaves>(k_fill_f32, blocks > 0 ? blocks : 1, SDP4_FILL_BPC, s, y, n, value);
}

int launch_copy_f32(const float *x, float *y, int64_t n, hipStream_t s)
{
    const int64_t chunks = n / 4 / (kBlockThreads * kCopyU);
    return launch<kWavesPerBlock>(k_copy_f32, chunks > 0 ? chunks : 1, SDP4_COPY_BPC, s, x, y, n);
}

} // namespace sdp4
