// kernels.hip -- gfx950 kernels of the SDP4Bit compression hot path and
// their host-side launchers (called by the C ABI layer in abi.cpp after it
// has validated every argument).
//
// Every kernel is a persistent grid-stride loop over wave tiles of 64*E
// consecutive elements (see device.hpp for the lane layout).  Blocks have
// four independent wavefronts, each with its own LDS staging region; no
// kernel needs a block-wide barrier.  All quantities a wave needs for a
// tile are derived from the tile alone, so results do not depend on the
// grid size.
#include "device.hpp"
#include "launch.hpp"

#include <mutex>
#include <tuple>
#include <unordered_map>

namespace sdp4 {

// ---------------------------------------------------------------------------
// qWD encode: d = w_new - widen(w_prev); asymmetric 4-bit codes per group
// ---------------------------------------------------------------------------
template <bool BF16, int E>
__global__ __launch_bounds__(kBlockThreads) void k_qwd_encode(
    const float *__restrict__ w_new, const void *__restrict__ w_prev, int64_t n, int group,
    uint8_t *__restrict__ codes, float *__restrict__ scale, float *__restrict__ minv)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    __shared__ u32x4 lds_all[kWavesPerBlock][kWave * R];
    const int wave = threadIdx.x / kWave;
    u32x4 *lds = lds_all[wave];
    const int lane = lane_id();
    const int64_t ntiles = (n + W - 1) / W;
    const int lanes_per_group = group / E;

    for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave; t < ntiles;
         t += (int64_t)gridDim.x * kWavesPerBlock) {
        const int64_t base = t * W;
        const int valid = (int)(n - base < W ? n - base : W);
        float d[E];
        {
            u32x4 c[R];
            stage_in<R>(reinterpret_cast<const u32x4 *>(w_new + base), valid / 4, lds, c);
            chunks_to_f32<E>(c, d);
        }
        float p[E];
        if constexpr (BF16) {
            u32x4 c[E / 8];
            stage_in<E / 8>(reinterpret_cast<const u32x4 *>(
                                static_cast<const uint16_t *>(w_prev) + base),
                            valid / 8, lds, c);
            bf16_chunks_to_f32<E>(c, p);
        } else {
            u32x4 c[R];
            stage_in<R>(reinterpret_cast<const u32x4 *>(static_cast<const float *>(w_prev) + base),
                        valid / 4, lds, c);
            chunks_to_f32<E>(c, p);
        }
#pragma unroll
        for (int i = 0; i < E; ++i)
            d[i] = d[i] - p[i];

        float mn = d[0], mx = d[0];
#pragma unroll
        for (int i = 1; i < E; ++i) {
            mn = fminf(mn, d[i]);
            mx = fmaxf(mx, d[i]);
        }
        minmax_lanes(mn, mx, lanes_per_group);
        const float range = mx - mn;
        const float r = 15.0f / range;
        const bool degenerate = !(range > 0.0f) || !__builtin_isfinite(range) || !__builtin_isfinite(r);
        const float s = degenerate ? 0.0f : range / 15.0f;
        const float inv = degenerate ? 0.0f : r;

        int q[E];
#pragma unroll
        for (int i = 0; i < E; ++i) {
            const float v = __builtin_rintf((d[i] - mn) * inv);
            q[i] = (int)__builtin_amdgcn_fmed3f(v, 0.0f, 15.0f);
        }
        u32x4 pk[E / 32];
        pack4<E>(q, pk);
        const int off = E * lane;
        if (off < valid) {
            u32x4 *dst = reinterpret_cast<u32x4 *>(codes + (base + off) / 2);
#pragma unroll
            for (int k = 0; k < E / 32; ++k)
                __builtin_nontemporal_store(pk[k], dst + k);
            if (off % group == 0) {
                const int64_t gi = (base + off) / group;
                scale[gi] = s;
                minv[gi] = mn;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// qWD decode: w_prev <- narrow(widen(w_prev) + fma(code, scale, min))
// ---------------------------------------------------------------------------
template <bool BF16, int E>
__global__ __launch_bounds__(kBlockThreads) void k_qwd_decode(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const float *__restrict__ minv, int64_t n, int group, void *__restrict__ w_prev)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    __shared__ u32x4 lds_all[kWavesPerBlock][kWave * R];
    const int wave = threadIdx.x / kWave;
    u32x4 *lds = lds_all[wave];
    const int lane = lane_id();
    const int64_t ntiles = (n + W - 1) / W;

    for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave; t < ntiles;
         t += (int64_t)gridDim.x * kWavesPerBlock) {
        const int64_t base = t * W;
        const int valid = (int)(n - base < W ? n - base : W);
        const int off = E * lane;
        const bool active = off < valid;
        u32x4 cw[E / 32];
        float s = 0.0f, mn = 0.0f;
        if (active) {
            const u32x4 *src = reinterpret_cast<const u32x4 *>(codes + (base + off) / 2);
#pragma unroll
            for (int k = 0; k < E / 32; ++k)
                cw[k] = __builtin_nontemporal_load(src + k);
            const int64_t gi = (base + off) / group;
            s = scale[gi];
            mn = minv[gi];
        } else {
#pragma unroll
            for (int k = 0; k < E / 32; ++k)
                cw[k] = u32x4{0u, 0u, 0u, 0u};
        }
        float w[E];
        if constexpr (BF16) {
            u32x4 c[E / 8];
            stage_in<E / 8>(reinterpret_cast<const u32x4 *>(static_cast<uint16_t *>(w_prev) + base),
                            valid / 8, lds, c);
            bf16_chunks_to_f32<E>(c, w);
        } else {
            u32x4 c[R];
            stage_in<R>(reinterpret_cast<const u32x4 *>(static_cast<float *>(w_prev) + base),
                        valid / 4, lds, c);
            chunks_to_f32<E>(c, w);
        }
#pragma unroll
        for (int i = 0; i < E; ++i) {
            const uint32_t word = cw[i / 32][(i / 8) % 4];
            const float code = (float)((word >> (4 * (i % 8))) & 0xFu);
            w[i] = w[i] + __builtin_fmaf(code, s, mn);
        }
        if constexpr (BF16) {
            u32x4 c[E / 8];
            f32_to_bf16_chunks<E>(w, c);
            stage_out<E / 8>(reinterpret_cast<u32x4 *>(static_cast<uint16_t *>(w_prev) + base),
                             valid / 8, lds, c);
        } else {
            u32x4 c[R];
            f32_to_chunks<E>(w, c);
            stage_out<R>(reinterpret_cast<u32x4 *>(static_cast<float *>(w_prev) + base), valid / 4,
                         lds, c);
        }
    }
}

// ---------------------------------------------------------------------------
// K1: blockwise Hadamard + symmetric BITS-bit group quantization
// ---------------------------------------------------------------------------
template <int BITS, int E>
__global__ __launch_bounds__(kBlockThreads) void k_grad_quant(
    const float *__restrict__ x, int64_t n, int nblk, int group, float cn,
    uint8_t *__restrict__ codes, float *__restrict__ scale)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    constexpr float qmax = BITS == 8 ? 127.0f : 7.0f;
    __shared__ u32x4 lds_all[kWavesPerBlock][kWave * R];
    const int wave = threadIdx.x / kWave;
    u32x4 *lds = lds_all[wave];
    const int lane = lane_id();
    const int64_t ntiles = (n + W - 1) / W;
    const int lanes_per_group = group / E;

    for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave; t < ntiles;
         t += (int64_t)gridDim.x * kWavesPerBlock) {
        const int64_t base = t * W;
        const int valid = (int)(n - base < W ? n - base : W);
        float v[E];
        {
            u32x4 c[R];
            stage_in<R>(reinterpret_cast<const u32x4 *>(x + base), valid / 4, lds, c);
            chunks_to_f32<E>(c, v);
        }
        if (nblk > 1)
            fwht_lane<E>(v, nblk, cn);

        float a = 0.0f;
#pragma unroll
        for (int i = 0; i < E; ++i)
            a = fmaxf(a, fabsf(v[i]));
        max_lanes<E>(a, lanes_per_group);
        float s, inv;
        sym_params(a, qmax, s, inv);

        int q[E];
#pragma unroll
        for (int i = 0; i < E; ++i)
            q[i] = quant_sym1(v[i], inv, qmax);

        const int off = E * lane;
        if (off < valid) {
            if constexpr (BITS == 8) {
                u32x4 pk[E / 16];
                pack8<E>(q, pk);
                u32x4 *dst = reinterpret_cast<u32x4 *>(codes + base + off);
#pragma unroll
                for (int k = 0; k < E / 16; ++k)
                    __builtin_nontemporal_store(pk[k], dst + k);
            } else {
                u32x4 pk[E / 32];
                pack4<E>(q, pk);
                u32x4 *dst = reinterpret_cast<u32x4 *>(codes + (base + off) / 2);
#pragma unroll
                for (int k = 0; k < E / 32; ++k)
                    __builtin_nontemporal_store(pk[k], dst + k);
            }
            if (off % group == 0)
                scale[(base + off) / group] = s;
        }
    }
}

// ---------------------------------------------------------------------------
// K2 / K3: dequantize + reduce over P chunks, then re-quantize (BITS_OUT 4/8)
// or inverse Hadamard + out_scale to float32 (BITS_OUT 0)
// ---------------------------------------------------------------------------
template <int BITS_IN, int BITS_OUT, int E>
__global__ __launch_bounds__(kBlockThreads) void k_dequant_reduce(
    PeerTable peers, int P, int64_t n, int nblk, int group, float cn, float out_scale,
    uint8_t *__restrict__ out_codes, float *__restrict__ out_scales, float *__restrict__ out_f32)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    constexpr int CW = E * BITS_IN / 128; // input chunks (16 B) per lane per peer
    constexpr int PB = 4;                 // peers loaded per batch
    __shared__ u32x4 lds_all[kWavesPerBlock][kWave * R];
    const int wave = threadIdx.x / kWave;
    u32x4 *lds = lds_all[wave];
    const int lane = lane_id();
    const int64_t ntiles = (n + W - 1) / W;

    for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave; t < ntiles;
         t += (int64_t)gridDim.x * kWavesPerBlock) {
        const int64_t base = t * W;
        const int valid = (int)(n - base < W ? n - base : W);
        const int off = E * lane;
        const bool active = off < valid;
        const int64_t gi = (base + off) / group;

        float acc[E];
#pragma unroll
        for (int i = 0; i < E; ++i)
            acc[i] = 0.0f;
        for (int p0 = 0; p0 < P; p0 += PB) {
            u32x4 cw[PB][CW];
            float s[PB];
#pragma unroll
            for (int j = 0; j < PB; ++j) {
                if (p0 + j < P && active) {
                    const u32x4 *src = reinterpret_cast<const u32x4 *>(
                        static_cast<const uint8_t *>(peers.codes[p0 + j]) + (base + off) * BITS_IN / 8);
#pragma unroll
                    for (int k = 0; k < CW; ++k)
                        cw[j][k] = __builtin_nontemporal_load(src + k);
                    s[j] = peers.scales[p0 + j][gi];
                } else {
#pragma unroll
                    for (int k = 0; k < CW; ++k)
                        cw[j][k] = u32x4{0u, 0u, 0u, 0u};
                    s[j] = 0.0f;
                }
            }
#pragma unroll
            for (int j = 0; j < PB; ++j) {
                if (p0 + j < P) {
                    uint32_t w[CW * 4];
#pragma unroll
                    for (int k = 0; k < CW; ++k) {
                        w[4 * k] = cw[j][k].x;
                        w[4 * k + 1] = cw[j][k].y;
                        w[4 * k + 2] = cw[j][k].z;
                        w[4 * k + 3] = cw[j][k].w;
                    }
#pragma unroll
                    for (int i = 0; i < E; ++i)
                        acc[i] = __builtin_fmaf(code_f<BITS_IN>(w, i), s[j], acc[i]);
                }
            }
        }

        if constexpr (BITS_OUT == 0) {
            if (nblk > 1)
                fwht_lane<E>(acc, nblk, cn);
            if (out_scale != 1.0f) {
#pragma unroll
                for (int i = 0; i < E; ++i)
                    acc[i] = acc[i] * out_scale;
            }
            u32x4 c[R];
            f32_to_chunks<E>(acc, c);
            stage_out<R>(reinterpret_cast<u32x4 *>(out_f32 + base), valid / 4, lds, c);
        } else {
            if (out_f32) {
                u32x4 c[R];
                f32_to_chunks<E>(acc, c);
                stage_out<R>(reinterpret_cast<u32x4 *>(out_f32 + base), valid / 4, lds, c);
            }
            constexpr float qmax = BITS_OUT == 8 ? 127.0f : 7.0f;
            float a = 0.0f;
#pragma unroll
            for (int i = 0; i < E; ++i)
                a = fmaxf(a, fabsf(acc[i]));
            max_lanes<E>(a, group / E);
            float s, inv;
            sym_params(a, qmax, s, inv);
            int q[E];
#pragma unroll
            for (int i = 0; i < E; ++i)
                q[i] = quant_sym1(acc[i], inv, qmax);
            if (active) {
                if constexpr (BITS_OUT == 8) {
                    u32x4 pk[E / 16];
                    pack8<E>(q, pk);
                    u32x4 *dst = reinterpret_cast<u32x4 *>(out_codes + base + off);
#pragma unroll
                    for (int k = 0; k < E / 16; ++k)
                        __builtin_nontemporal_store(pk[k], dst + k);
                } else {
                    u32x4 pk[E / 32];
                    pack4<E>(q, pk);
                    u32x4 *dst = reinterpret_cast<u32x4 *>(out_codes + (base + off) / 2);
#pragma unroll
                    for (int k = 0; k < E / 32; ++k)
                        __builtin_nontemporal_store(pk[k], dst + k);
                }
                if (off % group == 0)
                    out_scales[gi] = s;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// standalone Hadamard (unfused variant); in place allowed
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kBlockThreads) void k_hadamard(const float *x, float *y, int64_t n,
                                                             int nblk, float cn)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    __shared__ u32x4 lds_all[kWavesPerBlock][kWave * R];
    const int wave = threadIdx.x / kWave;
    u32x4 *lds = lds_all[wave];
    const int64_t ntiles = (n + W - 1) / W;
    for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave; t < ntiles;
         t += (int64_t)gridDim.x * kWavesPerBlock) {
        const int64_t base = t * W;
        const int valid = (int)(n - base < W ? n - base : W);
        u32x4 c[R];
        stage_in<R>(reinterpret_cast<const u32x4 *>(x + base), valid / 4, lds, c);
        float v[E];
        chunks_to_f32<E>(c, v);
        fwht_lane<E>(v, nblk, cn);
        f32_to_chunks<E>(v, c);
        stage_out<R>(reinterpret_cast<u32x4 *>(y + base), valid / 4, lds, c);
    }
}

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
    // tail (n not a multiple of 4)
    for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float a = 0.0f;
        for (int p = 0; p < P; ++p)
            a = a + xs.p[p][i];
        y[i] = a;
    }
}

__global__ __launch_bounds__(kBlockThreads) void k_copy_f32(const float *__restrict__ x,
                                                             float *__restrict__ y, int64_t n)
{
    const int64_t n4 = n / 4;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
        __builtin_nontemporal_store(__builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(x) + i),
                                    reinterpret_cast<u32x4 *>(y) + i);
    for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        y[i] = x[i];
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
namespace {

std::mutex g_occ_mu;
std::unordered_map<const void *, int> g_occ; // kernel -> resident blocks per CU
int g_cus[64];

// Persistent grid: one full wave of resident blocks, never more than the
// number of tiles needs.
template <typename K>
int grid_for(K kernel, int64_t nwork_blocks, hipError_t &err)
{
    int dev = 0;
    err = hipGetDevice(&dev);
    if (err != hipSuccess)
        return 0;
    int per_cu;
    int cus;
    {
        std::lock_guard<std::mutex> lk(g_occ_mu);
        if (dev < 64 && g_cus[dev] == 0) {
            int v = 0;
            err = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev);
            if (err != hipSuccess)
                return 0;
            g_cus[dev] = v;
        }
        cus = dev < 64 ? g_cus[dev] : 256;
        auto it = g_occ.find(reinterpret_cast<const void *>(kernel));
        if (it == g_occ.end()) {
            int nb = 0;
            err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, kBlockThreads, 0);
            if (err != hipSuccess)
                return 0;
            it = g_occ.emplace(reinterpret_cast<const void *>(kernel), nb > 0 ? nb : 1).first;
        }
        per_cu = it->second;
    }
    int64_t g = (int64_t)cus * per_cu;
    if (nwork_blocks < g)
        g = nwork_blocks;
    return (int)(g > 0 ? g : 1);
}

template <typename... Params, typename... Args>
int launch(void (*kernel)(Params...), int64_t nwork_blocks, hipStream_t stream, Args... args)
{
    hipError_t err;
    const int grid = grid_for(kernel, nwork_blocks, err);
    if (err != hipSuccess)
        return set_hip_error(err);
    std::tuple<Params...> values(args...);
    void *argv[sizeof...(Params)];
    std::apply([&](auto &...v) {
        int i = 0;
        ((argv[i++] = static_cast<void *>(&v)), ...);
    }, values);
    err = hipLaunchKernel(reinterpret_cast<const void *>(kernel), dim3(grid), dim3(kBlockThreads), argv,
                          0, stream);
    if (err != hipSuccess)
        return set_hip_error(err);
    return 0;
}

inline int64_t wave_blocks(int64_t n, int E)
{
    const int64_t W = (int64_t)kWave * E;
    const int64_t tiles = (n + W - 1) / W;
    return (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
}

} // namespace

int launch_qwd_encode(const float *w_new, const void *w_prev, bool bf16, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s)
{
    if (group > 64 * 32) {
        auto k = bf16 ? k_qwd_encode<true, 64> : k_qwd_encode<false, 64>;
        return launch(k, wave_blocks(n, 64), s, w_new, w_prev, n, group, codes, scale, minv);
    }
    auto k = bf16 ? k_qwd_encode<true, 32> : k_qwd_encode<false, 32>;
    return launch(k, wave_blocks(n, 32), s, w_new, w_prev, n, group, codes, scale, minv);
}

int launch_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                      int group, void *w_prev, bool bf16, hipStream_t s)
{
    auto k = bf16 ? k_qwd_decode<true, 32> : k_qwd_decode<false, 32>;
    return launch(k, wave_blocks(n, 32), s, codes, scale, minv, n, group, w_prev);
}

int launch_grad_quant(const float *x, int64_t n, int bits, int nblk, int group, float cn,
                      uint8_t *codes, float *scale, hipStream_t s)
{
    if (group > 64 * 32) {
        auto k = bits == 8 ? k_grad_quant<8, 64> : k_grad_quant<4, 64>;
        return launch(k, wave_blocks(n, 64), s, x, n, nblk, group, cn, codes, scale);
    }
    auto k = bits == 8 ? k_grad_quant<8, 32> : k_grad_quant<4, 32>;
    return launch(k, wave_blocks(n, 32), s, x, n, nblk, group, cn, codes, scale);
}

int launch_dequant_reduce(const PeerTable &peers, int P, int64_t n, int bits_in, int group,
                          int bits_out, int nblk, float cn, float out_scale, uint8_t *out_codes,
                          float *out_scales, float *out_f32, hipStream_t s)
{
    using K = void (*)(PeerTable, int, int64_t, int, int, float, float, uint8_t *, float *, float *);
    const bool wide = group > 64 * 32;
    K k;
    if (bits_in == 8) {
        if (bits_out == 0) k = wide ? k_dequant_reduce<8, 0, 64> : k_dequant_reduce<8, 0, 32>;
        else if (bits_out == 4) k = wide ? k_dequant_reduce<8, 4, 64> : k_dequant_reduce<8, 4, 32>;
        else k = wide ? k_dequant_reduce<8, 8, 64> : k_dequant_reduce<8, 8, 32>;
    } else {
        if (bits_out == 0) k = wide ? k_dequant_reduce<4, 0, 64> : k_dequant_reduce<4, 0, 32>;
        else if (bits_out == 4) k = wide ? k_dequant_reduce<4, 4, 64> : k_dequant_reduce<4, 4, 32>;
        else k = wide ? k_dequant_reduce<4, 8, 64> : k_dequant_reduce<4, 8, 32>;
    }
    return launch(k, wave_blocks(n, wide ? 64 : 32), s, peers, P, n, nblk, group, cn, out_scale,
                  out_codes, out_scales, out_f32);
}

int launch_hadamard(const float *x, float *y, int64_t n, int nblk, float cn, hipStream_t s)
{
    return launch(k_hadamard<32>, wave_blocks(n, 32), s, x, y, n, nblk, cn);
}

int launch_reduce_f32(const F32Table &xs, int P, int64_t n, float *y, hipStream_t s)
{
    const int64_t blocks = (n / 4 + kBlockThreads - 1) / kBlockThreads;
    return launch(k_reduce_f32, blocks > 0 ? blocks : 1, s, xs, P, n, y);
}

int launch_copy_f32(const float *x, float *y, int64_t n, hipStream_t s)
{
    const int64_t blocks = (n / 4 + kBlockThreads - 1) / kBlockThreads;
    return launch(k_copy_f32, blocks > 0 ? blocks : 1, s, x, y, n);
}

} // namespace sdp4
