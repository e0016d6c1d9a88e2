// launch.hpp -- interface between the C ABI layer (abi.cpp) and the kernel
// launchers (*.hip).  Launchers assume validated arguments.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <tuple>

namespace sdp4 {

constexpr int kMaxPeers = 16;

// Pointer tables passed by value in the kernel arguments.
struct PeerTable {
    const void *codes[kMaxPeers];
    const float *scales[kMaxPeers];
};
struct F32Table {
    const float *p[kMaxPeers];
};

// Records `err` as the calling thread's last HIP error and returns SDP4_EHIP.
int set_hip_error(hipError_t err);

// per_cu_cap values that ask for one block per work block (up to kMaxGrid):
// the hardware dispatches blocks in index order, so the chip's accesses sweep
// memory from front to back, which HBM serves faster than the scattered
// fronts of a persistent grid (every kernel loops over its tiles, so any
// grid size computes the same result).  kFullGrid leaves residency to the
// kernel's occupancy; -k (1 <= k < 64) also reserves enough LDS per block
// that at most k blocks are resident on a compute unit at once.
constexpr int kFullGrid = -64;
constexpr int64_t kMaxGrid = 0x7FFFFFFF;

struct LaunchShape {
    int grid;
    size_t dyn_lds; // LDS bytes reserved per block beyond the kernel's own
};

// Grid of a kernel that loops over its work blocks: with per_cu_cap < 0 one
// block per work block (see kFullGrid); otherwise a persistent grid of the
// blocks of `kernel` (block_threads threads each) that are resident at once
// on the current device (capped at per_cu_cap per compute unit when
// per_cu_cap > 0), and never more than nwork_blocks.
LaunchShape shape_for(const void *kernel, int64_t nwork_blocks, int per_cu_cap, int block_threads, hipError_t &err);
int grid_for(const void *kernel, int64_t nwork_blocks, int per_cu_cap, int block_threads, hipError_t &err);

// Rate of the device's constant wall clock in kHz (cached per device).
int wall_clock_khz(hipError_t &err);

// Launch `kernel` with blocks of WAVES wavefronts.
template <int WAVES, typename... Params, typename... Args>
int launch(void (*kernel)(Params...), int64_t nwork_blocks, int per_cu_cap, hipStream_t stream, Args... args)
{
    hipError_t err;
    const LaunchShape sh = shape_for(reinterpret_cast<const void *>(kernel), nwork_blocks, per_cu_cap, 64 * WAVES, err);
    if (err != hipSuccess)
        return set_hip_error(err);
    std::tuple<Params...> values(args...);
    void *argv[sizeof...(Params)];
    std::apply([&](auto &...v) {
        int i = 0;
        ((argv[i++] = static_cast<void *>(&v)), ...);
    }, values);
    err = hipLaunchKernel(reinterpret_cast<const void *>(kernel), dim3(sh.grid), dim3(64 * WAVES), argv, sh.dyn_lds,
                          stream);
    if (err != hipSuccess)
        return set_hip_error(err);
    return 0;
}

int launch_qwd_encode(const float *w_new, const void *w_prev, bool bf16, bool sym, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s);
int launch_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                      int group, void *w_prev, bool bf16, bool sym, hipStream_t s);
int launch_grad_quant(const float *x, int64_t n, int bits, int nblk, int group, float cn,
                      uint8_t *codes, float *scale, hipStream_t s);
int launch_dequant_reduce(const PeerTable &peers, int P, int64_t n, int bits_in, int group,
                          int bits_out, int nblk, float cn, float out_scale, uint8_t *out_codes,
                          float *out_scales, float *out_f32, hipStream_t s);
int launch_dequant_reduce_f32_in8(const PeerTable &peers, int P, int64_t n, int group, int nblk, float cn,
                                  float out_scale, float *out_f32, hipStream_t s);
int launch_dequant_reduce_f32_in4(const PeerTable &peers, int P, int64_t n, int group, int nblk, float cn,
                                  float out_scale, float *out_f32, hipStream_t s);
int launch_grad_quant_sr(const float *x, int64_t n, int bits, int nblk, int group, float cn, uint64_t seed,
                         uint64_t offset, uint8_t *codes, float *scale, hipStream_t s);
int launch_dequant_reduce_sr(const PeerTable &peers, int P, int64_t n, int bits_in, int group, int bits_out,
                             uint64_t seed, uint64_t offset, uint8_t *out_codes, float *out_scales,
                             float *out_f32, hipStream_t s);
int launch_hadamard(const float *x, float *y, int64_t n, int nblk, float cn, hipStream_t s);
int launch_reduce_f32(const F32Table &xs, int P, int64_t n, float *y, hipStream_t s);
int launch_copy_f32(const float *x, float *y, int64_t n, hipStream_t s);
int launch_read_f32(const float *x, int64_t n, uint32_t *sink, hipStream_t s);
int launch_fill_f32(float *y, int64_t n, float value, hipStream_t s);

} // namespace sdp4
