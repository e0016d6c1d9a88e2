// launch.hpp -- interface between the C ABI layer (abi.cpp) and the kernel
// launchers (kernels.hip).  Launchers assume validated arguments.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

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

int launch_qwd_encode(const float *w_new, const void *w_prev, bool bf16, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s);
int launch_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                      int group, void *w_prev, bool bf16, hipStream_t s);
int launch_grad_quant(const float *x, int64_t n, int bits, int nblk, int group, float cn,
                      uint8_t *codes, float *scale, hipStream_t s);
int launch_dequant_reduce(const PeerTable &peers, int P, int64_t n, int bits_in, int group,
                          int bits_out, int nblk, float cn, float out_scale, uint8_t *out_codes,
                          float *out_scales, float *out_f32, hipStream_t s);
int launch_hadamard(const float *x, float *y, int64_t n, int nblk, float cn, hipStream_t s);
int launch_reduce_f32(const F32Table &xs, int P, int64_t n, float *y, hipStream_t s);
int launch_copy_f32(const float *x, float *y, int64_t n, hipStream_t s);

} // namespace sdp4
