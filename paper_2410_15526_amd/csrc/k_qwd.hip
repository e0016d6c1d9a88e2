// k_qwd.hip -- launchers of the qWD encode and decode kernels.
#include "kernels.hpp"

namespace sdp4 {

int launch_qwd_encode(const float *w_new, const void *w_prev, bool bf16, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s)
{
    if (use_wide_lanes(group, SDP4_E_ENC)) {
        auto k = bf16 ? k_qwd_encode<true, 64, kDepth> : k_qwd_encode<false, 64, kDepth>;
        return launch(k, wave_blocks(n, 64), kCap, s, w_new, w_prev, n, group, codes, scale, minv);
    }
    auto k = bf16 ? k_qwd_encode<true, 32, kDepth> : k_qwd_encode<false, 32, kDepth>;
    return launch(k, wave_blocks(n, 32), kCap, s, w_new, w_prev, n, group, codes, scale, minv);
}

int launch_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                      int group, void *w_prev, bool bf16, hipStream_t s)
{
    if (SDP4_E_DEC == 64 && group >= 64) {
        auto k = bf16 ? k_qwd_decode<true, 64, kDepth> : k_qwd_decode<false, 64, kDepth>;
        return launch(k, wave_blocks(n, 64), kCap, s, codes, scale, minv, n, group, w_prev);
    }
    auto k = bf16 ? k_qwd_decode<true, 32, kDepth> : k_qwd_decode<false, 32, kDepth>;
    return launch(k, wave_blocks(n, 32), kCap, s, codes, scale, minv, n, group, w_prev);
}

} // namespace sdp4
