// k_qwd.hip -- launchers of the qWD encode and decode kernels (asymmetric
// and symmetric codecs).
#include "kernels.hpp"

namespace sdp4 {

namespace {

template <int E>
int qwd_encode_e(const float *w_new, const void *w_prev, bool bf16, bool sym, int64_t n, int group,
                 uint8_t *codes, float *scale, float *minv, hipStream_t s)
{
    constexpr int WPB = kEncWaves;
    // groups of 64 take the instantiation whose header buffer holds 32 per tile
    auto k = group >= 128 || E != 32
                 ? (bf16 ? (sym ? k_qwd_encode<true, true, E, kDepth, WPB> : k_qwd_encode<true, false, E, kDepth, WPB>)
                         : (sym ? k_qwd_encode<false, true, E, kDepth, WPB> : k_qwd_encode<false, false, E, kDepth, WPB>))
                 : (bf16 ? (sym ? k_qwd_encode<true, true, E, kDepth, WPB, 64>
                                : k_qwd_encode<true, false, E, kDepth, WPB, 64>)
                         : (sym ? k_qwd_encode<false, true, E, kDepth, WPB, 64>
                                : k_qwd_encode<false, false, E, kDepth, WPB, 64>));
    // Read/write phases for large launches with 32 elements per lane and a
    // group of at least kEncPhaseMinGroup; everything else streams as usual.
    uint64_t period = 0, read_ticks = 0;
    const uint64_t us = bf16 ? SDP4_ENC_PHASE_US : SDP4_ENC_PHASE_US_F32;
    const uint64_t pct = bf16 ? SDP4_ENC_READ_PCT : SDP4_ENC_READ_PCT_F32;
    if (E == 32 && us > 0 && n >= kPhaseMinElements && group >= kEncPhaseMinGroup) {
        hipError_t err;
        const int khz = wall_clock_khz(err);
        if (err != hipSuccess)
            return set_hip_error(err);
        // the period is set for the buffer of groups >= 128 and scales with
        // the buffer of the instantiation that runs
        const int cap = enc_phase_cap(group >= 128 ? 128 : 64);
        period = khz > 0 ? (uint64_t)khz * us * cap / (1000 * enc_phase_cap(128)) : 0;
        read_ticks = period * pct / 100;
        // Both phases must last at least one clock tick, or a wave could wait
        // for a phase that never comes: otherwise stream.
        if (read_ticks == 0 || read_ticks >= period)
            period = read_ticks = 0;
    }
    if (period == 0) { // streaming: the instantiation without the phased mode's LDS buffers
        auto ks = bf16 ? (sym ? k_qwd_encode<true, true, E, kDepth, WPB, 128, false>
                              : k_qwd_encode<true, false, E, kDepth, WPB, 128, false>)
                       : (sym ? k_qwd_encode<false, true, E, kDepth, WPB, 128, false>
                              : k_qwd_encode<false, false, E, kDepth, WPB, 128, false>);
        return launch<WPB>(ks, wave_blocks<WPB>(n, E), kEncStreamCap, s, w_new, w_prev, n, group, codes, scale, minv,
                           period, read_ticks);
    }
    return launch<WPB>(k, wave_blocks<WPB>(n, E), kEncCap, s, w_new, w_prev, n, group, codes, scale, minv, period,
                       read_ticks);
}

template <int E>
int qwd_decode_e(const uint8_t *codes, const float *scale, const float *minv, int64_t n, int group,
                 void *w_prev, bool bf16, bool sym, hipStream_t s)
{
    constexpr int WPB = kDecWaves;
    auto k = bf16 ? (sym ? k_qwd_decode<true, true, E, kDepth, WPB> : k_qwd_decode<true, false, E, kDepth, WPB>)
                  : (sym ? k_qwd_decode<false, true, E, kDepth, WPB> : k_qwd_decode<false, false, E, kDepth, WPB>);
    return launch<WPB>(k, wave_blocks<WPB>(n, E), kDecCap, s, codes, scale, minv, n, group, w_prev);
}

} // namespace

int launch_qwd_encode(const float *w_new, const void *w_prev, bool bf16, bool sym, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s)
{
    if (use_wide_lanes(group, SDP4_E_ENC))
        return qwd_encode_e<64>(w_new, w_prev, bf16, sym, n, group, codes, scale, minv, s);
    return qwd_encode_e<32>(w_new, w_prev, bf16, sym, n, group, codes, scale, minv, s);
}

int launch_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                      int group, void *w_prev, bool bf16, bool sym, hipStream_t s)
{
    if (SDP4_E_DEC == 64 && group >= 64)
        return qwd_decode_e<64>(codes, scale, minv, n, group, w_prev, bf16, sym, s);
    return qwd_decode_e<32>(codes, scale, minv, n, group, w_prev, bf16, sym, s);
}

} // namespace sdp4
