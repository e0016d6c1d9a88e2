// k_qwd.hip -- launchers of the qWD encode and decode kernels (asymmetric
// and symmetric codecs).
#include "kernels.hpp"

namespace sdp4 {

namespace {

// Streaming encoder: the instantiation without the phased mode's LDS buffers.
template <int E>
int qwd_encode_stream(const float *w_new, const void *w_prev, bool bf16, bool sym, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s)
{
    constexpr int WPB = kEncWaves;
    auto k = bf16 ? (sym ? k_qwd_encode<true, true, E, kDepth, WPB, 128, false>
                         : k_qwd_encode<true, false, E, kDepth, WPB, 128, false>)
                  : (sym ? k_qwd_encode<false, true, E, kDepth, WPB, 128, false>
                         : k_qwd_encode<false, false, E, kDepth, WPB, 128, false>);
    return launch<WPB>(k, wave_blocks<WPB>(n, E), kEncStreamCap, s, w_new, w_prev, n, group, codes, scale, minv,
                       uint64_t(0), uint64_t(0));
}

// Read/write phase period and read ticks of a launch (32 elements per lane), or 0 when it streams:
// large launches with a group of at least kEncPhaseMinGroup and a period for their weight type.
uint64_t phase_period(bool bf16, int64_t n, int group, uint64_t &read_ticks, hipError_t &err)
{
    err = hipSuccess;
    read_ticks = 0;
    const uint64_t us = bf16 ? SDP4_ENC_PHASE_US : SDP4_ENC_PHASE_US_F32;
    const uint64_t pct = bf16 ? SDP4_ENC_READ_PCT : SDP4_ENC_READ_PCT_F32;
    if (us == 0 || n < kPhaseMinElements || group < kEncPhaseMinGroup)
        return 0;
    const int khz = wall_clock_khz(err);
    if (err != hipSuccess)
        return 0;
    // the period is set for the buffer of groups >= 128 and scales with the buffer of the
    // instantiation that runs
    const int cap = enc_phase_cap(group >= 128 ? 128 : 64);
    const uint64_t period = khz > 0 ? (uint64_t)khz * us * cap / (1000 * enc_phase_cap(128)) : 0;
    read_ticks = period * pct / 100;
    // Both phases must last at least one clock tick, or a wave could wait for a phase that never
    // comes: otherwise stream.
    if (read_ticks == 0 || read_ticks >= period) {
        read_ticks = 0;
        return 0;
    }
    return period;
}

int qwd_encode_phased(const float *w_new, const void *w_prev, bool bf16, bool sym, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, uint64_t period, uint64_t read_ticks,
                      hipStream_t s)
{
    constexpr int E = 32, WPB = kEncWaves;
    // groups of 64 take the instantiation whose header buffer holds 32 per tile
    auto k = group >= 128
                 ? (bf16 ? (sym ? k_qwd_encode<true, true, E, kDepth, WPB> : k_qwd_encode<true, false, E, kDepth, WPB>)
                         : (sym ? k_qwd_encode<false, true, E, kDepth, WPB> : k_qwd_encode<false, false, E, kDepth, WPB>))
                 : (bf16 ? (sym ? k_qwd_encode<true, true, E, kDepth, WPB, 64>
                                : k_qwd_encode<true, false, E, kDepth, WPB, 64>)
                         : (sym ? k_qwd_encode<false, true, E, kDepth, WPB, 64>
                                : k_qwd_encode<false, false, E, kDepth, WPB, 64>));
    return launch<WPB>(k, wave_blocks<WPB>(n, E), kEncCap, s, w_new, w_prev, n, group, codes, scale, minv, period,
                       read_ticks);
}

template <int E>
int qwd_decode_e(const uint8_t *codes, const float *scale, const float *minv, int64_t n, int group,
                 void *w_prev, bool bf16, bool sym, hipStream_t s)
{
    if (bf16) {
        constexpr int WPB = kDecWaves;
        auto k = sym ? k_qwd_decode<true, true, E, kDepth, WPB> : k_qwd_decode<true, false, E, kDepth, WPB>;
        return launch<WPB>(k, wave_blocks<WPB>(n, E), kDecCap, s, codes, scale, minv, n, group, w_prev);
    }
    constexpr int WPB = kDecF32Waves;
    auto k = sym ? k_qwd_decode<false, true, E, kDepth, WPB> : k_qwd_decode<false, false, E, kDepth, WPB>;
    return launch<WPB>(k, wave_blocks<WPB>(n, E), kDecF32Cap, s, codes, scale, minv, n, group, w_prev);
}

} // namespace

int launch_qwd_encode(const float *w_new, const void *w_prev, bool bf16, bool sym, int64_t n, int group,
                      uint8_t *codes, float *scale, float *minv, hipStream_t s)
{
    if (use_wide_lanes(group, 32)) // a group must fit one wavefront: 64 elements per lane
        return qwd_encode_stream<64>(w_new, w_prev, bf16, sym, n, group, codes, scale, minv, s);
    hipError_t err;
    uint64_t read_ticks = 0;
    const uint64_t period = phase_period(bf16, n, group, read_ticks, err);
    if (err != hipSuccess)
        return set_hip_error(err);
    if (period)
        return qwd_encode_phased(w_new, w_prev, bf16, sym, n, group, codes, scale, minv, period, read_ticks, s);
    if (SDP4_E_ENC_STREAM == 16 && group <= kWave * 16)
        return qwd_encode_stream<16>(w_new, w_prev, bf16, sym, n, group, codes, scale, minv, s);
    return qwd_encode_stream<32>(w_new, w_prev, bf16, sym, n, group, codes, scale, minv, s);
}

int launch_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                      int group, void *w_prev, bool bf16, bool sym, hipStream_t s)
{
    // elements per lane by weight type (every group, >= 32, spans whole lane slices)
    if (bf16)
        return qwd_decode_e<SDP4_E_DEC_BF16>(codes, scale, minv, n, group, w_prev, true, sym, s);
    return qwd_decode_e<SDP4_E_DEC_F32>(codes, scale, minv, n, group, w_prev, false, sym, s);
}

} // namespace sdp4
