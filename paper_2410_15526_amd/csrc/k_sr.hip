// k_sr.hip -- launchers of the stochastically rounded gradient quantizers:
// Hadamard + quantization (K1) and dequantize-reduce + re-quantization (K2).
#include "kernels.hpp"

namespace sdp4 {

namespace {

template <int NB>
struct GradQuantSR {
    static int run(const float *x, int64_t n, int bits, int group, float cn, uint64_t seed, uint64_t offset,
                   uint8_t *codes, float *scale, hipStream_t s)
    {
        if (use_wide_lanes(group, 32)) {   // 64 elements per lane: the default shape's register budget
            constexpr int WPB = kWavesPerBlock;
            auto k = bits == 8 ? k_grad_quant<8, 64, NB, kDepth, WPB, true> : k_grad_quant<4, 64, NB, kDepth, WPB, true>;
            return launch<WPB>(k, wave_blocks<WPB>(n, 64), kK1SrCap, s, x, n, group, cn, codes, scale, seed, offset);
        }
        if constexpr (SDP4_E_K1_SR == 16 && NB <= kWave * 16) {
            if (bits == 8 && group <= kWave * 16) { // 8-bit codes, a group within one wavefront
                constexpr int WPB = kK1Sr16Waves;
                return launch<WPB>(k_grad_quant<8, 16, NB, kDepth, WPB, true>, wave_blocks<WPB>(n, 16), kK1Sr16Cap, s,
                                   x, n, group, cn, codes, scale, seed, offset);
            }
        }
        constexpr int WPB = kK1Waves32;
        auto k = bits == 8 ? k_grad_quant<8, 32, NB, kDepth, WPB, true> : k_grad_quant<4, 32, NB, kDepth, WPB, true>;
        return launch<WPB>(k, wave_blocks<WPB>(n, 32), kK1SrCap, s, x, n, group, cn, codes, scale, seed, offset);
    }
};

} // namespace

int launch_grad_quant_sr(const float *x, int64_t n, int bits, int nblk, int group, float cn, uint64_t seed,
                         uint64_t offset, uint8_t *codes, float *scale, hipStream_t s)
{
    return with_block<GradQuantSR>(nblk, x, n, bits, group, cn, seed, offset, codes, scale, s);
}

int launch_dequant_reduce_sr(const PeerTable &peers, int P, int64_t n, int bits_in, int group, int bits_out,
                             uint64_t seed, uint64_t offset, uint8_t *out_codes, float *out_scales,
                             float *out_f32, hipStream_t s)
{
    const bool wide = use_wide_lanes(group, SDP4_E_RED);
    if (bits_in == 8 && SDP4_E_RQ8 == 16 && group <= kWave * 16) { // a group must fit one wavefront
        if (bits_out == 4)
            return dr_launch<8, 4, 16, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s, seed,
                                                offset);
        return dr_launch<8, 8, 16, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s, seed,
                                            offset);
    }
    if (bits_in == 8) {
        if (bits_out == 4)
            return wide ? dr_launch<8, 4, 64, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32,
                                                      s, seed, offset)
                        : dr_launch<8, 4, 32, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32,
                                                      s, seed, offset);
        return wide ? dr_launch<8, 8, 64, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s,
                                                  seed, offset)
                    : dr_launch<8, 8, 32, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s,
                                                  seed, offset);
    }
    if (bits_out == 4)
        return wide ? dr_launch<4, 4, 64, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s,
                                                  seed, offset)
                    : dr_launch<4, 4, 32, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s,
                                                  seed, offset);
    return wide ? dr_launch<4, 8, 64, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s, seed,
                                              offset)
                : dr_launch<4, 8, 32, 0, true>(peers, P, n, group, 1.0f, 1.0f, out_codes, out_scales, out_f32, s, seed,
                                              offset);
}

} // namespace sdp4
