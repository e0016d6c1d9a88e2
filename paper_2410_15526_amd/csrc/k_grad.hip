// k_grad.hip -- launchers of the Hadamard + quantization kernel (K1) and of
// the standalone Hadamard transform.
#include "kernels.hpp"

namespace sdp4 {

namespace {

template <int NB>
struct GradQuant {
    static int run(const float *x, int64_t n, int bits, int group, float cn, uint8_t *codes, float *scale,
                   hipStream_t s)
    {
        if (use_wide_lanes(group, 32)) {   // 64 elements per lane: the default shape's register budget
            constexpr int WPB = kWavesPerBlock;
            auto k = bits == 8 ? k_grad_quant<8, 64, NB, kDepth, WPB> : k_grad_quant<4, 64, NB, kDepth, WPB>;
            return launch<WPB>(k, wave_blocks<WPB>(n, 64), kCap, s, x, n, group, cn, codes, scale, uint64_t(0),
                               uint64_t(0));
        }
        if constexpr (NB == 0) {   // no transform: its own lane width and block shape
            constexpr int WPB = kK1PlainWaves;
            if (SDP4_E_K1_PLAIN == 16 && group <= kWave * 16) {
                auto k = bits == 8 ? k_grad_quant<8, 16, 0, kDepth, WPB> : k_grad_quant<4, 16, 0, kDepth, WPB>;
                return launch<WPB>(k, wave_blocks<WPB>(n, 16), kK1PlainCap, s, x, n, group, cn, codes, scale,
                                   uint64_t(0), uint64_t(0));
            }
            auto k = bits == 8 ? k_grad_quant<8, 32, 0, kDepth, WPB> : k_grad_quant<4, 32, 0, kDepth, WPB>;
            return launch<WPB>(k, wave_blocks<WPB>(n, 32), kK1PlainCap, s, x, n, group, cn, codes, scale, uint64_t(0),
                               uint64_t(0));
        }
        if constexpr (NB <= kWave * 8) { // a Hadamard block must fit one wavefront
            if (bits == 8 && SDP4_E_K1 == 8 && group <= kWave * 8) { // and so must a group
                constexpr int WPB = kK1Waves8;
                return launch<WPB>(k_grad_quant<8, 8, NB, kDepth, WPB>, wave_blocks<WPB>(n, 8), kK1Cap8, s, x, n, group,
                                   cn, codes, scale, uint64_t(0), uint64_t(0));
            }
        }
        if (bits == 8 && (SDP4_E_K1 == 8 || SDP4_E_K1 == 16) && group <= kWave * 16) { // a group must fit one wavefront
            constexpr int WPB = kK1Waves;
            return launch<WPB>(k_grad_quant<8, 16, NB, kDepth, WPB>, wave_blocks<WPB>(n, 16), kK1Cap, s, x, n, group, cn,
                               codes, scale, uint64_t(0), uint64_t(0));
        }
        constexpr int WPB = kK1Waves32;
        auto k = bits == 8 ? k_grad_quant<8, 32, NB, kDepth, WPB> : k_grad_quant<4, 32, NB, kDepth, WPB>;
        return launch<WPB>(k, wave_blocks<WPB>(n, 32), kK1Cap32, s, x, n, group, cn, codes, scale, uint64_t(0),
                           uint64_t(0));
    }
};

template <int NB>
struct Hadamard {
    static int run(const float *x, float *y, int64_t n, float cn, hipStream_t s)
    {
        if constexpr (NB < 2)
            return 1;
        else if constexpr (SDP4_E_HAD == 16 && NB <= kWave * 16)
            return launch<kWavesPerBlock>(k_hadamard<16, NB, kDepth, kWavesPerBlock>, wave_blocks<kWavesPerBlock>(n, 16),
                                          kHadCap, s, x, y, n, cn);
        else
            return launch<kWavesPerBlock>(k_hadamard<32, NB, kDepth, kWavesPerBlock>, wave_blocks<kWavesPerBlock>(n, 32),
                                          kHadCap, s, x, y, n, cn);
    }
};

} // namespace

int launch_grad_quant(const float *x, int64_t n, int bits, int nblk, int group, float cn,
                      uint8_t *codes, float *scale, hipStream_t s)
{
    return with_block<GradQuant>(nblk, x, n, bits, group, cn, codes, scale, s);
}

int launch_hadamard(const float *x, float *y, int64_t n, int nblk, float cn, hipStream_t s)
{
    return with_block<Hadamard>(nblk, x, y, n, cn, s);
}

} // namespace sdp4
