// k_reduce_f32_in8.hip -- launcher of the dequantize-reduce kernel with a
// float32 result and optional inverse Hadamard (K3), for 8-bit inputs.
#include "kernels.hpp"

namespace sdp4 {

namespace {

template <int NB>
struct DequantReduceF32 {
    static int run(const PeerTable &peers, int P, int64_t n, int group, float cn, float out_scale,
                   float *out_f32, hipStream_t s)
    {
        if (use_wide_lanes(group, SDP4_E_RED))
            return dr_launch<8, 0, 64, NB>(peers, P, n, group, cn, out_scale, nullptr, nullptr, out_f32, s);
        if constexpr (SDP4_E_RF8 == 16 && NB <= kWave * 16)
            return dr_launch<8, 0, 16, NB>(peers, P, n, group, cn, out_scale, nullptr, nullptr, out_f32, s);
        return dr_launch<8, 0, 32, NB>(peers, P, n, group, cn, out_scale, nullptr, nullptr, out_f32, s);
    }
};

} // namespace

int launch_dequant_reduce_f32_in8(const PeerTable &peers, int P, int64_t n, int group, int nblk, float cn,
                                  float out_scale, float *out_f32, hipStream_t s)
{
    return with_block<DequantReduceF32>(nblk, peers, P, n, group, cn, out_scale, out_f32, s);
}

} // namespace sdp4
