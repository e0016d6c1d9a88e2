// device.hpp -- wavefront building blocks shared by the gfx950 kernels.
//
// Register layout used by every element-wise kernel: a wavefront owns a
// "wave tile" of 64*E consecutive elements and lane l holds the E
// consecutive elements [E*el, E*el + E) of it, where the element lane el is
// l itself, or, in the kernels whose Hadamard blocks span several lanes, a
// fixed permutation of l inside each row of 16 lanes (element_lane) that
// puts every butterfly partner within DPP reach.  Quantization groups and
// Hadamard blocks are aligned to E-element lane slices (group >= E), so a
// group or block is either inside one lane (handled in registers) or spans
// an aligned block of 2^k lanes (handled with cross-lane exchanges).
//
// Global memory is read and written in the coalesced order (instruction i,
// lane l touches the 16-byte chunk 64*i + l of the tile) and transposed to
// or from the lane-contiguous layout through a wave-private LDS region, with
// an XOR swizzle of the chunk index that keeps both access patterns of each
// transpose free of LDS bank conflicts.  The LDS serves a 16-byte read to 16
// lanes per cycle over 64 banks of 4 bytes, a 16-byte write to 8 lanes over
// 32 (as the bank-conflict counters show), so a transpose in (coalesced
// write, lane-contiguous read) and a transpose out (lane-contiguous write,
// coalesced read) take different swizzles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define SDP4_DEV __device__ __forceinline__

namespace sdp4 {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#ifndef SDP4_WAVES_PER_BLOCK
#define SDP4_WAVES_PER_BLOCK 4
#endif

constexpr int kWave = 64;
constexpr int kWavesPerBlock = SDP4_WAVES_PER_BLOCK; // independent wavefronts per block
constexpr int kBlockThreads = kWave * kWavesPerBlock;

SDP4_DEV int lane_id() { return __lane_id(); }

// Order LDS traffic of one wavefront: everything before is visible to every
// lane of the wave after, and the compiler does not move memory ops across.
SDP4_DEV void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// cross-lane exchange: value of lane (lane ^ D)
// ---------------------------------------------------------------------------
template <int D>
SDP4_DEV float xor_lane(float v)
{
    static_assert(D == 1 || D == 2 || D == 4 || D == 8 || D == 16 || D == 32, "distance");
    const int iv = __builtin_bit_cast(int, v);
    int r;
    if constexpr (D == 1) {
        r = __builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, true); // quad_perm [1,0,3,2]
    } else if constexpr (D == 2) {
        r = __builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, true); // quad_perm [2,3,0,1]
    } else if constexpr (D < 32) {
        r = __builtin_amdgcn_ds_swizzle(iv, (D << 10) | 0x1F); // bit mode: lane ^ D within 32
    } else {
        r = __builtin_amdgcn_ds_bpermute((lane_id() ^ 32) << 2, iv);
    }
    return __builtin_bit_cast(float, r);
}

// DPP exchanges inside rows of 16 lanes: quad_perm [1,0,3,2] (lane ^ 1),
// quad_perm [2,3,0,1] (lane ^ 2), row_half_mirror (lane ^ 7 within 8 lanes),
// row_ror:8 (lane ^ 8 within 16 lanes).  Every source lane is valid, so no
// lane falls back to the `old` operand.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppRor8 = 0x128;

// s_waitcnt immediate (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8) that waits for every outstanding vector-memory load and
// for nothing else.
constexpr int kWaitVmcnt0 = 0x0F70;

template <int CTRL>
SDP4_DEV uint32_t dpp_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

template <int CTRL>
SDP4_DEV float dpp_f32(float v)
{
    return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(v)));
}

// Largest value over an aligned block of `lanes` (power of two, 1..64)
// neighbouring lanes, for a >= +0 (a largest magnitude).  Non-negative
// floats order like their bit patterns, so this is an unsigned maximum,
// which the compiler fuses with the DPP exchange.  A maximum may join the
// lanes of the block in any order: lane ^ 1, lane ^ 2, the mirror within 8
// (lane ^ 7), lane ^ 8 within 16, then lane ^ 16 and lane ^ 32.
SDP4_DEV void max_lanes(float &a, int lanes)
{
    uint32_t b = __float_as_uint(a);
    if (lanes > 1) b = max(b, dpp_u32<kDppXor1>(b));
    if (lanes > 2) b = max(b, dpp_u32<kDppXor2>(b));
    if (lanes > 4) b = max(b, dpp_u32<kDppHalfMirror>(b));
    if (lanes > 8) b = max(b, dpp_u32<kDppRor8>(b));
    if (lanes > 16) b = max(b, (uint32_t)__builtin_amdgcn_ds_swizzle((int)b, (16 << 10) | 0x1F));
    if (lanes > 32) b = max(b, (uint32_t)__builtin_amdgcn_ds_bpermute((lane_id() ^ 32) << 2, (int)b));
    a = __uint_as_float(b);
}

// Smallest and largest value over an aligned block of `lanes` lanes.
SDP4_DEV void minmax_lanes(float &mn, float &mx, int lanes)
{
    if (lanes > 1) { mn = fminf(mn, dpp_f32<kDppXor1>(mn)); mx = fmaxf(mx, dpp_f32<kDppXor1>(mx)); }
    if (lanes > 2) { mn = fminf(mn, dpp_f32<kDppXor2>(mn)); mx = fmaxf(mx, dpp_f32<kDppXor2>(mx)); }
    if (lanes > 4) { mn = fminf(mn, dpp_f32<kDppHalfMirror>(mn)); mx = fmaxf(mx, dpp_f32<kDppHalfMirror>(mx)); }
    if (lanes > 8) { mn = fminf(mn, dpp_f32<kDppRor8>(mn)); mx = fmaxf(mx, dpp_f32<kDppRor8>(mx)); }
    if (lanes > 16) { mn = fminf(mn, xor_lane<16>(mn)); mx = fmaxf(mx, xor_lane<16>(mx)); }
    if (lanes > 32) { mn = fminf(mn, xor_lane<32>(mn)); mx = fmaxf(mx, xor_lane<32>(mx)); }
}

// ---------------------------------------------------------------------------
// LDS staging between the coalesced and the lane-contiguous layouts
// ---------------------------------------------------------------------------
// R = 16-byte chunks per lane; the wave tile has 64*R chunks.  Both
// swizzles permute chunks within aligned blocks of R (or 8) chunks.
//
// Transpose out: lanes l .. l+7 write chunks R*l + k (rows R apart) and
// lanes l .. l+15 read the consecutive chunks c .. c+15.
template <int R>
SDP4_DEV int swz(int c)
{
    if constexpr (R >= 8)
        return c ^ ((c / R) & 7);
    else
        return c ^ ((c >> 3) & 7);
}

// Transpose in: lanes l .. l+7 write consecutive chunks and lanes
// l .. l+15 read chunks R*l + k, whose bits 4 and up hold the lane's low
// bits; folding them into the chunk's low bits spreads the 16 reads over
// the 16 bank quads.
template <int R>
SDP4_DEV int swz_in(int c)
{
    static_assert(R >= 1 && R <= 16 && (R & (R - 1)) == 0, "chunks per lane");
    return c ^ ((c >> 4) & (R - 1));
}

// Coalesced global loads of one tile: instruction i, lane l reads chunk
// 64*i + l.  Chunks at or beyond `valid` are not read and are zero.
// WHOLE_FAST: a whole tile (every tile but the last) is loaded without
// per-chunk guards.  Callers that batch the loads of several buffers (the
// peers of a dequantize-reduce) keep the guarded form, whose loads the
// compiler schedules together.
template <int R, bool WHOLE_FAST = true>
SDP4_DEV void gload(const u32x4 *__restrict__ g, int valid, u32x4 (&t)[R])
{
    const int lane = lane_id();
    if (WHOLE_FAST && valid >= kWave * R) {
#pragma unroll
        for (int i = 0; i < R; ++i)
            t[i] = __builtin_nontemporal_load(g + kWave * i + lane);
        return;
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int c = kWave * i + lane;
        t[i] = c < valid ? __builtin_nontemporal_load(g + c) : u32x4{0u, 0u, 0u, 0u};
    }
}

// Coalesced chunks -> lane-contiguous chunks through the wave's LDS region:
// lane l gets the chunks R*el .. R*el+R-1 of element lane el (el = l unless
// the kernel relabels its lanes, see element_lane).
template <int R>
SDP4_DEV void transpose_in(const u32x4 (&t)[R], u32x4 *lds, u32x4 (&out)[R], int el)
{
    const int lane = lane_id();
#pragma unroll
    for (int i = 0; i < R; ++i)
        lds[swz_in<R>(kWave * i + lane)] = t[i];
    wave_lds_sync();
#pragma unroll
    for (int k = 0; k < R; ++k)
        out[k] = lds[swz_in<R>(R * el + k)];
    wave_lds_sync();
}

template <int R>
SDP4_DEV void transpose_in(const u32x4 (&t)[R], u32x4 *lds, u32x4 (&out)[R])
{
    transpose_in<R>(t, lds, out, lane_id());
}

// The same through an LDS region of half the tile (32*R chunks): lanes
// 0..31 take their chunks from the first half of the coalesced chunks,
// lanes 32..63 from the second, one half after the other.
template <int R>
SDP4_DEV void transpose_in_halves(const u32x4 (&t)[R], u32x4 *lds, u32x4 (&out)[R])
{
    static_assert(R % 2 == 0, "halves");
    const int lane = lane_id();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int i = 0; i < R / 2; ++i)
            lds[swz_in<R>(kWave * i + lane)] = t[h * (R / 2) + i];
        wave_lds_sync();
        if ((lane >> 5) == h) {
#pragma unroll
            for (int k = 0; k < R; ++k)
                out[k] = lds[swz_in<R>(R * (lane & 31) + k)];
        }
        wave_lds_sync();
    }
}

// Global (coalesced) -> registers (lane-contiguous).
template <int R>
SDP4_DEV void stage_in(const u32x4 *__restrict__ g, int valid, u32x4 *lds, u32x4 (&out)[R])
{
    u32x4 t[R];
    gload<R>(g, valid, t);
    transpose_in<R>(t, lds, out);
}

// Registers (lane-contiguous, element lane el) -> global (coalesced).
// Chunks at or beyond `valid` are not written.
template <int R>
SDP4_DEV void stage_out(u32x4 *__restrict__ g, int valid, u32x4 *lds, const u32x4 (&in)[R], int el)
{
    const int lane = lane_id();
#pragma unroll
    for (int k = 0; k < R; ++k)
        lds[swz<R>(R * el + k)] = in[k];
    wave_lds_sync();
    if (valid >= kWave * R) {
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const int c = kWave * i + lane;
            __builtin_nontemporal_store(lds[swz<R>(c)], g + c);
        }
    } else {
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const int c = kWave * i + lane;
            const u32x4 t = lds[swz<R>(c)];
            if (c < valid)
                __builtin_nontemporal_store(t, g + c);
        }
    }
    wave_lds_sync();
}

template <int R>
SDP4_DEV void stage_out(u32x4 *__restrict__ g, int valid, u32x4 *lds, const u32x4 (&in)[R])
{
    stage_out<R>(g, valid, lds, in, lane_id());
}

template <int E>
SDP4_DEV void chunks_to_f32(const u32x4 (&c)[E / 4], float (&v)[E])
{
#pragma unroll
    for (int k = 0; k < E / 4; ++k) {
        v[4 * k + 0] = __uint_as_float(c[k].x);
        v[4 * k + 1] = __uint_as_float(c[k].y);
        v[4 * k + 2] = __uint_as_float(c[k].z);
        v[4 * k + 3] = __uint_as_float(c[k].w);
    }
}

template <int E>
SDP4_DEV void f32_to_chunks(const float (&v)[E], u32x4 (&c)[E / 4])
{
#pragma unroll
    for (int k = 0; k < E / 4; ++k)
        c[k] = u32x4{__float_as_uint(v[4 * k]), __float_as_uint(v[4 * k + 1]),
                     __float_as_uint(v[4 * k + 2]), __float_as_uint(v[4 * k + 3])};
}

// bfloat16 pairs (E/8 chunks) <-> float
template <int E>
SDP4_DEV void bf16_chunks_to_f32(const u32x4 (&c)[E / 8], float (&v)[E])
{
#pragma unroll
    for (int k = 0; k < E / 8; ++k) {
        const uint32_t w[4] = {c[k].x, c[k].y, c[k].z, c[k].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[8 * k + 2 * j] = __uint_as_float(w[j] << 16);
            v[8 * k + 2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
        }
    }
}

// Two floats -> packed bfloat16 (first in the low half), round to nearest
// even: one v_cvt_pk_bf16_f32 on gfx950 (finite inputs; denormals kept).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

SDP4_DEV uint32_t bf16x2_rne(float a, float b)
{
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

template <int E>
SDP4_DEV void f32_to_bf16_chunks(const float (&v)[E], u32x4 (&c)[E / 8])
{
#pragma unroll
    for (int k = 0; k < E / 8; ++k)
        c[k] = u32x4{bf16x2_rne(v[8 * k], v[8 * k + 1]), bf16x2_rne(v[8 * k + 2], v[8 * k + 3]),
                     bf16x2_rne(v[8 * k + 4], v[8 * k + 5]), bf16x2_rne(v[8 * k + 6], v[8 * k + 7])};
}

// ---------------------------------------------------------------------------
// blockwise Hadamard transform on the lane layout
// ---------------------------------------------------------------------------
// Butterfly stages of width h = 1, 2, ..., nblk/2 in that order, then one
// multiplication by cn.  Widths below E pair registers of one lane; width
// h >= E pairs register i of lane l with register i of lane l ^ (h / E):
// the lower lane keeps a + b and the upper one a - b, both computed as a
// single-rounding fma(own, +-1, other).  This form keeps the sign of every
// zero as the plain butterfly does; the standalone transform uses it.  The
// fused kernels use the cheaper relabeled form further below.
template <int E, int D>
SDP4_DEV void fwht_cross(float (&v)[E])
{
    const float sg = (lane_id() & D) ? -1.0f : 1.0f;
#pragma unroll
    for (int i = 0; i < E; ++i) {
        const float p = xor_lane<D>(v[i]);
        v[i] = __builtin_fmaf(v[i], sg, p);
    }
}

template <int E, int NB>
SDP4_DEV void fwht_lane(float (&v)[E], float cn)
{
    static_assert(NB >= 2 && (NB & (NB - 1)) == 0 && NB <= 64 * E, "block");
#pragma unroll
    for (int h = 1; h < E && h < NB; h <<= 1) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
            if (i & h)
                continue;
            const float a = v[i], b = v[i + h];
            v[i] = a + b;
            v[i + h] = a - b;
        }
    }
    if constexpr (NB > E) fwht_cross<E, 1>(v);
    if constexpr (NB > 2 * E) fwht_cross<E, 2>(v);
    if constexpr (NB > 4 * E) fwht_cross<E, 4>(v);
    if constexpr (NB > 8 * E) fwht_cross<E, 8>(v);
    if constexpr (NB > 16 * E) fwht_cross<E, 16>(v);
    if constexpr (NB > 32 * E) fwht_cross<E, 32>(v);
#pragma unroll
    for (int i = 0; i < E; ++i)
        v[i] = v[i] * cn;
}

// Relabeled lanes for the fused Hadamard kernels.  Inside each row of 16
// lanes, physical lane p holds element lane el = p ^ (3 * p2) (bits 0 and 1
// flipped when bit 2 is set; bits 2 and up unchanged; the map is its own
// inverse).  Element-lane partners el ^ 1, el ^ 2, el ^ 4, el ^ 8 then sit at
// physical lanes p ^ 1, p ^ 2, p ^ 7, p ^ 8, all reachable by DPP, and the
// element lanes of an aligned block of 2^k lanes sit on one aligned block of
// physical lanes (the same block for 2^k >= 8), so a group reduction over
// aligned physical blocks still joins exactly the lanes of each group.
SDP4_DEV int element_lane(int p)
{
    const int b = (p >> 2) & 1;
    return p ^ (b * 3);
}

// One cross-lane butterfly stage as a single v_fmac_f32_dpp per element:
// v = v + sg * partner, sg = +1 in the lower lane (element-lane bit D clear)
// and -1 in the upper one.  The upper lane thus holds b - a = -(a - b):
// each lane carries its value up to a sign that depends only on the lane,
// and since round-to-nearest-even is symmetric, fl(+-(a + b)) and
// fl(+-(a - b)) are exactly the negated roundings.  (Values that carry a
// sign flip and the matching partner signs always give sg = +-1 as above:
// both lanes of a pair carry the same flip before the stage.)  The 16
// instructions of a block start after 5 wait states, the longest DPP read
// hazard (a VALU write of the source VGPR needs 2, of EXEC 5).
#define SDP4_FMAC_DPP_I(i, CTRL) "v_fmac_f32_dpp %" #i ", %" #i ", %16 " CTRL " row_mask:0xf bank_mask:0xf\n\t"
#define SDP4_FMAC_DPP_16(CTRL, w, s)                                                                             \
    asm volatile("s_nop 4\n\t" SDP4_FMAC_DPP_I(0, CTRL) SDP4_FMAC_DPP_I(1, CTRL) SDP4_FMAC_DPP_I(2, CTRL)        \
                     SDP4_FMAC_DPP_I(3, CTRL) SDP4_FMAC_DPP_I(4, CTRL) SDP4_FMAC_DPP_I(5, CTRL)                 \
                         SDP4_FMAC_DPP_I(6, CTRL) SDP4_FMAC_DPP_I(7, CTRL) SDP4_FMAC_DPP_I(8, CTRL)             \
                             SDP4_FMAC_DPP_I(9, CTRL) SDP4_FMAC_DPP_I(10, CTRL) SDP4_FMAC_DPP_I(11, CTRL)       \
                                 SDP4_FMAC_DPP_I(12, CTRL) SDP4_FMAC_DPP_I(13, CTRL) SDP4_FMAC_DPP_I(14, CTRL)  \
                                     SDP4_FMAC_DPP_I(15, CTRL)                                                  \
                 : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]), "+v"(w[4]), "+v"(w[5]), "+v"(w[6]),         \
                   "+v"(w[7]), "+v"(w[8]), "+v"(w[9]), "+v"(w[10]), "+v"(w[11]), "+v"(w[12]), "+v"(w[13]),      \
                   "+v"(w[14]), "+v"(w[15])                                                                     \
                 : "v"(s))
// The same for a lane slice of 8 elements.
#define SDP4_FMAC_DPP_I8(i, CTRL) "v_fmac_f32_dpp %" #i ", %" #i ", %8 " CTRL " row_mask:0xf bank_mask:0xf\n\t"
#define SDP4_FMAC_DPP_8(CTRL, w, s)                                                                              \
    asm volatile("s_nop 4\n\t" SDP4_FMAC_DPP_I8(0, CTRL) SDP4_FMAC_DPP_I8(1, CTRL) SDP4_FMAC_DPP_I8(2, CTRL)     \
                     SDP4_FMAC_DPP_I8(3, CTRL) SDP4_FMAC_DPP_I8(4, CTRL) SDP4_FMAC_DPP_I8(5, CTRL)              \
                         SDP4_FMAC_DPP_I8(6, CTRL) SDP4_FMAC_DPP_I8(7, CTRL)                                    \
                 : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]), "+v"(w[4]), "+v"(w[5]), "+v"(w[6]),         \
                   "+v"(w[7])                                                                                   \
                 : "v"(s))

template <int E, int D>
SDP4_DEV void fwht_cross_signed(float (&v)[E], int el)
{
    static_assert(E % 8 == 0, "lane slice");
    const float sg = (el & D) ? -1.0f : 1.0f;
    if constexpr (D <= 8 && E % 16 != 0) {
        float(&w)[8] = *reinterpret_cast<float(*)[8]>(v);
        if constexpr (D == 1)
            SDP4_FMAC_DPP_8("quad_perm:[1,0,3,2]", w, sg);
        else if constexpr (D == 2)
            SDP4_FMAC_DPP_8("quad_perm:[2,3,0,1]", w, sg);
        else if constexpr (D == 4)
            SDP4_FMAC_DPP_8("row_half_mirror", w, sg);
        else
            SDP4_FMAC_DPP_8("row_ror:8", w, sg);
    } else if constexpr (D <= 8) {
#pragma unroll
        for (int b = 0; b < E / 16; ++b) {
            float(&w)[16] = *reinterpret_cast<float(*)[16]>(v + 16 * b);
            if constexpr (D == 1)
                SDP4_FMAC_DPP_16("quad_perm:[1,0,3,2]", w, sg);
            else if constexpr (D == 2)
                SDP4_FMAC_DPP_16("quad_perm:[2,3,0,1]", w, sg);
            else if constexpr (D == 4)
                SDP4_FMAC_DPP_16("row_half_mirror", w, sg);
            else
                SDP4_FMAC_DPP_16("row_ror:8", w, sg);
        }
    } else {
#pragma unroll
        for (int i = 0; i < E; ++i)
            v[i] = __builtin_fmaf(xor_lane<D>(v[i]), sg, v[i]);
    }
}

// The blockwise transform of fwht_lane on relabeled lanes (element lane el):
// the same stages in the same order with the same roundings, cross-lane
// stages as fwht_cross_signed.  After the last stage a lane's values carry
// the sign (-1)^popcount(el & (NB/E - 1)), which the final scaling by +-cn
// removes; it is one fma with a +0 addend, so an exact zero comes out as +0
// (the only difference from fwht_lane: -0 results become +0).
template <int E, int NB>
SDP4_DEV void fwht_lane_signed(float (&v)[E], float cn, int el)
{
    static_assert(NB > E && (NB & (NB - 1)) == 0 && NB <= 64 * E, "block");
#pragma unroll
    for (int h = 1; h < E; h <<= 1) {
#pragma unroll
        for (int i = 0; i < E; ++i) {
            if (i & h)
                continue;
            const float a = v[i], b = v[i + h];
            v[i] = a + b;
            v[i + h] = a - b;
        }
    }
    fwht_cross_signed<E, 1>(v, el);
    if constexpr (NB > 2 * E) fwht_cross_signed<E, 2>(v, el);
    if constexpr (NB > 4 * E) fwht_cross_signed<E, 4>(v, el);
    if constexpr (NB > 8 * E) fwht_cross_signed<E, 8>(v, el);
    if constexpr (NB > 16 * E) fwht_cross_signed<E, 16>(v, el);
    if constexpr (NB > 32 * E) fwht_cross_signed<E, 32>(v, el);
    const float c = (__builtin_popcount(el & (NB / E - 1)) & 1) ? -cn : cn;
#pragma unroll
    for (int i = 0; i < E; ++i)
        v[i] = __builtin_fmaf(v[i], c, 0.0f);
}

// log2 of a group size (a power of two, checked on the host): header indices
// are shifts instead of runtime 64-bit divisions.
SDP4_DEV int group_shift(int group) { return __builtin_ctz((unsigned)group); }

// ---------------------------------------------------------------------------
// quantize and pack
// ---------------------------------------------------------------------------
// Per-group symmetric parameters from the group's largest magnitude `a`.
SDP4_DEV void sym_params(float a, float qmax, float &scale, float &inv)
{
    const float r = qmax / a;
    const bool degenerate = !(a > 0.0f) || !__builtin_isfinite(r);
    scale = degenerate ? 0.0f : a / qmax;
    inv = degenerate ? 0.0f : r;
}

// Code bits of one element: fl(x * inv) rounded to the nearest integer,
// ties to even, and returned in the low bits of a word.  Adding 1.5 * 2^23
// to a float of magnitude below 2^22 rounds it to an integer in round-to-
// nearest-even mode (exactly what rint does) and leaves that integer,
// two's complement, in the low mantissa bits.  No clamp is needed: with
// inv = fl(qmax / s) and |x| <= s, |fl(x * inv)| <= fl(qmax (1 + 2^-24)),
// which rounds to at most qmax (and likewise 0..15 for the asymmetric
// case, where 0 <= fl(x - mn) <= fl(mx - mn)).
constexpr float kRoundMagic = 12582912.0f; // 1.5 * 2^23

SDP4_DEV uint32_t code_bits(float x, float inv)
{
    const float v = x * inv;
    return __float_as_uint(v + kRoundMagic);
}

// low bytes of t0..t3 -> one word, t0 in the lowest byte
SDP4_DEV uint32_t pack_bytes4(uint32_t t0, uint32_t t1, uint32_t t2, uint32_t t3)
{
    const uint32_t lo = __builtin_amdgcn_perm(t1, t0, 0x0C0C0400u); // t0.b0, t1.b0
    const uint32_t hi = __builtin_amdgcn_perm(t3, t2, 0x0C0C0400u); // t2.b0, t3.b0
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// E code words -> E bytes (int8) as E/16 chunks
template <int E>
SDP4_DEV void pack8(const uint32_t (&t)[E], u32x4 (&c)[E / 16])
{
#pragma unroll
    for (int k = 0; k < E / 16; ++k) {
        const uint32_t *p = t + 16 * k;
        c[k] = u32x4{pack_bytes4(p[0], p[1], p[2], p[3]), pack_bytes4(p[4], p[5], p[6], p[7]),
                     pack_bytes4(p[8], p[9], p[10], p[11]), pack_bytes4(p[12], p[13], p[14], p[15])};
    }
}

// 8 code words -> 8 nibbles, element 0 in the lowest nibble
SDP4_DEV uint32_t pack_nibbles8(const uint32_t *p)
{
    const uint32_t ev = pack_bytes4(p[0], p[2], p[4], p[6]);
    const uint32_t od = pack_bytes4(p[1], p[3], p[5], p[7]);
    return (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
}

// E code words -> E/2 bytes (nibbles, even element low) as E/32 chunks
template <int E>
SDP4_DEV void pack4(const uint32_t (&t)[E], u32x4 (&c)[E / 32])
{
#pragma unroll
    for (int k = 0; k < E / 32; ++k) {
        const uint32_t *p = t + 32 * k;
        c[k] = u32x4{pack_nibbles8(p), pack_nibbles8(p + 8), pack_nibbles8(p + 16), pack_nibbles8(p + 24)};
    }
}

// ---------------------------------------------------------------------------
// stochastic rounding: counter-based Philox4x32 with 10 rounds (Salmon,
// Moraes, Dror, Shaw, SC'11) keyed by a 64-bit seed
// ---------------------------------------------------------------------------
SDP4_DEV void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
        const uint32_t x0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
        const uint32_t x2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
        c[1] = (uint32_t)p1;
        c[3] = (uint32_t)p0;
        c[0] = x0;
        c[2] = x2;
    }
}

// 16-bit uniforms u[i] in [0, 1) of elements e0 .. e0 + E - 1 (e0 a multiple
// of 8): block e / 8 of the generator gives 8 elements, element e takes half
// (e % 2) of word (e / 2) % 4.
template <int E>
SDP4_DEV void sr_uniforms(uint64_t seed, uint64_t e0, float (&u)[E])
{
    static_assert(E % 8 == 0, "lane slice");
#pragma unroll
    for (int j = 0; j < E / 8; ++j) {
        const uint64_t blk = e0 / 8 + j;
        uint32_t c[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), 0u, 0u};
        philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            u[8 * j + 2 * w] = (float)(c[w] & 0xFFFFu) * (1.0f / 65536.0f);
            u[8 * j + 2 * w + 1] = (float)(c[w] >> 16) * (1.0f / 65536.0f);
        }
    }
}

// Stochastically rounded code bits: floor(fl(fl(x * inv) + u)) clamped to
// [-qmax, qmax] (fl(x * inv) may exceed qmax by an ulp, so the floor of the
// sum can reach qmax + 1), returned like code_bits.
SDP4_DEV uint32_t code_bits_sr(float x, float inv, float u, float qmax)
{
    const float v = x * inv;
    const float f = __builtin_amdgcn_fmed3f(__builtin_floorf(v + u), -qmax, qmax);
    return __float_as_uint(f + kRoundMagic);
}

// signed code e of a chunk array holding `bits`-wide codes
template <int BITS>
SDP4_DEV float code_f(const uint32_t *w, int e)
{
    if constexpr (BITS == 8)
        return (float)((int32_t)(w[e >> 2] << (24 - 8 * (e & 3))) >> 24);
    else
        return (float)((int32_t)(w[e >> 3] << (28 - 4 * (e & 7))) >> 28);
}

} // namespace sdp4
