// kernels.hpp -- gfx950 kernel templates of the SDP4Bit compression hot
// path; the .hip files instantiate and launch them.
//
// Every kernel is a persistent loop of wavefronts over wave tiles of 64*E
// consecutive elements (see device.hpp for the lane layout).  Blocks hold
// independent wavefronts, each with its own LDS staging region; no kernel
// needs a block-wide barrier.  A wave keeps D >= 1 tile buffers and issues
// a tile's global loads once it has processed the tile D places before it:
// with the default D = 1 a wave's loads and its compute alternate, and the
// other waves of the CU cover the load latency.  (With D >= 2 the compiler's
// wait for one tile's loads also covers the later tiles' -- where a partial
// tile's loads are guarded the number in flight depends on the path -- so
// a deeper ring has not paid.)  Everything a wave computes for a tile
// depends on that tile alone, so results do not depend on the grid size or
// on D.
//
// The SDP4_* macros below are build-time tuning knobs; their defaults are
// the measured best on MI355X: one tile buffer per wave and, per kernel
// family, a lane width E (8 to 64 elements per lane), a block shape and a
// grid mode.  Most kernels launch one block per work block, which the
// hardware dispatches in address order, so the chip's accesses sweep memory
// front to back (HBM serves that faster than the scattered fronts of a
// persistent grid), some with a cap on resident blocks per CU where that
// measured faster.  The clock-phased qWD encoder (one block of four waves
// per CU) and the stochastically rounded K1 with 4-bit codes keep persistent
// grids.  (How many bytes a CU keeps in flight, and how far compute spreads
// its requests out, moves the mixed read/write bandwidth of HBM by several
// per cent.)
#pragma once

#include "device.hpp"
#include "launch.hpp"

#ifndef SDP4_PIPE
#define SDP4_PIPE 1 // tile buffers per wave (a tile's loads follow the processing of the one D before)
#endif
#ifndef SDP4_PEER_LDS
#define SDP4_PEER_LDS 1 // int8 peer chunks: coalesced loads + LDS transpose
#endif
// Elements per lane of each kernel family (groups of 4096 always take 64).
#ifndef SDP4_E_ENC_STREAM
#define SDP4_E_ENC_STREAM 16 // the streaming qWD encoder (16 or 32; the phased one takes 32)
#endif
#ifndef SDP4_E_DEC_BF16
#define SDP4_E_DEC_BF16 16 // qWD decode, bf16 model weights
#endif
#ifndef SDP4_E_DEC_F32
#define SDP4_E_DEC_F32 8 // qWD decode, float32 model weights
#endif
#ifndef SDP4_E_K1
#define SDP4_E_K1 16 // 8-bit K1 only (8 or 16): 4-bit codes need 32 per lane to fill a 16-byte store
#endif
#ifndef SDP4_E_RED
#define SDP4_E_RED 32
#endif
#ifndef SDP4_E_K3
#define SDP4_E_K3 32 // dequantize-reduce of 4-bit messages to float32 (K3): 16 or 32 elements per lane
#endif
#ifndef SDP4_E_RF8
#define SDP4_E_RF8 16 // dequantize-reduce of 8-bit messages to float32: 16 or 32 elements per lane
#endif
#ifndef SDP4_E_HAD
#define SDP4_E_HAD 16 // the standalone Hadamard transform: 16 or 32 elements per lane
#endif
#ifndef SDP4_HAD_BPC
#define SDP4_HAD_BPC -4
#endif
#ifndef SDP4_E_RQ8
// Elements per lane of the re-quantizing dequantize-reduce of 8-bit messages,
// deterministic or stochastically rounded (16: one 16-byte chunk per peer and
// lane; groups up to 1024).
#define SDP4_E_RQ8 16
#endif
// Block caps: n > 0 runs a persistent grid of at most n resident blocks per
// compute unit (0: as many as fit); -k (k < 64) one block per work block,
// dispatched in address order, at most k resident per compute unit;
// -64 the same with residency left to occupancy (launch.hpp, kFullGrid).
#ifndef SDP4_BLOCKS_PER_CU
#define SDP4_BLOCKS_PER_CU -4 // block cap of the kernels without one of their own below
#endif
// Block shapes (waves per block, block cap) of the qWD encoder and of the K1
// variants; the standalone transform and the yardsticks use
// SDP4_WAVES_PER_BLOCK (device.hpp) and caps of their own.
#ifndef SDP4_ENC_WAVES
#define SDP4_ENC_WAVES 4
#endif
#ifndef SDP4_ENC_BPC
#define SDP4_ENC_BPC 1 // the clock-phased encoder
#endif
#ifndef SDP4_ENC_STREAM_BPC
#define SDP4_ENC_STREAM_BPC -4 // the streaming encoder (launches that are not phased), without the phased LDS buffers
#endif
#ifndef SDP4_K1_WAVES
#define SDP4_K1_WAVES 4 // K1 with 16 elements per lane
#endif
#ifndef SDP4_K1_WAVES_8
#define SDP4_K1_WAVES_8 4 // K1 with 8 elements per lane
#endif
#ifndef SDP4_K1_BPC_8
#define SDP4_K1_BPC_8 -8
#endif
#ifndef SDP4_K1_WAVES_32
#define SDP4_K1_WAVES_32 8 // K1 with 32 elements per lane (4-bit codes; rounded K1 with 4-bit codes or groups of 2048)
#endif
#ifndef SDP4_E_K1_PLAIN
#define SDP4_E_K1_PLAIN 16 // K1 without a transform: 16 or 32 elements per lane
#endif
#ifndef SDP4_K1_WAVES_PLAIN
#define SDP4_K1_WAVES_PLAIN 4
#endif
#ifndef SDP4_K1_PLAIN_BPC
#define SDP4_K1_PLAIN_BPC -6
#endif
#ifndef SDP4_E_K1_SR
#define SDP4_E_K1_SR 16 // K1 with stochastic rounding, 8-bit codes: 16 or 32 elements per lane
#endif
#ifndef SDP4_K1_SR16_WAVES
#define SDP4_K1_SR16_WAVES 4 // ... with 16 elements per lane: a full grid of 4-wave blocks
#endif
#ifndef SDP4_K1_SR16_BPC
#define SDP4_K1_SR16_BPC -64
#endif
#ifndef SDP4_K1_SR_BPC
#define SDP4_K1_SR_BPC 1 // K1 with stochastic rounding, 32 or 64 per lane: one persistent block per compute unit
#endif
#ifndef SDP4_K1_BPC
#define SDP4_K1_BPC -5 // K1 with a transform, 16 elements per lane
#endif
#ifndef SDP4_K1_BPC_32
#define SDP4_K1_BPC_32 -3 // ... 32 elements per lane
#endif

// Block shapes of the qWD decoder, of the dequantize-reduce with
// re-quantization (K2; 8-bit messages with 16 elements per lane have their
// own) and of the dequantize-reduce to float32 (K3).
#ifndef SDP4_DEC_WAVES
#define SDP4_DEC_WAVES 2 // qWD decode, bf16 model weights
#endif
#ifndef SDP4_DEC_BPC
#define SDP4_DEC_BPC -8
#endif
#ifndef SDP4_DEC_F32_WAVES
#define SDP4_DEC_F32_WAVES 2 // qWD decode, float32 model weights
#endif
#ifndef SDP4_DEC_F32_BPC
#define SDP4_DEC_F32_BPC -8
#endif
#ifndef SDP4_RQ_WAVES
#define SDP4_RQ_WAVES 4
#endif
#ifndef SDP4_RQ_BPC
#define SDP4_RQ_BPC -4
#endif
#ifndef SDP4_RQ8_WAVES // ... of 8-bit messages with 16 elements per lane
#define SDP4_RQ8_WAVES 8
#endif
#ifndef SDP4_RQ8_BPC
#define SDP4_RQ8_BPC -3
#endif
#ifndef SDP4_RQ8_SR_WAVES // ... the same with stochastic rounding
#define SDP4_RQ8_SR_WAVES 8
#endif
#ifndef SDP4_RQ8_SR_BPC
#define SDP4_RQ8_SR_BPC -64
#endif
#ifndef SDP4_RF_WAVES
#define SDP4_RF_WAVES 4
#endif
#ifndef SDP4_RF_BPC
#define SDP4_RF_BPC -4
#endif

#ifndef SDP4_ENC_PHASE_US
#define SDP4_ENC_PHASE_US 66 // qWD encoder read/write period in microseconds (0: ordinary stream)
#endif
#ifndef SDP4_ENC_READ_PCT
#define SDP4_ENC_READ_PCT 92 // per cent of the period spent reading
#endif
#ifndef SDP4_ENC_PHASE_US_F32
#define SDP4_ENC_PHASE_US_F32 0 // the same with float32 model weights (0: they stream, measured faster)
#endif
#ifndef SDP4_ENC_READ_PCT_F32
#define SDP4_ENC_READ_PCT_F32 94
#endif
#ifndef SDP4_ENC_PHASE_DEPTH
#define SDP4_ENC_PHASE_DEPTH 1 // tiles each phased encoder wave keeps loading ahead
#endif
#ifndef SDP4_ENC_EARLY_LOAD_F32
#define SDP4_ENC_EARLY_LOAD_F32 1 // phased encoder, float32 weights: a read phase's first tile loads the next first
#endif
#ifndef SDP4_ENC_EARLY_LOAD_BF16
#define SDP4_ENC_EARLY_LOAD_BF16 0 // the same for bf16 weights
#endif
#ifndef SDP4_ENC_FLUSH_PCT
#define SDP4_ENC_FLUSH_PCT 10 // phased encoder: a buffer that fills with more than this share of the period
                              // left to read is written out at once (else the wave sleeps to the write phase)
#endif
#ifndef SDP4_ENC_HALF_T
#define SDP4_ENC_HALF_T 1 // encoder: transpose its inputs through an LDS region of half a tile
#endif
#ifndef SDP4_ENC_PHASE_CAP
#define SDP4_ENC_PHASE_CAP (SDP4_ENC_HALF_T ? 31 : 27) // tiles each encoder wave buffers in LDS (groups >= 128)
#endif
#ifndef SDP4_ENC_PHASE_CAP64
#define SDP4_ENC_PHASE_CAP64 (SDP4_ENC_HALF_T ? 28 : 25) // the same for groups of 64
#endif

namespace sdp4 {

constexpr int kDepth = SDP4_PIPE;
constexpr int kEncPhaseCap = SDP4_ENC_PHASE_CAP; // tiles buffered per wave by the phased encoder
constexpr int kEncPhaseCap64 = SDP4_ENC_PHASE_CAP64; // ... when its headers are those of groups of 64
constexpr int kEncPhaseDepth = SDP4_ENC_PHASE_DEPTH;
static_assert(SDP4_ENC_READ_PCT > 0 && SDP4_ENC_READ_PCT < 100, "the encoder's read phase is part of its period");
static_assert(SDP4_ENC_READ_PCT_F32 > 0 && SDP4_ENC_READ_PCT_F32 < 100, "the encoder's read phase is part of its period");
static_assert(SDP4_ENC_PHASE_CAP >= 1 && SDP4_ENC_PHASE_DEPTH >= 1, "phased encoder buffers");
constexpr int kEncPhaseMinGroup = 64;       // smallest group the phased encoder buffers headers for
// Tiles buffered per wave for a given smallest group: headers for groups of 64
// take twice the room of those for groups of 128 and up, and the buffers of
// four waves must fit the 160 KiB of LDS.
constexpr int enc_phase_cap(int min_group) { return min_group >= 128 ? kEncPhaseCap : kEncPhaseCap64; }
constexpr int64_t kPhaseMinElements = 1 << 26; // smaller launches use the ordinary stream

// Persistent loop of one wavefront over its tiles t, t + S, t + 2S, ...
// (S = waves in the grid, WPB waves per block).  DEPTH = 0 loads and
// processes one tile at a time; DEPTH = D >= 1 keeps a ring of D register
// buffers (indexed at compile time by unrolling): a tile's loads go out
// once the tile D places earlier is processed, so D - 1 later tiles are in
// flight while one is processed.
template <int DEPTH, int WPB, class Tile, class Load, class Proc>
SDP4_DEV void tile_loop(int64_t ntiles, Load load, Proc proc)
{
    const int wave = threadIdx.x / kWave;
    const int64_t stride = (int64_t)gridDim.x * WPB;
    int64_t t = (int64_t)blockIdx.x * WPB + wave;
    if constexpr (DEPTH == 0) {
        for (; t < ntiles; t += stride) {
            Tile in;
            load(t, in);
            proc(t, in);
        }
    } else {
        Tile buf[DEPTH];
#pragma unroll
        for (int k = 0; k < DEPTH; ++k)
            if (t + k * stride < ntiles)
                load(t + k * stride, buf[k]);
        for (;;) {
#pragma unroll
            for (int k = 0; k < DEPTH; ++k) {
                if (t >= ntiles)
                    return;
                proc(t, buf[k]);
                if (t + DEPTH * stride < ntiles)
                    load(t + DEPTH * stride, buf[k]);
                t += stride;
            }
        }
    }
}

SDP4_DEV int tile_valid(int64_t n, int64_t base, int W) { return (int)(n - base < W ? n - base : W); }

// HBM serves a pure read stream or a pure write stream faster than a mix of
// the two, and every CU reads the same constant-rate wall clock.  In a
// phased loop all waves of the chip issue loads only while
// (clock mod period) < read_ticks and keep each tile's (small) output in a
// wave-private LDS buffer of up to `cap` tiles, which they write out in the
// rest of the period -- so the memory system sees long read-only and
// write-only stretches instead of a mix.  proc(t, in, slot) computes tile t
// into buffer slot `slot`; flush(k) writes slots 0..k-1.  DEPTH tile
// buffers per wave, as in tile_loop (a ring of register buffers, indexed at
// compile time by unrolling).  Every wait is a short sleep until the clock moves to the
// other phase (0 < read_ticks < period, so both phases come round), and the
// loop ends once the wave has no tile left and an empty buffer, so every
// wave exits.  Results do not depend on the timing.
//
// EARLY: the first tile of each read phase issues the next tile's loads
// before its own compute (on a copy of its registers), while the memory
// system would otherwise idle; later tiles compute first, keeping one load
// in flight per wave.
template <int DEPTH, int WPB, bool EARLY, class Tile, class Load, class Proc, class Flush>
SDP4_DEV void phased_tile_loop(int64_t ntiles, int cap, uint64_t period, uint64_t read_ticks, uint64_t flush_ticks,
                               Load load, Proc proc, Flush flush)
{
    static_assert(DEPTH >= 1, "depth");
    const int wave = threadIdx.x / kWave;
    const int64_t stride = (int64_t)gridDim.x * WPB;
    int64_t t = (int64_t)blockIdx.x * WPB + wave;
    Tile buf[DEPTH];
#pragma unroll
    for (int k = 0; k < DEPTH; ++k)
        if (t + k * stride < ntiles)
            load(t + k * stride, buf[k]);
    int nbuf = 0;
    bool fresh = true; // no tile processed since the last flush or wait
    // Phase boundaries on the common grid of multiples of `period`, found by
    // one division here and then advanced by additions.
    uint64_t now = (uint64_t)wall_clock64();
    uint64_t start = now - now % period;
    for (;;) {
#pragma unroll
        for (int k = 0; k < DEPTH; ++k) {
            // tile t is in buf[k]; wait until it may be processed
            for (;;) {
                const bool have = t < ntiles;
                now = (uint64_t)wall_clock64();
                while (now - start >= period)
                    start += period;
                const bool reading = now - start < read_ticks;
                if (have && nbuf < cap && reading) {
                    if (EARLY && fresh && t + DEPTH * stride < ntiles) {
                        Tile cur = buf[k];
                        // this tile's loads landed long ago: settle them before
                        // the next ones go out, or the compiler's wait before the
                        // first use of `cur` also waits for the new loads
                        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
                        load(t + DEPTH * stride, buf[k]);
                        proc(t, cur, nbuf);
                    } else {
                        proc(t, buf[k], nbuf);
                        if (t + DEPTH * stride < ntiles)
                            load(t + DEPTH * stride, buf[k]);
                    }
                    fresh = false;
                    ++nbuf;
                    t += stride;
                    break;
                } else if (nbuf > 0 && (!reading || !have || (nbuf == cap && read_ticks - (now - start) > flush_ticks))) {
                    // write phase, no tile left, or a full buffer with more than flush_ticks of the read
                    // phase left (with less, a short sleep costs less than writes amid the reads)
                    flush(nbuf);
                    nbuf = 0;
                    fresh = true;
                } else if (!have) {
                    return; // no tile left and the buffer is empty
                } else {
                    __builtin_amdgcn_s_sleep(1); // empty buffer in a write phase (or full in a read phase)
                    fresh = true;
                }
            }
        }
    }
}

// Store the packed codes of a tile (element lane el owns bytes
// [el*E*BITS/8, ...)): one 16-byte chunk per lane goes out directly; more
// go through the wave's LDS region so that every store instruction writes
// 1 KiB contiguous.
template <int E, int BITS>
SDP4_DEV void store_codes(uint8_t *__restrict__ dst, int valid, u32x4 *lds, const uint32_t (&q)[E], int el)
{
    if constexpr (E * BITS == 64) { // 16 nibbles or 8 bytes per lane: 512 contiguous bytes per wave
        if (E * el < valid) {
            if constexpr (BITS == 4)
                __builtin_nontemporal_store(u32x2{pack_nibbles8(q), pack_nibbles8(q + 8)},
                                            reinterpret_cast<u32x2 *>(dst) + el);
            else
                __builtin_nontemporal_store(
                    u32x2{pack_bytes4(q[0], q[1], q[2], q[3]), pack_bytes4(q[4], q[5], q[6], q[7])},
                    reinterpret_cast<u32x2 *>(dst) + el);
        }
    } else {
        constexpr int RC = E * BITS / 128; // 16-byte chunks per lane
        u32x4 pk[RC];
        if constexpr (BITS == 8)
            pack8<E>(q, pk);
        else
            pack4<E>(q, pk);
        if constexpr (RC == 1) {
            if (E * el < valid)
                __builtin_nontemporal_store(pk[0], reinterpret_cast<u32x4 *>(dst) + el);
        } else {
            stage_out<RC>(reinterpret_cast<u32x4 *>(dst), valid * BITS / 128, lds, pk, el);
        }
    }
}

template <int E, int BITS>
SDP4_DEV void store_codes(uint8_t *__restrict__ dst, int valid, u32x4 *lds, const uint32_t (&q)[E])
{
    store_codes<E, BITS>(dst, valid, lds, q, lane_id());
}

template <int E, int NB>
SDP4_DEV void maybe_fwht(float (&v)[E], float cn)
{
    if constexpr (NB > 1)
        fwht_lane<E, NB>(v, cn);
}

// Fused transform of a kernel whose lanes follow element_lane when blocks
// span several lanes (NB > E); within one lane, the plain transform.
template <int E, int NB>
SDP4_DEV void fused_fwht(float (&v)[E], float cn, int el)
{
    if constexpr (NB > E)
        fwht_lane_signed<E, NB>(v, cn, el);
    else
        maybe_fwht<E, NB>(v, cn);
}

// ---------------------------------------------------------------------------
// qWD encode: d = w_new - widen(w_prev); 4-bit codes per group, asymmetric
// (codes 0..15, scale and minimum) or, with SYM, symmetric (codes -7..7,
// scale only; minv is not touched)
// ---------------------------------------------------------------------------
template <bool BF16, bool SYM, int E, int DEPTH, int WPB, int PMIN = 128, bool PHASE = true>
__global__ __launch_bounds__(kWave * WPB) void k_qwd_encode(
    const float *__restrict__ w_new, const void *__restrict__ w_prev, int64_t n, int group,
    uint8_t *__restrict__ codes, float *__restrict__ scale, float *__restrict__ minv, uint64_t period,
    uint64_t read_ticks)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;                       // f32 chunks per lane
    constexpr int RP = BF16 ? E / 8 : E / 4;       // previous-weight chunks per lane
    // Phased mode (E = 32: one 16-byte code chunk per lane and tile) buffers
    // CAP tiles per wave: codes, then scales and minima of up to HMAX groups
    // (groups of at least PMIN elements).  PHASE = false: the streaming form
    // only, without the buffers' LDS (so that more blocks fit a CU).
    constexpr bool PHASED = E == 32 && PHASE;
    constexpr int CAP = PHASED ? enc_phase_cap(PMIN) : 1;
    constexpr int HMAX = W / PMIN;
    // inputs of 8 chunks per lane pass through the LDS in two halves
    constexpr bool HALFT = SDP4_ENC_HALF_T && R == 8;
    __shared__ u32x4 lds_all[WPB][kWave * (HALFT ? R / 2 : R)];
    __shared__ u32x4 cbuf_all[PHASED ? WPB : 1][PHASED ? CAP * kWave : 1];
    __shared__ float hbuf_all[PHASED ? WPB : 1][PHASED ? CAP * 2 * HMAX : 1];
    __shared__ int64_t tbuf_all[PHASED ? WPB : 1][PHASED ? CAP : 1];
    const int wv = threadIdx.x / kWave;
    u32x4 *lds = lds_all[wv];
    const int lane = lane_id();
    const int gs = group_shift(group);
    const int lanes_per_group = group / E;
    const int off = E * lane;
    struct Tile {
        u32x4 a[R];
        u32x4 b[RP];
    };
    auto load = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        const int valid = tile_valid(n, base, W);
        gload<R>(reinterpret_cast<const u32x4 *>(w_new + base), valid / 4, in.a);
        if constexpr (BF16)
            gload<RP>(reinterpret_cast<const u32x4 *>(static_cast<const uint16_t *>(w_prev) + base), valid / 8,
                      in.b);
        else
            gload<RP>(reinterpret_cast<const u32x4 *>(static_cast<const float *>(w_prev) + base), valid / 4,
                      in.b);
    };
    // d = w_new - widen(w_prev), the group parameters (scale s, minimum mn;
    // SYM: mn = 0, unused) and the code bits of this lane's E elements.
    auto quantize = [&](Tile &in, uint32_t (&q)[E], float &s, float &mn) {
        float d[E], p[E];
        {
            u32x4 c[R];
            if constexpr (HALFT)
                transpose_in_halves<R>(in.a, lds, c);
            else
                transpose_in<R>(in.a, lds, c);
            chunks_to_f32<E>(c, d);
        }
        {
            u32x4 c[RP];
            if constexpr (HALFT && RP == R)
                transpose_in_halves<RP>(in.b, lds, c);
            else
                transpose_in<RP>(in.b, lds, c);
            if constexpr (BF16)
                bf16_chunks_to_f32<E>(c, p);
            else
                chunks_to_f32<E>(c, p);
        }
#pragma unroll
        for (int i = 0; i < E; ++i)
            d[i] = d[i] - p[i];
        if constexpr (SYM) {
            float a = 0.0f;
#pragma unroll
            for (int i = 0; i < E; ++i)
                a = fmaxf(a, fabsf(d[i]));
            max_lanes(a, lanes_per_group);
            float inv;
            sym_params(a, 7.0f, s, inv);
            mn = 0.0f;
#pragma unroll
            for (int i = 0; i < E; ++i)
                q[i] = code_bits(d[i], inv);
        } else {
            mn = d[0];
            float mx = d[0];
#pragma unroll
            for (int i = 1; i < E; ++i) {
                mn = fminf(mn, d[i]);
                mx = fmaxf(mx, d[i]);
            }
            minmax_lanes(mn, mx, lanes_per_group);
            const float range = mx - mn;
            const float r = 15.0f / range;
            const bool degenerate = !(range > 0.0f) || !__builtin_isfinite(range) || !__builtin_isfinite(r);
            s = degenerate ? 0.0f : range / 15.0f;
            const float inv = degenerate ? 0.0f : r;
#pragma unroll
            for (int i = 0; i < E; ++i)
                q[i] = code_bits(d[i] - mn, inv);
        }
    };
    const int64_t ntiles = (n + W - 1) / W;
    if (!PHASED || period == 0) { // ordinary stream: each tile's output is stored at once
        (void)cbuf_all;
        (void)hbuf_all;
        (void)tbuf_all;
        auto proc = [&](int64_t t, Tile &in) {
            const int64_t base = t * W;
            const int valid = tile_valid(n, base, W);
            uint32_t q[E];
            float s, mn;
            quantize(in, q, s, mn);
            store_codes<E, 4>(codes + base / 2, valid, lds, q);
            if (off < valid && (off & (group - 1)) == 0) {
                const int64_t gi = (base + off) >> gs;
                scale[gi] = s;
                if constexpr (!SYM)
                    minv[gi] = mn;
            }
        };
        tile_loop<DEPTH, WPB, Tile>(ntiles, load, proc);
        return;
    }
    if constexpr (PHASED) { // group >= PMIN (the launcher checks)
        u32x4 *cbuf = cbuf_all[wv];
        float *hbuf = hbuf_all[wv];
        int64_t *tbuf = tbuf_all[wv];
        auto proc = [&](int64_t t, Tile &in, int slot) {
            uint32_t q[E];
            float s, mn;
            quantize(in, q, s, mn);
            u32x4 pk[1];
            pack4<E>(q, pk);
            cbuf[slot * kWave + lane] = pk[0];
            if ((off & (group - 1)) == 0) {
                const int g = off >> gs; // group within the tile, < W / group <= HMAX
                hbuf[slot * 2 * HMAX + g] = s;
                hbuf[slot * 2 * HMAX + HMAX + g] = mn;
            }
            if (lane == 0)
                tbuf[slot] = t;
        };
        auto flush = [&](int k) {
            wave_lds_sync();
            const int hl = W >> gs; // headers per tile
            for (int j = 0; j < k; ++j) {
                const int64_t base = tbuf[j] * W;
                const int valid = tile_valid(n, base, W);
                if (off < valid)
                    __builtin_nontemporal_store(cbuf[j * kWave + lane],
                                                reinterpret_cast<u32x4 *>(codes + base / 2) + lane);
                if (lane < hl && (lane << gs) < valid) {
                    const int64_t gi = (base >> gs) + lane;
                    scale[gi] = hbuf[j * 2 * HMAX + lane];
                    if constexpr (!SYM)
                        minv[gi] = hbuf[j * 2 * HMAX + HMAX + lane];
                }
            }
            wave_lds_sync();
        };
        // early loads measured faster with float32 model weights only
        constexpr bool EARLY = BF16 ? SDP4_ENC_EARLY_LOAD_BF16 : SDP4_ENC_EARLY_LOAD_F32;
        // a buffer that fills with more than SDP4_ENC_FLUSH_PCT per cent of the period left to read is
        // written out at once
        const uint64_t flush_ticks = period * SDP4_ENC_FLUSH_PCT / 100;
        phased_tile_loop<kEncPhaseDepth, WPB, EARLY, Tile>(ntiles, CAP, period, read_ticks, flush_ticks, load, proc,
                                                           flush);
    }
}

// ---------------------------------------------------------------------------
// qWD decode: w_prev <- narrow(widen(w_prev) + value) with value =
// fma(code, scale, min), or with SYM value = code * scale (signed codes,
// minv not read)
// ---------------------------------------------------------------------------
template <bool BF16, bool SYM, int E, int DEPTH, int WPB>
__global__ __launch_bounds__(kWave * WPB) void k_qwd_decode(
    const uint8_t *__restrict__ codes, const float *__restrict__ scale,
    const float *__restrict__ minv, int64_t n, int group, void *__restrict__ w_prev)
{
    static_assert(E == 8 || E == 16 || E % 32 == 0, "lane slice");
    constexpr int W = kWave * E;
    constexpr int RP = BF16 ? E / 8 : E / 4;   // 16-byte chunks of weights per lane
    constexpr int CWD = E / 8;                 // 32-bit words of codes per lane
    __shared__ u32x4 lds_all[WPB][kWave * (E / 4)];
    u32x4 *lds = lds_all[threadIdx.x / kWave];
    const int lane = lane_id();
    const int gs = group_shift(group);
    struct Tile {
        uint32_t c[CWD];
        float s, mn;
        u32x4 w[RP];
    };
    auto load = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        const int valid = tile_valid(n, base, W);
        const int off = E * lane;
        if (off < valid) {
            const uint8_t *src = codes + (base + off) / 2;
            if constexpr (CWD >= 4) {
#pragma unroll
                for (int k = 0; k < CWD / 4; ++k) {
                    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src) + k);
                    in.c[4 * k] = v.x;
                    in.c[4 * k + 1] = v.y;
                    in.c[4 * k + 2] = v.z;
                    in.c[4 * k + 3] = v.w;
                }
            } else if constexpr (CWD == 2) {
                const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(src));
                in.c[0] = v.x;
                in.c[1] = v.y;
            } else {
                in.c[0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(src));
            }
            const int64_t gi = (base + off) >> gs;
            in.s = scale[gi];
            in.mn = SYM ? 0.0f : minv[gi];
        } else {
#pragma unroll
            for (int k = 0; k < CWD; ++k)
                in.c[k] = 0u;
            in.s = 0.0f;
            in.mn = 0.0f;
        }
        if constexpr (BF16)
            gload<RP>(reinterpret_cast<const u32x4 *>(static_cast<const uint16_t *>(w_prev) + base), valid / 8,
                      in.w);
        else
            gload<RP>(reinterpret_cast<const u32x4 *>(static_cast<const float *>(w_prev) + base), valid / 4,
                      in.w);
    };
    auto proc = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        const int valid = tile_valid(n, base, W);
        float w[E];
        u32x4 c[RP];
        transpose_in<RP>(in.w, lds, c);
        if constexpr (BF16)
            bf16_chunks_to_f32<E>(c, w);
        else
            chunks_to_f32<E>(c, w);
#pragma unroll
        for (int k = 0; k < CWD; ++k) { // word k: the nibbles of elements 8k .. 8k+7, even ones low
            const uint32_t word = in.c[k];
            if constexpr (SYM) {
#pragma unroll
                for (int m = 0; m < 8; ++m) {
                    const float code = (float)((int32_t)(word << (28 - 4 * m)) >> 28);
                    const float value = code * in.s;
                    w[8 * k + m] = w[8 * k + m] + value;
                }
            } else {
                // byte j of lo / hi: the code of element 8k + 2j / 8k + 2j + 1
                const uint32_t lo = word & 0x0F0F0F0Fu, hi = (word >> 4) & 0x0F0F0F0Fu;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float c0 = (float)((lo >> (8 * j)) & 0xFFu), c1 = (float)((hi >> (8 * j)) & 0xFFu);
                    w[8 * k + 2 * j] = w[8 * k + 2 * j] + __builtin_fmaf(c0, in.s, in.mn);
                    w[8 * k + 2 * j + 1] = w[8 * k + 2 * j + 1] + __builtin_fmaf(c1, in.s, in.mn);
                }
            }
        }
        if constexpr (BF16) {
            f32_to_bf16_chunks<E>(w, c);
            stage_out<RP>(reinterpret_cast<u32x4 *>(static_cast<uint16_t *>(w_prev) + base), valid / 8, lds, c);
        } else {
            f32_to_chunks<E>(w, c);
            stage_out<RP>(reinterpret_cast<u32x4 *>(static_cast<float *>(w_prev) + base), valid / 4, lds, c);
        }
    };
    tile_loop<DEPTH, WPB, Tile>((n + W - 1) / W, load, proc);
}

// ---------------------------------------------------------------------------
// K1: blockwise Hadamard (block NB, 0 = none) + symmetric BITS-bit group quantization
// ---------------------------------------------------------------------------
template <int BITS, int E, int NB, int DEPTH, int WPB, bool SR = false>
__global__ __launch_bounds__(kWave * WPB) void k_grad_quant(
    const float *__restrict__ x, int64_t n, int group, float cn, uint8_t *__restrict__ codes,
    float *__restrict__ scale, uint64_t seed = 0, uint64_t offset = 0)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    constexpr float qmax = BITS == 8 ? 127.0f : 7.0f;
    __shared__ u32x4 lds_all[WPB][kWave * R];
    u32x4 *lds = lds_all[threadIdx.x / kWave];
    const int lane = lane_id();
    const int el = NB > E ? element_lane(lane) : lane; // element lane of this lane
    const int off = E * el;
    const int gs = group_shift(group);
    const int lanes_per_group = group / E;
    struct Tile {
        u32x4 a[R];
    };
    auto load = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        gload<R>(reinterpret_cast<const u32x4 *>(x + base), tile_valid(n, base, W) / 4, in.a);
    };
    auto proc = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        const int valid = tile_valid(n, base, W);
        float v[E];
        {
            u32x4 c[R];
            transpose_in<R>(in.a, lds, c, el);
            chunks_to_f32<E>(c, v);
        }
        fused_fwht<E, NB>(v, cn, el);
        float a = 0.0f;
#pragma unroll
        for (int i = 0; i < E; ++i)
            a = fmaxf(a, fabsf(v[i]));
        max_lanes(a, lanes_per_group);
        float s, inv;
        sym_params(a, qmax, s, inv);
        uint32_t q[E];
        if constexpr (SR) {
            float u[E];
            sr_uniforms<E>(seed, offset + (uint64_t)(base + off), u);
#pragma unroll
            for (int i = 0; i < E; ++i)
                q[i] = code_bits_sr(v[i], inv, u[i], qmax);
        } else {
#pragma unroll
            for (int i = 0; i < E; ++i)
                q[i] = code_bits(v[i], inv);
        }
        store_codes<E, BITS>(codes + base * BITS / 8, valid, lds, q, el);
        if (off < valid && (off & (group - 1)) == 0)
            scale[(base + off) >> gs] = s;
    };
    tile_loop<DEPTH, WPB, Tile>((n + W - 1) / W, load, proc);
}

// ---------------------------------------------------------------------------
// K2 / K3: dequantize + reduce over P <= PMAX chunks, then re-quantize
// (BITS_OUT 4/8) or inverse Hadamard (block NB) + out_scale to float32
// (BITS_OUT 0)
// ---------------------------------------------------------------------------
template <int BITS_IN, int BITS_OUT, int E, int NB, int PMAX, int DEPTH, int WPB, bool SR = false>
__global__ __launch_bounds__(kWave * WPB) void k_dequant_reduce(
    PeerTable peers, int P, int64_t n, int group, float cn, float out_scale, uint8_t *__restrict__ out_codes,
    float *__restrict__ out_scales, float *__restrict__ out_f32, uint64_t seed = 0, uint64_t offset = 0)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    // input chunks (16 B) per lane per peer; HALF: 8 bytes (16 elements of 4-bit codes), kept in a
    // chunk's first two words
    constexpr bool HALF = E * BITS_IN == 64;
    constexpr int CW = HALF ? 1 : E * BITS_IN / 128;
    __shared__ u32x4 lds_all[WPB][kWave * R];
    u32x4 *lds = lds_all[threadIdx.x / kWave];
    const int lane = lane_id();
    // element lane: relabeled when the fused inverse transform spans lanes
    const int el = (BITS_OUT == 0 && NB > E) ? element_lane(lane) : lane;
    const int off = E * el;
    const int gs = group_shift(group);
    struct Tile {
        u32x4 c[PMAX][CW];
        float s[PMAX];
    };
    auto load = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        const bool active = off < tile_valid(n, base, W);
        const int64_t gi = (base + off) >> gs;
#pragma unroll
        for (int j = 0; j < PMAX; ++j) {
            if constexpr (SDP4_PEER_LDS && CW > 1) {
                if (j < P) {
                    const auto *src = static_cast<const uint8_t *>(peers.codes[j]) + base * BITS_IN / 8;
                    gload<CW, false>(reinterpret_cast<const u32x4 *>(src), tile_valid(n, base, W) * BITS_IN / 128,
                                     in.c[j]);
                    in.s[j] = active ? peers.scales[j][gi] : 0.0f;
                }
                continue;
            }
            if (j < P && active) {
                const uint8_t *src = static_cast<const uint8_t *>(peers.codes[j]) + (base + off) * BITS_IN / 8;
                if constexpr (HALF) {
                    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(src));
                    in.c[j][0] = u32x4{v.x, v.y, 0u, 0u};
                } else {
#pragma unroll
                    for (int k = 0; k < CW; ++k)
                        in.c[j][k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src) + k);
                }
                in.s[j] = peers.scales[j][gi];
            } else {
#pragma unroll
                for (int k = 0; k < CW; ++k)
                    in.c[j][k] = u32x4{0u, 0u, 0u, 0u};
                in.s[j] = 0.0f;
            }
        }
    };
    auto proc = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        const int valid = tile_valid(n, base, W);
        float acc[E];
#pragma unroll
        for (int i = 0; i < E; ++i)
            acc[i] = 0.0f;
#pragma unroll
        for (int j = 0; j < PMAX; ++j) {
            if (j < P) {
                if constexpr (SDP4_PEER_LDS && CW > 1) {
                    u32x4 tmp[CW];
                    transpose_in<CW>(in.c[j], lds, tmp, el);
#pragma unroll
                    for (int k = 0; k < CW; ++k)
                        in.c[j][k] = tmp[k];
                }
                uint32_t w[CW * 4];
#pragma unroll
                for (int k = 0; k < CW; ++k) {
                    w[4 * k] = in.c[j][k].x;
                    w[4 * k + 1] = in.c[j][k].y;
                    w[4 * k + 2] = in.c[j][k].z;
                    w[4 * k + 3] = in.c[j][k].w;
                }
#pragma unroll
                for (int i = 0; i < E; ++i)
                    acc[i] = __builtin_fmaf(code_f<BITS_IN>(w, i), in.s[j], acc[i]);
            }
        }
        if constexpr (BITS_OUT == 0) {
            fused_fwht<E, NB>(acc, cn, el);
            if (out_scale != 1.0f) {
#pragma unroll
                for (int i = 0; i < E; ++i)
                    acc[i] = acc[i] * out_scale;
            }
            u32x4 c[R];
            f32_to_chunks<E>(acc, c);
            stage_out<R>(reinterpret_cast<u32x4 *>(out_f32 + base), valid / 4, lds, c, el);
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
            max_lanes(a, group / E);
            float s, inv;
            sym_params(a, qmax, s, inv);
            uint32_t q[E];
            if constexpr (SR) {
                float u[E];
                sr_uniforms<E>(seed, offset + (uint64_t)(base + off), u);
#pragma unroll
                for (int i = 0; i < E; ++i)
                    q[i] = code_bits_sr(acc[i], inv, u[i], qmax);
            } else {
#pragma unroll
                for (int i = 0; i < E; ++i)
                    q[i] = code_bits(acc[i], inv);
            }
            store_codes<E, BITS_OUT>(out_codes + base * BITS_OUT / 8, valid, lds, q);
            if (off < valid && (off & (group - 1)) == 0)
                out_scales[(base + off) >> gs] = s;
        }
    };
    tile_loop<DEPTH, WPB, Tile>((n + W - 1) / W, load, proc);
}

// ---------------------------------------------------------------------------
// standalone Hadamard (unfused variant); in place allowed
// ---------------------------------------------------------------------------
template <int E, int NB, int DEPTH, int WPB>
__global__ __launch_bounds__(kWave * WPB) void k_hadamard(const float *x, float *y, int64_t n, float cn)
{
    constexpr int W = kWave * E;
    constexpr int R = E / 4;
    __shared__ u32x4 lds_all[WPB][kWave * R];
    u32x4 *lds = lds_all[threadIdx.x / kWave];
    struct Tile {
        u32x4 a[R];
    };
    // In place, a prefetched tile is never one a previous iteration wrote
    // (each wave only ever touches its own tiles), so prefetching is safe.
    auto load = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        gload<R>(reinterpret_cast<const u32x4 *>(x + base), tile_valid(n, base, W) / 4, in.a);
    };
    auto proc = [&](int64_t t, Tile &in) {
        const int64_t base = t * W;
        u32x4 c[R];
        transpose_in<R>(in.a, lds, c);
        float v[E];
        chunks_to_f32<E>(c, v);
        fwht_lane<E, NB>(v, cn);
        f32_to_chunks<E>(v, c);
        stage_out<R>(reinterpret_cast<u32x4 *>(y + base), tile_valid(n, base, W) / 4, lds, c);
    };
    tile_loop<DEPTH, WPB, Tile>((n + W - 1) / W, load, proc);
}

// ---------------------------------------------------------------------------
// launch helpers shared by the .hip translation units
// ---------------------------------------------------------------------------
template <int WPB>
int64_t wave_blocks(int64_t n, int E)
{
    const int64_t W = (int64_t)kWave * E;
    const int64_t tiles = (n + W - 1) / W;
    return (tiles + WPB - 1) / WPB;
}

constexpr int kCap = SDP4_BLOCKS_PER_CU;
constexpr int kEncWaves = SDP4_ENC_WAVES, kEncCap = SDP4_ENC_BPC, kEncStreamCap = SDP4_ENC_STREAM_BPC;
constexpr int kK1Waves = SDP4_K1_WAVES, kK1Waves32 = SDP4_K1_WAVES_32, kK1Cap = SDP4_K1_BPC, kK1Cap32 = SDP4_K1_BPC_32;
constexpr int kK1SrCap = SDP4_K1_SR_BPC, kK1Sr16Waves = SDP4_K1_SR16_WAVES, kK1Sr16Cap = SDP4_K1_SR16_BPC;
constexpr int kK1Waves8 = SDP4_K1_WAVES_8, kK1Cap8 = SDP4_K1_BPC_8;
constexpr int kK1PlainWaves = SDP4_K1_WAVES_PLAIN, kK1PlainCap = SDP4_K1_PLAIN_BPC;
constexpr int kHadCap = SDP4_HAD_BPC;
constexpr int kDecWaves = SDP4_DEC_WAVES, kDecCap = SDP4_DEC_BPC;
constexpr int kDecF32Waves = SDP4_DEC_F32_WAVES, kDecF32Cap = SDP4_DEC_F32_BPC;
constexpr int kRqWaves = SDP4_RQ_WAVES, kRqCap = SDP4_RQ_BPC, kRfWaves = SDP4_RF_WAVES, kRfCap = SDP4_RF_BPC;
constexpr int kRq8Waves = SDP4_RQ8_WAVES, kRq8Cap = SDP4_RQ8_BPC, kRq8SrWaves = SDP4_RQ8_SR_WAVES, kRq8SrCap = SDP4_RQ8_SR_BPC;

// 64 elements per lane: required for groups of 4096 (a group must fit one
// wavefront), allowed (preferred_e == 64) for any group of at least 64 (a
// lane slice must not straddle groups); otherwise 32.
inline bool use_wide_lanes(int group, int preferred_e) { return group > 64 * 32 || (preferred_e == 64 && group >= 64); }

// Hadamard block sizes the kernels are compiled for: 0 (none), 2 .. 1024.
template <template <int> class F, typename... A>
int with_block(int nb, A... a)
{
    switch (nb) {
    case 0: return F<0>::run(a...);
    case 2: return F<2>::run(a...);
    case 4: return F<4>::run(a...);
    case 8: return F<8>::run(a...);
    case 16: return F<16>::run(a...);
    case 32: return F<32>::run(a...);
    case 64: return F<64>::run(a...);
    case 128: return F<128>::run(a...);
    case 256: return F<256>::run(a...);
    case 512: return F<512>::run(a...);
    case 1024: return F<1024>::run(a...);
    default: return 1;
    }
}

// Peer counts 1..16: loads of up to 8 peers are batched (and prefetched);
// more than 8 peers use a 16-wide batch without prefetch.
// The re-quantizing variant keeps P chunks per lane in flight already and
// is fastest without the extra prefetch buffer (measured); the float32
// variant prefetches.
template <int BITS_IN, int BITS_OUT, int E, int NB, bool SR = false>
int dr_launch(const PeerTable &peers, int P, int64_t n, int group, float cn, float out_scale,
              uint8_t *out_codes, float *out_scales, float *out_f32, hipStream_t s, uint64_t seed = 0,
              uint64_t offset = 0)
{
    constexpr int pipe = BITS_OUT == 0 ? kDepth : 0;
    constexpr int WPB = BITS_OUT == 0 ? kRfWaves : E == 16 ? (SR ? kRq8SrWaves : kRq8Waves) : kRqWaves;
    constexpr int cap = BITS_OUT == 0 ? kRfCap : E == 16 ? (SR ? kRq8SrCap : kRq8Cap) : kRqCap;
    if (P <= 4)
        return launch<WPB>(k_dequant_reduce<BITS_IN, BITS_OUT, E, NB, 4, pipe, WPB, SR>, wave_blocks<WPB>(n, E), cap,
                           s, peers, P, n, group, cn, out_scale, out_codes, out_scales, out_f32, seed, offset);
    if (P <= 8)
        return launch<WPB>(k_dequant_reduce<BITS_IN, BITS_OUT, E, NB, 8, pipe, WPB, SR>, wave_blocks<WPB>(n, E), cap,
                           s, peers, P, n, group, cn, out_scale, out_codes, out_scales, out_f32, seed, offset);
    return launch<WPB>(k_dequant_reduce<BITS_IN, BITS_OUT, E, NB, 16, 0, WPB, SR>, wave_blocks<WPB>(n, E), cap, s,
                       peers, P, n, group, cn, out_scale, out_codes, out_scales, out_f32, seed, offset);
}

} // namespace sdp4
