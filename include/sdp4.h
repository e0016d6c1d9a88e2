/*
 * sdp4.h -- C ABI of the MI355X (gfx950) compression hot path of SDP4Bit
 * (Jia et al., "SDP4Bit: Toward 4-bit Communication Quantization in Sharded
 * Data Parallelism for LLM Training", NeurIPS 2024, arXiv 2410.15526).
 *
 * Two per-GPU paths, each a few HIP kernels:
 *   - qWD (Sec. 3.1, Alg. 2): 4-bit group-wise quantization of the weight
 *     difference d = w_main - w_model before the weight all-gather, and the
 *     matching dequantize-and-accumulate into the resident model weights.
 *   - TLq-HS (Sec. 3.2, Alg. 4, Sec. 3.3): blockwise Hadamard transform and
 *     8-bit group quantization before the intra-node all-to-all; dequantize,
 *     reduce over P chunks and re-quantize to 4 bits before the inter-node
 *     all-to-all; dequantize, reduce over Q chunks and apply the inverse
 *     Hadamard transform.
 *
 * Conventions common to every entry point
 * ---------------------------------------
 *  Memory     All array arguments are device pointers (HBM), except the
 *             pointer *tables* of sdp4_dequant_reduce / sdp4_reduce_f32,
 *             which are host arrays of device pointers read during the call
 *             only.  The caller owns every buffer; the library allocates
 *             nothing, frees nothing and keeps no state between calls.
 *             The library sees addresses only: every buffer must hold
 *             the bytes its call touches (given with each entry point);
 *             a shorter one is overrun on the device.
 *  Streams    `stream` is a hipStream_t (NULL = the default stream).  Calls
 *             enqueue their kernels and return; results are visible after
 *             the usual stream synchronization.  Calls are thread-safe.
 *  Errors     Arguments are checked on the host before anything is
 *             enqueued; on any error nothing is written and nothing is
 *             launched.  Device faults surface at the caller's next sync.
 *  Sizes      n / n_chunk count elements and may be 0 (no-op), at most
 *             SDP4_MAX_ELEMENTS.  They must be multiples of
 *             lcm(group, hadamard_block), which for the allowed powers of
 *             two is max(group, hadamard_block).
 *  Alignment  Element arrays (float data, codes) must be 16-byte aligned;
 *             per-group header arrays (scales, minima) 4-byte aligned.
 *  Aliasing   Outputs must not overlap inputs, except where stated.
 *  Inputs     Must be finite; non-finite inputs give unspecified codes.
 *
 * Quantized message layout (identical on the wire and in memory)
 * ---------------------------------------------------------------
 *  8-bit codes: int8, one per element, two's complement, range [-127, 127].
 *  4-bit codes: two per byte, element 2j in the low nibble of byte j and
 *               element 2j+1 in the high nibble.  Gradient codes are signed
 *               two's-complement nibbles in [-7, 7]; weight-difference codes
 *               are unsigned in [0, 15] (signed in [-7, 7] for the
 *               symmetric qWD codec).
 *  Headers:     one float32 per group of `group` consecutive elements, in
 *               group order (scale; plus the group minimum for qWD).
 *  Chunk j of a message of n_chunk elements starts at byte
 *  j * n_chunk * bits / 8 of the codes and at float j * n_chunk / group of
 *  the headers, so a message is split for an all-to-all by pointer
 *  arithmetic alone.
 *
 * Numerics (the paper leaves these unstated; this library fixes them and
 * every kernel follows them exactly, so results are reproducible bit for bit)
 *  - symmetric quantizer (Sec. 2.2), k = 8 or 4 bits, qmax = 2^(k-1) - 1:
 *      s = max |x| over the group, scale = s / qmax, inv = qmax / s,
 *      code = clamp(rint(x * inv), -qmax, qmax), value = code * scale;
 *      a group with s = 0 (or with qmax / s overflowing) has scale 0 and
 *      all-zero codes;
 *  - asymmetric quantizer (qWD): mn, mx = min, max of the group,
 *      R = mx - mn, scale = R / 15, inv = 15 / R,
 *      code = clamp(rint((x - mn) * inv), 0, 15), value = fma(code, scale, mn);
 *      a group with R = 0 has scale 0 and all-zero codes (value = mn);
 *  - Hadamard: per block of n = hadamard_block consecutive elements,
 *      y = (H_n / sqrt(n)) x with H_n the Sylvester matrix
 *      H_n[i][j] = (-1)^popcount(i & j); computed by butterflies of width
 *      1, 2, 4, ..., n/2 followed by one multiplication by the float nearest
 *      to 1/sqrt(n).  The map is symmetric, orthogonal and its own inverse;
 *  - dequantize-reduce: r = +0, then r = fma(code_p, scale_p, r) for
 *      p = 0, 1, ..., P-1 in order;
 *  - bfloat16 model weights are widened exactly and narrowed with
 *      round-to-nearest-even.
 *  All float arithmetic is IEEE binary32 with round-to-nearest-even and no
 *  flush of denormals; division is correctly rounded.
 */
#ifndef SDP4_H
#define SDP4_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
#define SDP4_OK 0
#define SDP4_EINVAL 1 /* null pointer, bad bit width, group, block, dtype, overlap */
#define SDP4_EALIGN 2 /* size not a multiple of lcm(group, block), or pointer misaligned */
#define SDP4_ERANGE 3 /* peer count outside [1, 16] */
#define SDP4_EHIP 4   /* a HIP launch failed; see sdp4_last_hip_error() */

/* Model-weight element types for qWD. */
#define SDP4_F32 0  /* float32 */
#define SDP4_BF16 1 /* bfloat16 stored as uint16 bit patterns */

/* Limits. */
#define SDP4_MIN_GROUP 32
#define SDP4_MAX_GROUP 4096
#define SDP4_MAX_HADAMARD 1024
#define SDP4_MAX_PEERS 16
#define SDP4_MAX_ELEMENTS ((int64_t)1 << 48) /* n above this is EINVAL (byte counts stay in range) */

/*
 * qWD encode -- Alg. 2, CompressedForwardPass, first two steps: the weight
 * difference d = w_main[p] - w_model[p] of this GPU's shard, quantized to
 * 4 bits per group (Sec. 3.1).
 *
 *   w_new   [n] float32        main (optimizer) weights of the shard
 *   w_prev  [n] prev_dtype     model weights as last communicated
 *                              (float32, or bfloat16 bits when SDP4_BF16)
 *   n                          elements; multiple of group
 *   group                      power of two in [32, 4096]
 *   codes   [n/2] uint8        out: packed unsigned 4-bit codes
 *   scale   [n/group] float32  out: (max - min) / 15 of each group
 *   minv    [n/group] float32  out: minimum of each group
 * Inputs are not modified.  Errors: EINVAL (null, bad group or dtype,
 * overlap of an output with an input), EALIGN, EHIP.
 * Large launches (n >= 2^26, group >= 64) pace their memory traffic by the
 * device's constant-rate wall clock: every wave reads in one part of a
 * fixed period and writes its buffered output in the rest.  The outputs do
 * not depend on the timing; other work on the same GPU only slows the call.
 */
int sdp4_qwd_encode(const float *w_new, const void *w_prev, int prev_dtype, int64_t n, int group,
                    uint8_t *codes, float *scale, float *minv, void *stream);

/*
 * qWD decode -- Alg. 2, CompressedForwardPass, w_model <- w_model + d after
 * the all-gather; in place on the model weights, which double as the
 * previous weights so no extra buffer is needed (Sec. 3.3, memory
 * efficiency for weight differences).
 *
 *   codes, scale, minv   a message produced by sdp4_qwd_encode (any shard)
 *   n, group             as for the encoder
 *   w_prev [n] prev_dtype  in/out: w_prev[i] <- narrow(widen(w_prev[i]) + value[i])
 * Errors: EINVAL, EALIGN, EHIP.  w_prev must not overlap the message.
 */
int sdp4_qwd_decode(const uint8_t *codes, const float *scale, const float *minv, int64_t n,
                    int group, void *w_prev, int prev_dtype, void *stream);

/*
 * Symmetric qWD encode -- the weight difference of Alg. 2 quantized with the
 * paper's own symmetric quantizer of Sec. 2.2 at 4 bits instead of the
 * asymmetric min-max codec:
 *      s = max |d| per group, scale = s / 7, inv = 7 / s,
 *      code = clamp(rint(d * inv), -7, 7), value = code * scale;
 *      a group with s = 0 has scale 0 and all-zero codes.
 *
 *   w_new, w_prev, prev_dtype, n, group   as for sdp4_qwd_encode
 *   codes   [n/2] uint8        out: packed two's-complement nibbles
 *                              (even element in the low nibble; -8 unused)
 *   scale   [n/group] float32  out: s / 7 of each group
 * The message is 4 + 32/group bits per element (no minimum).  Inputs are
 * not modified.  Errors: EINVAL, EALIGN, EHIP as for sdp4_qwd_encode, and
 * large launches are paced by the wall clock in the same way.
 */
int sdp4_qwd_encode_sym(const float *w_new, const void *w_prev, int prev_dtype, int64_t n, int group,
                        uint8_t *codes, float *scale, void *stream);

/*
 * Symmetric qWD decode: w_prev[i] <- narrow(widen(w_prev[i]) + code[i] *
 * scale[i / group]) in place (the product and the sum each round once).
 *
 *   codes, scale   a message produced by sdp4_qwd_encode_sym
 *   n, group, w_prev, prev_dtype   as for sdp4_qwd_decode
 * Errors: EINVAL, EALIGN, EHIP.  w_prev must not overlap the message.
 */
int sdp4_qwd_decode_sym(const uint8_t *codes, const float *scale, int64_t n, int group, void *w_prev,
                        int prev_dtype, void *stream);

/*
 * Gradient quantization, first level -- Alg. 4, g^ <- Hadamard(grad) then
 * Quantize8Bit (bits = 8, TLq-HS); bits = 4 gives the uniform-level 4-bit
 * variant (ULq), hadamard_block = 0 the variant without smoother (TLq).
 *
 *   x      [n] float32           gradient (this GPU's full local gradient)
 *   n                            multiple of max(group, hadamard_block)
 *   bits                         8 or 4
 *   hadamard_block               0 (no transform) or a power of two in [2, 1024]
 *   group                        power of two in [32, 4096]
 *   codes  [n*bits/8] bytes      out: int8 codes, or packed signed nibbles
 *   scale  [n/group] float32     out: per-group scale
 * Errors: EINVAL, EALIGN, EHIP.
 */
int sdp4_grad_quant(const float *x, int64_t n, int bits, int hadamard_block, int group, void *codes,
                    float *scale, void *stream);

/*
 * Dequantize + Reduction over P received chunks -- Alg. 4 after each
 * all-to-all -- fused with what follows it on the path:
 *   bits_out = 4 or 8: re-quantization of the reduced values (Quantize4Bit
 *     before the inter-node all-to-all).  No Hadamard transform here: it is
 *     removed by the simplification of Sec. 3.3 (H H = I), so
 *     hadamard_block must be 0.
 *   bits_out = 0: float32 result; with hadamard_block > 0 the inverse
 *     transform (the same transform, Sec. 3.3 moves it past the reduction),
 *     then multiplication by out_scale unless out_scale == 1 (e.g. 1/(P*Q)
 *     to average instead of sum).
 *
 *   P                    number of chunks, 1..16
 *   codes  [P] (host)    device pointers to each chunk's codes (bits_in wide)
 *   scales [P] (host)    device pointers to each chunk's per-group scales
 *   n_chunk              elements per chunk; multiple of max(group, hadamard_block)
 *   bits_in              8 or 4 (signed codes)
 *   group                power of two in [32, 4096], shared by input and output
 *   bits_out             0, 4 or 8
 *   hadamard_block       0 or power of two in [2, 1024] (0 when bits_out > 0)
 *   out_scale            finite factor applied last when bits_out = 0
 *   out_codes  [n_chunk*bits_out/8]   out (bits_out > 0)
 *   out_scales [n_chunk/group] float  out (bits_out > 0)
 *   out_f32    [n_chunk] float32      out: the result when bits_out = 0;
 *                                     optional (may be NULL) when bits_out > 0,
 *                                     then it receives the reduced values
 *                                     before re-quantization
 * Errors: ERANGE (P outside 1..16), EINVAL, EALIGN, EHIP.
 */
int sdp4_dequant_reduce(int P, const void *const *codes, const float *const *scales,
                        int64_t n_chunk, int bits_in, int group, int bits_out, int hadamard_block,
                        float out_scale, void *out_codes, float *out_scales, float *out_f32,
                        void *stream);

/*
 * Stochastically rounded variants of the two gradient quantizers.  The
 * convergence analysis (Sec. 4.2: U_g in Alg. 3 is an unbiased compressor,
 * Definition of the unbiased kappa-approximate compressor) assumes unbiased
 * gradient compression; with stochastic rounding the symmetric quantizer is
 * unbiased: code = clamp(floor(fl(x * inv) + u), -qmax, qmax) with
 * u in [0, 1) drawn per element, so E[code * scale] = x (up to 2^-16 of a
 * quantization step).
 *
 * u of element e = offset + i (i the index within this call) is the 16-bit
 * uniform u = h / 65536, h = half (e % 2: 0 low, 1 high) of word (e / 2) % 4
 * of Philox4x32-10 (Salmon et al., SC'11) with counter (e / 8 as two 32-bit
 * words low first, 0, 0) and key (seed low word, seed high word).  The same
 * (seed, e) always gives the same u, so a buffer quantized in pieces with
 * matching offsets equals the one-call result.
 *
 *   seed     64-bit key of the generator (e.g. derived from the step and rank)
 *   offset   element position of x[0] in the caller's stream; multiple of 8
 * Other arguments, layouts and errors as sdp4_grad_quant / the bits_out > 0
 * mode of sdp4_dequant_reduce (bits_out must be 4 or 8; there is no
 * transform in this mode).  offset not a multiple of 8: EALIGN.
 */
int sdp4_grad_quant_sr(const float *x, int64_t n, int bits, int hadamard_block, int group, uint64_t seed,
                       uint64_t offset, void *codes, float *scale, void *stream);
int sdp4_dequant_reduce_sr(int P, const void *const *codes, const float *const *scales, int64_t n_chunk,
                           int bits_in, int group, int bits_out, uint64_t seed, uint64_t offset,
                           void *out_codes, float *out_scales, float *out_f32, void *stream);

/*
 * Standalone blockwise Hadamard transform (the unfused "HS w/o fused"
 * variant of Table 4, Sec. 5.4): y = (H_n / sqrt(n)) x per block.
 *   x, y [n] float32   y == x (in place) is allowed; partial overlap is not
 *   block              power of two in [2, 1024]; n a multiple of it
 * Errors: EINVAL, EALIGN, EHIP.
 */
int sdp4_hadamard(const float *x, float *y, int64_t n, int block, void *stream);

/*
 * Standalone float32 reduction of P chunks (the Reduction step of Alg. 4
 * for the unfused variant): y[i] = +0 + x_0[i] + ... + x_{P-1}[i], summed
 * in peer order.
 *   xs [P] (host)  device pointers; y [n] must not overlap any of them
 * Errors: ERANGE, EINVAL, EALIGN, EHIP.
 */
int sdp4_reduce_f32(int P, const float *const *xs, float *y, int64_t n, void *stream);

/*
 * Plain device copy y[i] = x[i] (no overlap), the bandwidth yardstick the
 * benchmark measures the hot path against.
 */
int sdp4_copy_f32(const float *x, float *y, int64_t n, void *stream);

/*
 * Read-only stream over x[0..n) (a bandwidth yardstick: the rate HBM gives
 * pure reads).  XOR-accumulates the bit patterns of x[i] into sink[i % 4]:
 *   x    [n] device, 16-byte aligned
 *   sink [4] device uint32, 4-byte aligned, must not overlap x; the caller
 *        clears it first (the call only XORs into it)
 * Errors: EINVAL (null pointer, n < 0 or beyond the limit, overlap), EALIGN,
 * EHIP.
 */
int sdp4_read_f32(const float *x, int64_t n, uint32_t *sink, void *stream);

/*
 * Write-only stream y[i] = value for i in [0, n) (a bandwidth yardstick: the
 * rate HBM gives pure writes).
 *   y [n] device, 16-byte aligned
 * Errors: EINVAL, EALIGN, EHIP.
 */
int sdp4_fill_f32(float *y, int64_t n, float value, void *stream);

/* Pure helpers (no device work). */
int64_t sdp4_codes_bytes(int64_t n, int bits);  /* n * bits / 8, or -1 if bits not 4 or 8 */
int64_t sdp4_num_groups(int64_t n, int group); /* n / group, or -1 if not a valid group */
const char *sdp4_status_string(int status);
const char *sdp4_version(void);
/* HIP error code of the most recent EHIP returned on the calling thread (0 if none). */
int sdp4_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SDP4_H */
