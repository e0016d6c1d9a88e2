/*
 * sdp4_oracle.c -- plain, slow, obviously-correct CPU reference of the
 * SDP4Bit per-GPU compression hot path (arXiv 2410.15526).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product (the HIP
 * library) never calls it, and the two share no source: no header, helper,
 * table or constant.
 *
 * Arithmetic rules (build with -O2 -ffp-contract=off, never -ffast-math):
 *   - every float operation is written out and rounds once, to nearest
 *     even, in the order written; fmaf() appears only where the convention
 *     calls for a single-rounding multiply-add;
 *   - rounding to an integer code uses nearbyintf() under the default
 *     round-to-nearest-even mode;
 *   - groups and Hadamard blocks are processed one after another, elements
 *     in index order.
 *
 * Readings of the paper that this file fixes (the paper is silent on them):
 *   - s in the quantizer of Sec. 2.2 is the largest magnitude of the group;
 *   - code = round(x * inv), inv = fl(qmax / s), stored scale = fl(s / qmax);
 *     a group whose s is 0 (or whose inv is not finite) gets scale 0 and
 *     all-zero codes;
 *   - the weight-difference quantizer is asymmetric min-max 4-bit, codes
 *     0..15, header (scale, min), value = fmaf(code, scale, min);
 *   - the Hadamard smoother is the Sylvester matrix scaled by 1/sqrt(n)
 *     (symmetric, orthogonal and its own inverse), applied by the butterfly
 *     with stage widths 1, 2, 4, ..., n/2 and one scaling at the end;
 *   - dequantize-and-reduce sums peers in index order with one fmaf per
 *     peer, starting from +0;
 *   - packing: int8 codes one per byte; 4-bit codes two per byte, even
 *     element in the low nibble, signed codes as two's-complement nibbles.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define REF_OK 0
#define REF_EINVAL 1
#define REF_ENONFINITE 2

static int is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

static int all_finite(const float *x, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        if (!isfinite(x[i]))
            return 0;
    return 1;
}

const char *sdp4ref_version(void) { return "sdp4ref 1"; }

/* ------------------------------------------------------------------------
 * bfloat16 <-> float32.  Model weights are kept in bfloat16 in the paper's
 * mixed-precision setting (Sec. 5.1 Baselines).
 * ---------------------------------------------------------------------- */

float sdp4ref_bf16_to_f32(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16; /* exact: bfloat16 is the top half of a float32 */
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Round a finite float32 to the nearest bfloat16, ties to the even one.
 * Written as the definition: take the two bfloat16 values that bracket x,
 * compare the exact distances (in double, where both differences are exact)
 * and keep the nearer; on a tie keep the one with an even last bit. */
uint16_t sdp4ref_f32_to_bf16_rne(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    uint16_t lo = (uint16_t)(u >> 16);   /* same sign, magnitude truncated */
    if ((u & 0xFFFFu) == 0)
        return lo;                        /* exactly representable */
    uint16_t hi = (uint16_t)(lo + 1);    /* next magnitude up (may be inf) */
    double ax = fabs((double)x);
    double alo = fabs((double)sdp4ref_bf16_to_f32(lo));
    double ahi = ((hi & 0x7FFFu) == 0x7F80u) ? ldexp(1.0, 128) /* overflow threshold */
                                             : fabs((double)sdp4ref_bf16_to_f32(hi));
    double dlo = ax - alo, dhi = ahi - ax;
    if (dlo < dhi)
        return lo;
    if (dhi < dlo)
        return hi;
    return (lo & 1u) ? hi : lo;
}

/* ------------------------------------------------------------------------
 * Hadamard smoother (Sec. 3.2.2; Alg. 4 first and last step; Sec. 3.3).
 * ---------------------------------------------------------------------- */

/* The float nearest to 1/sqrt(n), from long-double arithmetic. */
float sdp4ref_hadamard_scale(int n)
{
    long double t = 1.0L / sqrtl((long double)n);
    return (float)t;
}

/* In place, for each block of `block` consecutive elements of x[0..n):
 * butterfly stages of width h = 1, 2, 4, ..., block/2 -- pair (i, i+h) with
 * bit h of i clear becomes (a+b, a-b) -- then every element times
 * c = hadamard_scale(block).  The result is (H_block / sqrt(block)) x per
 * block, H the Sylvester matrix H[i][j] = (-1)^popcount(i & j). */
int sdp4ref_fwht(float *x, int64_t n, int block)
{
    if (!x || !is_pow2(block) || block < 2 || n % block)
        return REF_EINVAL;
    const float c = sdp4ref_hadamard_scale(block);
    for (int64_t b0 = 0; b0 < n; b0 += block) {
        float *v = x + b0;
        for (int h = 1; h < block; h <<= 1) {
            for (int i = 0; i < block; ++i) {
                if (i & h)
                    continue;
                float a = v[i], b = v[i + h];
                v[i] = a + b;
                v[i + h] = a - b;
            }
        }
        for (int i = 0; i < block; ++i)
            v[i] = v[i] * c;
    }
    return REF_OK;
}

/* ------------------------------------------------------------------------
 * Symmetric linear group-wise quantizer (Sec. 2.2):
 *   x_int = round(x / s * (2^(k-1) - 1)),  s = max |x| over the group.
 * One int8 per element holds the code; `pre` (optional) receives the float
 * value that was rounded (0 for a degenerate group).
 * ---------------------------------------------------------------------- */
int sdp4ref_quant_sym(const float *x, int64_t n, int group, int bits,
                      int8_t *q, float *scale, float *pre)
{
    if (!x || !q || !scale || group < 1 || n % group || bits < 2 || bits > 8)
        return REF_EINVAL;
    if (!all_finite(x, n))
        return REF_ENONFINITE;
    const float qmax = (float)((1 << (bits - 1)) - 1);
    for (int64_t g0 = 0, gi = 0; g0 < n; g0 += group, ++gi) {
        float s = 0.0f;
        for (int i = 0; i < group; ++i) {
            float m = fabsf(x[g0 + i]);
            if (m > s)
                s = m;
        }
        float inv = qmax / s;
        if (s == 0.0f || !isfinite(inv)) {
            scale[gi] = 0.0f;
            for (int i = 0; i < group; ++i) {
                q[g0 + i] = 0;
                if (pre)
                    pre[g0 + i] = 0.0f;
            }
            continue;
        }
        scale[gi] = s / qmax;
        for (int i = 0; i < group; ++i) {
            float v = x[g0 + i] * inv;
            if (pre)
                pre[g0 + i] = v;
            float r = nearbyintf(v);
            if (r > qmax)
                r = qmax;
            if (r < -qmax)
                r = -qmax;
            q[g0 + i] = (int8_t)r;
        }
    }
    return REF_OK;
}

/* value = code * scale (one rounding). */
int sdp4ref_dequant_sym(const int8_t *q, const float *scale, int64_t n, int group, float *out)
{
    if (!q || !scale || !out || group < 1 || n % group)
        return REF_EINVAL;
    for (int64_t i = 0; i < n; ++i)
        out[i] = (float)q[i] * scale[i / group];
    return REF_OK;
}

/* ------------------------------------------------------------------------
 * Asymmetric min-max 4-bit group quantizer for weight differences (qWD,
 * Sec. 3.1): 16 levels spread evenly over [min, max] of each group.
 * ---------------------------------------------------------------------- */
int sdp4ref_quant_asym4(const float *x, int64_t n, int group,
                        uint8_t *q, float *scale, float *minv, float *pre)
{
    if (!x || !q || !scale || !minv || group < 1 || n % group)
        return REF_EINVAL;
    if (!all_finite(x, n))
        return REF_ENONFINITE;
    for (int64_t g0 = 0, gi = 0; g0 < n; g0 += group, ++gi) {
        float mn = x[g0], mx = x[g0];
        for (int i = 1; i < group; ++i) {
            float v = x[g0 + i];
            if (v < mn)
                mn = v;
            if (v > mx)
                mx = v;
        }
        float range = mx - mn;
        float inv = 15.0f / range;
        minv[gi] = mn;
        if (range == 0.0f || !isfinite(range) || !isfinite(inv)) {
            scale[gi] = 0.0f;
            for (int i = 0; i < group; ++i) {
                q[g0 + i] = 0;
                if (pre)
                    pre[g0 + i] = 0.0f;
            }
            continue;
        }
        scale[gi] = range / 15.0f;
        for (int i = 0; i < group; ++i) {
            float t = x[g0 + i] - mn;
            float v = t * inv;
            if (pre)
                pre[g0 + i] = v;
            float r = nearbyintf(v);
            if (r > 15.0f)
                r = 15.0f;
            if (r < 0.0f)
                r = 0.0f;
            q[g0 + i] = (uint8_t)r;
        }
    }
    return REF_OK;
}

/* value = fmaf(code, scale, min) (one rounding). */
int sdp4ref_dequant_asym4(const uint8_t *q, const float *scale, const float *minv,
                          int64_t n, int group, float *out)
{
    if (!q || !scale || !minv || !out || group < 1 || n % group)
        return REF_EINVAL;
    for (int64_t i = 0; i < n; ++i)
        out[i] = fmaf((float)q[i], scale[i / group], minv[i / group]);
    return REF_OK;
}

/* ------------------------------------------------------------------------
 * Packing of codes into bytes.
 * ---------------------------------------------------------------------- */

/* byte j = low nibble of code 2j | low nibble of code 2j+1 << 4 */
int sdp4ref_pack4(const int8_t *codes, int64_t n, uint8_t *packed)
{
    if (!codes || !packed || n % 2)
        return REF_EINVAL;
    for (int64_t j = 0; j < n / 2; ++j) {
        unsigned lo = (unsigned)(uint8_t)codes[2 * j] & 0xFu;
        unsigned hi = (unsigned)(uint8_t)codes[2 * j + 1] & 0xFu;
        packed[j] = (uint8_t)(lo | (hi << 4));
    }
    return REF_OK;
}

/* inverse of pack4; is_signed selects two's-complement nibbles (-8..7)
 * or plain 0..15 */
int sdp4ref_unpack4(const uint8_t *packed, int64_t n, int is_signed, int8_t *codes)
{
    if (!codes || !packed || n % 2)
        return REF_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        int v = (packed[i / 2] >> (4 * (i % 2))) & 0xF;
        if (is_signed && v >= 8)
            v -= 16;
        codes[i] = (int8_t)v;
    }
    return REF_OK;
}

static int codes_ok(int bits) { return bits == 4 || bits == 8; }

/* ------------------------------------------------------------------------
 * qWD encode (Alg. 2, forward pass: d[p] = w_main[p] - w_model[p], then
 * QuantizeWeightsDiff).  prev_is_bf16 selects bfloat16 model weights
 * (uint16 bit patterns) instead of float32; widening is exact.
 * codes: n/2 packed bytes; scale, minv: n/group floats each.
 * ---------------------------------------------------------------------- */
int sdp4ref_qwd_encode(const float *w_new, const void *w_prev, int prev_is_bf16,
                       int64_t n, int group, uint8_t *codes, float *scale, float *minv,
                       float *pre)
{
    if (!w_new || !w_prev || !codes || !scale || !minv || group < 2 || n % group || group % 2)
        return REF_EINVAL;
    float *d = malloc(sizeof(float) * (size_t)(n ? n : 1));
    uint8_t *q = malloc((size_t)(n ? n : 1));
    if (!d || !q) {
        free(d);
        free(q);
        return REF_EINVAL;
    }
    for (int64_t i = 0; i < n; ++i) {
        float prev = prev_is_bf16 ? sdp4ref_bf16_to_f32(((const uint16_t *)w_prev)[i])
                                  : ((const float *)w_prev)[i];
        d[i] = w_new[i] - prev;
    }
    int rc = sdp4ref_quant_asym4(d, n, group, q, scale, minv, pre);
    if (rc == REF_OK)
        rc = sdp4ref_pack4((const int8_t *)q, n, codes);
    free(d);
    free(q);
    return rc;
}

/* qWD decode (Alg. 2: w_model <- w_model + d after the all-gather), in
 * place on the model weights, which double as the "previous" weights
 * (Sec. 3.3 buffer reuse).  bfloat16 weights are narrowed back with
 * round-to-nearest-even after the float32 add. */
int sdp4ref_qwd_decode(const uint8_t *codes, const float *scale, const float *minv,
                       int64_t n, int group, void *w_prev, int prev_is_bf16)
{
    if (!codes || !scale || !minv || !w_prev || group < 2 || n % group || group % 2)
        return REF_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        unsigned c = (codes[i / 2] >> (4 * (i % 2))) & 0xFu;
        float xh = fmaf((float)c, scale[i / group], minv[i / group]);
        if (prev_is_bf16) {
            uint16_t *w = (uint16_t *)w_prev;
            float sum = sdp4ref_bf16_to_f32(w[i]) + xh;
            w[i] = sdp4ref_f32_to_bf16_rne(sum);
        } else {
            float *w = (float *)w_prev;
            w[i] = w[i] + xh;
        }
    }
    return REF_OK;
}

/* ------------------------------------------------------------------------
 * Symmetric qWD: the weight difference of Alg. 2 quantized with the paper's
 * own symmetric quantizer of Sec. 2.2 at 4 bits (codes -7..7 packed as
 * two's-complement nibbles, scale = max|d| / 7 per group, no minimum), the
 * alternative to the asymmetric min-max codec above.
 * codes: n/2 packed bytes; scale: n/group floats.
 * ---------------------------------------------------------------------- */
int sdp4ref_qwd_encode_sym(const float *w_new, const void *w_prev, int prev_is_bf16,
                           int64_t n, int group, uint8_t *codes, float *scale, float *pre)
{
    if (!w_new || !w_prev || !codes || !scale || group < 2 || n % group || group % 2)
        return REF_EINVAL;
    float *d = malloc(sizeof(float) * (size_t)(n ? n : 1));
    int8_t *q = malloc((size_t)(n ? n : 1));
    if (!d || !q) {
        free(d);
        free(q);
        return REF_EINVAL;
    }
    for (int64_t i = 0; i < n; ++i) {
        float prev = prev_is_bf16 ? sdp4ref_bf16_to_f32(((const uint16_t *)w_prev)[i])
                                  : ((const float *)w_prev)[i];
        d[i] = w_new[i] - prev;
    }
    int rc = all_finite(d, n) ? sdp4ref_quant_sym(d, n, group, 4, q, scale, pre) : REF_ENONFINITE;
    if (rc == REF_OK)
        rc = sdp4ref_pack4(q, n, codes);
    free(d);
    free(q);
    return rc;
}

/* Symmetric qWD decode: value = code * scale (one rounding), then the same
 * in-place add and narrowing as sdp4ref_qwd_decode. */
int sdp4ref_qwd_decode_sym(const uint8_t *codes, const float *scale, int64_t n, int group,
                           void *w_prev, int prev_is_bf16)
{
    if (!codes || !scale || !w_prev || group < 2 || n % group || group % 2)
        return REF_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        int c = (codes[i / 2] >> (4 * (i % 2))) & 0xF;
        if (c >= 8)
            c -= 16;
        float xh = (float)c * scale[i / group];
        if (prev_is_bf16) {
            uint16_t *w = (uint16_t *)w_prev;
            float sum = sdp4ref_bf16_to_f32(w[i]) + xh;
            w[i] = sdp4ref_f32_to_bf16_rne(sum);
        } else {
            float *w = (float *)w_prev;
            w[i] = w[i] + xh;
        }
    }
    return REF_OK;
}

/* ------------------------------------------------------------------------
 * Gradient quantization, first level (Alg. 4: g^ <- Hadamard(grad), then
 * Quantize8Bit; with bits = 4 it is the uniform-level 4-bit variant).
 * hadamard_block = 0 skips the transform.  codes: n int8 (bits 8) or n/2
 * packed bytes (bits 4); scale: n/group floats.
 * ---------------------------------------------------------------------- */
int sdp4ref_grad_quant(const float *x, int64_t n, int bits, int hadamard_block, int group,
                       void *codes, float *scale, float *pre)
{
    if (!x || !codes || !scale || !codes_ok(bits) || group < 2 || n % group)
        return REF_EINVAL;
    if (hadamard_block && (n % hadamard_block || !is_pow2(hadamard_block) || hadamard_block < 2))
        return REF_EINVAL;
    float *y = malloc(sizeof(float) * (size_t)(n ? n : 1));
    int8_t *q = malloc((size_t)(n ? n : 1));
    if (!y || !q) {
        free(y);
        free(q);
        return REF_EINVAL;
    }
    memcpy(y, x, sizeof(float) * (size_t)n);
    int rc = hadamard_block ? sdp4ref_fwht(y, n, hadamard_block) : REF_OK;
    if (rc == REF_OK)
        rc = sdp4ref_quant_sym(y, n, group, bits, q, scale, pre);
    if (rc == REF_OK) {
        if (bits == 8)
            memcpy(codes, q, (size_t)n);
        else
            rc = sdp4ref_pack4(q, n, (uint8_t *)codes);
    }
    free(y);
    free(q);
    return rc;
}

/* Code i of a buffer of `bits`-bit signed codes. */
static int code_at(const void *codes, int64_t i, int bits)
{
    if (bits == 8)
        return ((const int8_t *)codes)[i];
    int v = (((const uint8_t *)codes)[i / 2] >> (4 * (i % 2))) & 0xF;
    return v >= 8 ? v - 16 : v;
}

/* ------------------------------------------------------------------------
 * Dequantize + Reduction over P received chunks (Alg. 4, after each
 * all-to-all), then either re-quantization (bits_out = 4 or 8: the 4-bit
 * inter-node step; no Hadamard here, Sec. 3.3 removes it) or a float32
 * result (bits_out = 0) with the inverse Hadamard (hadamard_block > 0; the
 * transform is its own inverse) and an optional final factor out_scale.
 *
 * r[i] = +0; r[i] = fmaf(code_p[i], scale_p[i / group], r[i]) for p = 0..P-1.
 * out_f32 (optional when bits_out > 0) receives r, or the final result.
 * ---------------------------------------------------------------------- */
int sdp4ref_dequant_reduce(int P, const void *const *codes, const float *const *scales,
                           int64_t n_chunk, int bits_in, int group, int bits_out,
                           int hadamard_block, float out_scale, void *out_codes,
                           float *out_scales, float *out_f32, float *pre)
{
    if (P < 1 || !codes || !scales || !codes_ok(bits_in) || group < 2 || n_chunk % group)
        return REF_EINVAL;
    if (bits_out != 0 && !codes_ok(bits_out))
        return REF_EINVAL;
    if (bits_out && (hadamard_block || !out_codes || !out_scales))
        return REF_EINVAL;
    if (!bits_out && !out_f32)
        return REF_EINVAL;
    if (hadamard_block && (n_chunk % hadamard_block || !is_pow2(hadamard_block) || hadamard_block < 2))
        return REF_EINVAL;
    for (int p = 0; p < P; ++p)
        if (!codes[p] || !scales[p])
            return REF_EINVAL;
    float *r = malloc(sizeof(float) * (size_t)(n_chunk ? n_chunk : 1));
    if (!r)
        return REF_EINVAL;
    for (int64_t i = 0; i < n_chunk; ++i) {
        float acc = 0.0f;
        for (int p = 0; p < P; ++p)
            acc = fmaf((float)code_at(codes[p], i, bits_in), scales[p][i / group], acc);
        r[i] = acc;
    }
    int rc = REF_OK;
    if (bits_out) {
        if (out_f32)
            memcpy(out_f32, r, sizeof(float) * (size_t)n_chunk);
        int8_t *q = malloc((size_t)(n_chunk ? n_chunk : 1));
        if (!q) {
            free(r);
            return REF_EINVAL;
        }
        rc = sdp4ref_quant_sym(r, n_chunk, group, bits_out, q, out_scales, pre);
        if (rc == REF_OK) {
            if (bits_out == 8)
                memcpy(out_codes, q, (size_t)n_chunk);
            else
                rc = sdp4ref_pack4(q, n_chunk, (uint8_t *)out_codes);
        }
        free(q);
    } else {
        if (hadamard_block)
            rc = sdp4ref_fwht(r, n_chunk, hadamard_block);
        if (out_scale != 1.0f)
            for (int64_t i = 0; i < n_chunk; ++i)
                r[i] = r[i] * out_scale;
        memcpy(out_f32, r, sizeof(float) * (size_t)n_chunk);
    }
    free(r);
    return rc;
}

/* ------------------------------------------------------------------------
 * Pieces of the unfused pipeline (the paper's "HS w/o fused" variant,
 * Table 4): a standalone transform and a standalone float32 reduction.
 * ---------------------------------------------------------------------- */
int sdp4ref_hadamard(const float *x, float *y, int64_t n, int block)
{
    if (!x || !y)
        return REF_EINVAL;
    if (x != y)
        memmove(y, x, sizeof(float) * (size_t)n);
    return sdp4ref_fwht(y, n, block);
}

/* y[i] = +0 + x_0[i] + x_1[i] + ... in peer order, each sum rounded. */
int sdp4ref_reduce_f32(int P, const float *const *xs, float *y, int64_t n)
{
    if (P < 1 || !xs || !y)
        return REF_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        float acc = 0.0f;
        for (int p = 0; p < P; ++p)
            acc = acc + xs[p][i];
        y[i] = acc;
    }
    return REF_OK;
}

/* ------------------------------------------------------------------------
 * Stochastic rounding for the gradient quantizers.  The convergence
 * analysis (Sec. 4.2, the compressor U_g of Alg. 3 and Definition
 * "unbiased kappa-approximate compressor") assumes an unbiased gradient
 * compressor; rounding the scaled value v up with probability frac(v) makes
 * the symmetric quantizer unbiased.
 *
 * The random numbers come from the counter-based generator Philox4x32 with
 * 10 rounds (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy
 * as 1, 2, 3", SC'11), keyed by a 64-bit seed and indexed by the element
 * position e = offset + i:
 *   counter = (e / 8 low word, e / 8 high word, 0, 0), key = (seed low, seed high),
 *   word    = output[(e / 2) % 4],
 *   u       = (e even ? low half : high half of word) / 65536        in [0, 1),
 *   code    = clamp(floor(fl(fl(x * inv) + u)), -qmax, qmax).
 * ---------------------------------------------------------------------- */

/* One Philox4x32 round: two 32x32->64 products, the halves mixed with the
 * other two counter words and the key. */
static void philox_round(uint32_t c[4], const uint32_t k[2])
{
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k[0];
    const uint32_t n1 = (uint32_t)p1;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k[1];
    const uint32_t n3 = (uint32_t)p0;
    c[0] = n0;
    c[1] = n1;
    c[2] = n2;
    c[3] = n3;
}

void sdp4ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    uint32_t k[2] = {key[0], key[1]};
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { /* key schedule: add the Weyl constants between rounds */
            k[0] += 0x9E3779B9u;
            k[1] += 0xBB67AE85u;
        }
        philox_round(c, k);
    }
    for (int i = 0; i < 4; ++i)
        out[i] = c[i];
}

float sdp4ref_sr_uniform(uint64_t seed, uint64_t e)
{
    const uint64_t blk = e / 8;
    const uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), 0u, 0u};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    sdp4ref_philox4x32_10(ctr, key, out);
    const uint32_t word = out[(e / 2) % 4];
    const uint32_t half = (e % 2) ? (word >> 16) : (word & 0xFFFFu);
    return (float)half / 65536.0f;
}

int sdp4ref_quant_sym_sr(const float *x, int64_t n, int group, int bits, uint64_t seed,
                         uint64_t offset, int8_t *q, float *scale, float *pre)
{
    if (!x || !q || !scale || group < 1 || n % group || bits < 2 || bits > 8)
        return REF_EINVAL;
    if (!all_finite(x, n))
        return REF_ENONFINITE;
    const float qmax = (float)((1 << (bits - 1)) - 1);
    for (int64_t g0 = 0, gi = 0; g0 < n; g0 += group, ++gi) {
        float s = 0.0f;
        for (int i = 0; i < group; ++i) {
            float m = fabsf(x[g0 + i]);
            if (m > s)
                s = m;
        }
        float inv = qmax / s;
        if (s == 0.0f || !isfinite(inv)) {
            scale[gi] = 0.0f;
            for (int i = 0; i < group; ++i) {
                q[g0 + i] = 0;
                if (pre)
                    pre[g0 + i] = 0.0f;
            }
            continue;
        }
        scale[gi] = s / qmax;
        for (int i = 0; i < group; ++i) {
            float v = x[g0 + i] * inv;
            if (pre)
                pre[g0 + i] = v;
            float u = sdp4ref_sr_uniform(seed, offset + (uint64_t)(g0 + i));
            float r = floorf(v + u);
            if (r > qmax)
                r = qmax;
            if (r < -qmax)
                r = -qmax;
            q[g0 + i] = (int8_t)r;
        }
    }
    return REF_OK;
}

/* grad_quant with stochastic rounding: transform (if any), then the
 * stochastically rounded symmetric quantizer; same layouts as grad_quant. */
int sdp4ref_grad_quant_sr(const float *x, int64_t n, int bits, int hadamard_block, int group,
                          uint64_t seed, uint64_t offset, void *codes, float *scale, float *pre)
{
    if (!x || !codes || !scale || !codes_ok(bits) || group < 2 || n % group || offset % 8)
        return REF_EINVAL;
    if (hadamard_block && (n % hadamard_block || !is_pow2(hadamard_block) || hadamard_block < 2))
        return REF_EINVAL;
    float *y = malloc(sizeof(float) * (size_t)(n ? n : 1));
    int8_t *q = malloc((size_t)(n ? n : 1));
    if (!y || !q) {
        free(y);
        free(q);
        return REF_EINVAL;
    }
    memcpy(y, x, sizeof(float) * (size_t)n);
    int rc = hadamard_block ? sdp4ref_fwht(y, n, hadamard_block) : REF_OK;
    if (rc == REF_OK)
        rc = sdp4ref_quant_sym_sr(y, n, group, bits, seed, offset, q, scale, pre);
    if (rc == REF_OK) {
        if (bits == 8)
            memcpy(codes, q, (size_t)n);
        else
            rc = sdp4ref_pack4(q, n, (uint8_t *)codes);
    }
    free(y);
    free(q);
    return rc;
}

/* dequantize-reduce with stochastically rounded re-quantization (bits_out
 * 4 or 8; no transform): the same reduction as sdp4ref_dequant_reduce. */
int sdp4ref_dequant_reduce_sr(int P, const void *const *codes, const float *const *scales,
                              int64_t n_chunk, int bits_in, int group, int bits_out, uint64_t seed,
                              uint64_t offset, void *out_codes, float *out_scales, float *out_f32,
                              float *pre)
{
    if (P < 1 || !codes || !scales || !codes_ok(bits_in) || !codes_ok(bits_out) || group < 2 ||
        n_chunk % group || !out_codes || !out_scales || offset % 8)
        return REF_EINVAL;
    for (int p = 0; p < P; ++p)
        if (!codes[p] || !scales[p])
            return REF_EINVAL;
    float *r = malloc(sizeof(float) * (size_t)(n_chunk ? n_chunk : 1));
    int8_t *q = malloc((size_t)(n_chunk ? n_chunk : 1));
    if (!r || !q) {
        free(r);
        free(q);
        return REF_EINVAL;
    }
    for (int64_t i = 0; i < n_chunk; ++i) {
        float acc = 0.0f;
        for (int p = 0; p < P; ++p)
            acc = fmaf((float)code_at(codes[p], i, bits_in), scales[p][i / group], acc);
        r[i] = acc;
    }
    if (out_f32)
        memcpy(out_f32, r, sizeof(float) * (size_t)n_chunk);
    int rc = sdp4ref_quant_sym_sr(r, n_chunk, group, bits_out, seed, offset, q, out_scales, pre);
    if (rc == REF_OK) {
        if (bits_out == 8)
            memcpy(out_codes, q, (size_t)n_chunk);
        else
            rc = sdp4ref_pack4(q, n_chunk, (uint8_t *)out_codes);
    }
    free(r);
    free(q);
    return rc;
}
