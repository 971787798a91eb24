/*
 * WUSH-KV CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, deliberately unoptimised reference for the online hot path
 * of WUSH-KV ("KV Cache Quantization with Data-Adaptive Transforms").  Only
 * the test suite, the smoke check and the benchmark's CPU-baseline leg load
 * it.  The GPU library never links, includes or calls anything here, and
 * nothing here is derived from the GPU code: the two are written separately
 * from the paper so that agreement between them means something.
 *
 * What each function follows:
 *   orc_append_head  Alg. 2 (inference and cache management), steps 3-4 and
 *                    7-11, with the window rules of Sec. 4.4.
 *   orc_next_quant_end  the S_quant update of Alg. 2 (0-based, exclusive).
 *   orc_quantize_group  Eq. (7): the OSCAR-style percentile-clipped affine
 *                    quantiser used for the end-to-end runs (Sec. 5.3).
 *   orc_quest_quantize_group  Eq. (5): the QuEST projection of Sec. 4.3, the
 *                    quantiser of the paper's analysis (App. B) and of its
 *                    reconstruction-error and perplexity runs (Sec. 5.1-5.2).
 *   orc_dequant      the reconstruction term of Eq. (7).
 *   orc_decode_head  Eq. (2) GQA attention for one query per query head,
 *                    with the query compensation of Eq. (3) (q -> T_K^{-T} q,
 *                    written in row form q^T T_K^{-1}).
 *   orc_attend       softmax attention of one query over S keys (Eq. (2)).
 *
 * Precision.  Transform products and attention are evaluated in fp64.  The
 * quantiser is the exception: its output is integer codes that the GPU must
 * reproduce bit for bit, so it follows one fixed fp32 operation sequence
 * (every operation rounded to nearest-even, no fused multiply-add; build with
 * -ffp-contract=off).  The sequence and every reading of the paper that it
 * needs (interpolation rule of the quantile, tie rule, fp16 scale and zero,
 * zero stored as the clipped minimum, degenerate groups) are listed in the
 * project's design notes and repeated at each function below.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Number formats.  Written from the IEEE-754 definitions; the tests compare */
/* them exhaustively against numpy's float16 and torch's bfloat16 casts.     */
/* ------------------------------------------------------------------------ */

static float f32_from_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t bits_from_f32(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

float orc_bf16_to_f32(uint16_t h) { return f32_from_bits((uint32_t)h << 16); }

/* fp32 -> bf16, round to nearest, ties to even.  bf16 keeps the top 16 bits
 * of the fp32 pattern; the dropped half decides the rounding.  A carry out of
 * the mantissa moves to the next binade (or to infinity), which is correct. */
uint16_t orc_f32_to_bf16(float x)
{
    uint32_t u = bits_from_f32(x);
    if (isnan(x)) return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t hi = u >> 16, dropped = u & 0xFFFFu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (hi & 1u))) hi += 1u;
    return (uint16_t)hi;
}

/* Round a finite non-negative double to the grid {r * q : r integer},
 * ties to even (nearbyint in the default rounding mode). */
static double round_to_grid(double a, double q) { return nearbyint(a / q) * q; }

/* fp64 -> bf16 in one rounding (no detour through fp32, which would round
 * twice).  bf16: 8 significant bits, min normal 2^-126, subnormal spacing
 * 2^-133, max finite (2 - 2^-7) 2^127. */
uint16_t orc_f64_to_bf16(double x)
{
    if (isnan(x)) return 0x7FC0u;
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    double a = fabs(x);
    if (a >= ldexp(2.0 - ldexp(1.0, -8), 127)) return sign | 0x7F80u;
    double q;
    if (a < ldexp(1.0, -126)) q = ldexp(1.0, -133);
    else { int e; frexp(a, &e); q = ldexp(1.0, e - 8); }
    float v = (float)round_to_grid(a, q);          /* exact: v is a bf16 value */
    return sign | (uint16_t)(bits_from_f32(v) >> 16);
}

/* fp32 -> fp16 (binary16), round to nearest, ties to even.  fp16: 11
 * significant bits, min normal 2^-14, subnormal spacing 2^-24, max finite
 * 65504; values at or above 65520 (halfway to 2^16) round to infinity. */
uint16_t orc_f32_to_f16(float x)
{
    uint32_t u = bits_from_f32(x);
    uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
    if (isnan(x)) return sign | 0x7E00u;
    double a = fabs((double)x);
    if (a >= 65520.0) return sign | 0x7C00u;
    if (a < ldexp(1.0, -14)) {
        /* subnormal grid; r == 1024 encodes the smallest normal, 0x0400 */
        double r = nearbyint(a / ldexp(1.0, -24));
        return sign | (uint16_t)r;
    }
    int e;
    frexp(a, &e);                                   /* a in [2^(e-1), 2^e) */
    double v = round_to_grid(a, ldexp(1.0, e - 11));
    int ev;
    double m = frexp(v, &ev);                       /* v = m 2^ev, m in [0.5,1) */
    int biased = (ev - 1) + 15;
    int frac = (int)((m * 2.0 - 1.0) * 1024.0);     /* exact */
    return sign | (uint16_t)(biased << 10) | (uint16_t)frac;
}

float orc_f16_to_f32(uint16_t h)
{
    int s = h >> 15, e = (h >> 10) & 0x1F, m = h & 0x3FF;
    double v;
    if (e == 0) v = ldexp((double)m, -24);
    else if (e == 31) v = m ? NAN : INFINITY;
    else v = ldexp((double)(m + 1024), e - 25);
    return (float)(s ? -v : v);
}

void orc_f32_to_bf16_array(const float *x, uint16_t *y, int64_t n)
{ for (int64_t i = 0; i < n; ++i) y[i] = orc_f32_to_bf16(x[i]); }
void orc_f32_to_f16_array(const float *x, uint16_t *y, int64_t n)
{ for (int64_t i = 0; i < n; ++i) y[i] = orc_f32_to_f16(x[i]); }
void orc_f16_to_f32_array(const uint16_t *x, float *y, int64_t n)
{ for (int64_t i = 0; i < n; ++i) y[i] = orc_f16_to_f32(x[i]); }
void orc_f64_to_bf16_array(const double *x, uint16_t *y, int64_t n)
{ for (int64_t i = 0; i < n; ++i) y[i] = orc_f64_to_bf16(x[i]); }

/* ------------------------------------------------------------------------ */
/* Quantiser, Eq. (7).                                                       */
/* ------------------------------------------------------------------------ */

/* Where the kappa-quantile of d values falls.  The paper does not fix the
 * interpolation rule; we take the linear rule (Hyndman-Fan type 7): with the
 * values sorted ascending a_0..a_{d-1}, pos = kappa (d-1), lo = floor(pos),
 * t = pos - lo, quantile = a_lo + t (a_{lo+1} - a_lo).  pos is formed in fp64
 * from the fp32 kappa, then t is rounded to fp32. */
void orc_kappa_position(float kappa, int d, int32_t *lo, float *t)
{
    double pos = (double)kappa * (double)(d - 1);
    double fl = floor(pos);
    if (fl < 0.0) fl = 0.0;
    if (fl > (double)(d - 1)) fl = (double)(d - 1);
    *lo = (int32_t)fl;
    *t = (float)(pos - fl);
}

static int cmp_float_asc(const void *pa, const void *pb)
{
    float a = *(const float *)pa, b = *(const float *)pb;
    return (a > b) - (a < b);
}

/* kappa-quantile of |x_i| over the d coordinates, as three fp32 operations. */
float orc_quantile_abs(const float *x, int d, int32_t lo, float t)
{
    float a[512];
    for (int i = 0; i < d; ++i) a[i] = fabsf(x[i]);
    qsort(a, (size_t)d, sizeof(float), cmp_float_asc);
    if (lo + 1 < d) {
        float diff = a[lo + 1] - a[lo];
        float prod = t * diff;
        return a[lo] + prod;
    }
    return a[d - 1];
}

/* Quantise one token-head group x[0..d) (fp32 values of bf16 entries) to
 * b-bit codes plus fp16 scale and zero, following Eq. (7):
 *   x_min = max(min_i x_i, -q),  x_max = min(max_i x_i, q),  q = quantile_kappa(|x|)
 *   Delta = (x_max - x_min) / (2^b - 1)
 *   code_i = round-to-nearest((x_i - x_min) / Delta), clamped to [0, 2^b - 1]
 * Readings (the paper leaves them open):
 *   - scale and zero are stored in fp16, and the codes are chosen against the
 *     stored (fp16-rounded) grid;
 *   - the stored offset is the clipped minimum itself ("zero" = x_min), so the
 *     reconstruction Delta (round(x/Delta + z) - z) with z = -x_min/Delta
 *     becomes Delta * code + x_min, one fused multiply-add;
 *   - ties round to even;
 *   - a group whose fp16 step is zero (constant group, or a step that
 *     underflows fp16) gets all codes 0 and reconstructs to the fp16 zero. */
void orc_quantize_group(const float *x, int d, int bits, int32_t lo, float t,
                        uint8_t *codes, uint16_t *s16_out, uint16_t *z16_out)
{
    float q = orc_quantile_abs(x, d, lo, t);
    float mn = x[0], mx = x[0];
    for (int i = 1; i < d; ++i) {
        if (x[i] < mn) mn = x[i];
        if (x[i] > mx) mx = x[i];
    }
    float x_min = (mn > -q) ? mn : -q;
    float x_max = (mx < q) ? mx : q;
    float levels = (float)((1 << bits) - 1);
    float delta = (x_max - x_min) / levels;
    uint16_t s16 = orc_f32_to_f16(delta);
    uint16_t z16 = orc_f32_to_f16(x_min);
    float s = orc_f16_to_f32(s16);
    float z = orc_f16_to_f32(z16);
    float inv = (s > 0.0f) ? 1.0f / s : 0.0f;
    for (int i = 0; i < d; ++i) {
        float y = (x[i] - z) * inv;
        float r = rintf(y);
        if (r < 0.0f) r = 0.0f;
        if (r > levels) r = levels;
        codes[i] = (uint8_t)r;
    }
    *s16_out = s16;
    *z16_out = z16;
}

/* Many groups at once: x [n][d] fp32 -> codes [n][d], params [n][2] (s16, z16). */
void orc_quantize_groups(const float *x, int64_t n, int d, int bits, float kappa,
                         uint8_t *codes, uint16_t *params)
{
    int32_t lo; float t;
    orc_kappa_position(kappa, d, &lo, &t);
    for (int64_t g = 0; g < n; ++g)
        orc_quantize_group(x + g * d, d, bits, lo, t, codes + g * d,
                           params + 2 * g, params + 2 * g + 1);
}

/* Eq. (5), the QuEST projection (Sec. 4.3), for one group x of d values:
 * the step is 2 alpha (2^b - 1)^-1 d^-1/2 ||x||, the code is the floor of
 * x / step clamped to [-2^(b-1), 2^(b-1) - 1], and the reconstruction is the
 * bin centre step (code + 1/2), so the 2^b levels run evenly from -alpha to
 * +alpha times the group's RMS.  Precision (the paper does not fix it):
 *   - ||x||^2 is summed in fp64 over the exact squares; the step is formed
 *     in fp64 as (2 alpha / (2^b - 1)) * sqrt(||x||^2 / d) and rounded once
 *     to fp32, then to the fp16 scale s;
 *   - the code is chosen on the stored grid, from the fp32 product x * (1/s);
 *   - the stored code is u = code + 2^(b-1) in [0, 2^b - 1] and the stored
 *     zero is fp16(s (1/2 - 2^(b-1))) (exact in fp32), so that the common
 *     reconstruction s u + zero is the bin centre s (code + 1/2), up to the
 *     fp16 rounding of the zero;
 *   - the zero group (or a step that underflows fp16) has s = 0: every code
 *     is 2^(b-1) and the reconstruction is 0, matching Q(0) = 0. */
void orc_quest_quantize_group(const float *x, int d, int bits, float alpha,
                              uint8_t *codes, uint16_t *s16_out, uint16_t *z16_out)
{
    double ss = 0.0;
    for (int i = 0; i < d; ++i) ss += (double)x[i] * (double)x[i];
    int h = 1 << (bits - 1);
    double coef = 2.0 * (double)alpha / (double)((1 << bits) - 1);
    float step = (float)(coef * sqrt(ss / (double)d));
    uint16_t s16 = orc_f32_to_f16(step);
    float s = orc_f16_to_f32(s16);
    uint16_t z16 = orc_f32_to_f16(s * (0.5f - (float)h));
    float inv = (s > 0.0f) ? 1.0f / s : 0.0f;
    for (int i = 0; i < d; ++i) {
        float c = floorf(x[i] * inv);
        if (c < (float)-h) c = (float)-h;
        if (c > (float)(h - 1)) c = (float)(h - 1);
        codes[i] = (uint8_t)(int)(c + (float)h);
    }
    *s16_out = s16;
    *z16_out = z16;
}

void orc_quest_quantize_groups(const float *x, int64_t n, int d, int bits, float alpha,
                               uint8_t *codes, uint16_t *params)
{
    for (int64_t g = 0; g < n; ++g)
        orc_quest_quantize_group(x + g * d, d, bits, alpha, codes + g * d,
                                 params + 2 * g, params + 2 * g + 1);
}

/* Reconstruction: scale * code + zero, one rounding to fp32. */
float orc_dequant(uint8_t code, uint16_t s16, uint16_t z16)
{
    return fmaf(orc_f16_to_f32(s16), (float)code, orc_f16_to_f32(z16));
}

/* ------------------------------------------------------------------------ */
/* Cache windows, Sec. 4.4 and Alg. 2.                                       */
/* ------------------------------------------------------------------------ */

static int64_t floor_div(int64_t a, int64_t b)
{
    int64_t q = a / b;
    if ((a % b != 0) && ((a < 0) != (b < 0))) q -= 1;
    return q;
}

/* The S_quant update of Alg. 2, after the cache has grown to s_new entries:
 *   S_start = max(S_quant, S_sink)
 *   S_quant = max(S_quant, S_start + floor((S - S_keep - S_start) / S_flush) * S_flush)
 * The paper counts positions from 1 and treats S_quant as inclusive; with
 * positions counted from 0 the same integer is an exclusive end, so the
 * positions quantised by one update are [S_start, S_quant). */
int32_t orc_next_quant_end(int32_t s_new, int32_t s_quant, int32_t s_sink,
                           int32_t s_keep, int32_t s_flush)
{
    int64_t start = s_quant > s_sink ? s_quant : s_sink;
    int64_t cand = start + floor_div((int64_t)s_new - s_keep - start, s_flush) * s_flush;
    return (int32_t)(cand > s_quant ? cand : s_quant);
}

/* Append n_new tokens to the logical cache of one (sequence, kv-head) and
 * apply the flush rule.  State, all row-major with row = position:
 *   kbits, vbits [cap][d]   bf16 patterns of the transformed key / value
 *   kc, vc       [cap][d]   codes of quantised positions
 *   kp, vp       [cap][2]   fp16 (scale, zero) of quantised positions
 * Step 3 of Alg. 2: k~ = T_K k, evaluated in fp64 from the bf16 inputs and
 * rounded once to bf16; values arrive already transformed (folded weights).
 * Step 4: append at full precision (here bf16).  Steps 7-11: quantise the
 * newly eligible positions from their stored bf16 values, so a token's codes
 * do not depend on whether it is quantised in the call that appends it or in
 * a later one.  Returns the new S_quant. */
int32_t orc_append_head(int d, int bits, int s_sink, int s_keep, int s_flush,
                        int codec, float kappa_k, float kappa_v, float alpha,
                        int32_t s_old, int32_t q_old, int32_t n_new,
                        const uint16_t *k_new, int64_t k_row_stride,
                        const uint16_t *v_new, int64_t v_row_stride,
                        const uint16_t *tk,
                        uint16_t *kbits, uint16_t *vbits,
                        uint8_t *kc, uint16_t *kp, uint8_t *vc, uint16_t *vp)
{
    for (int32_t t = 0; t < n_new; ++t) {
        int64_t p = (int64_t)s_old + t;
        const uint16_t *k = k_new + (int64_t)t * k_row_stride;
        const uint16_t *v = v_new + (int64_t)t * v_row_stride;
        for (int o = 0; o < d; ++o) {
            double acc = 0.0;
            for (int i = 0; i < d; ++i)
                acc += (double)orc_bf16_to_f32(tk[(int64_t)o * d + i]) * (double)orc_bf16_to_f32(k[i]);
            kbits[p * d + o] = orc_f64_to_bf16(acc);
            vbits[p * d + o] = v[o];
        }
    }
    int32_t s_new = s_old + n_new;
    int32_t q_new = orc_next_quant_end(s_new, q_old, s_sink, s_keep, s_flush);
    int32_t start = q_old > s_sink ? q_old : s_sink;
    int32_t lok, lov; float tkf, tvf;
    orc_kappa_position(kappa_k, d, &lok, &tkf);
    orc_kappa_position(kappa_v, d, &lov, &tvf);
    float x[512];
    for (int64_t p = start; p < q_new; ++p) {
        for (int i = 0; i < d; ++i) x[i] = orc_bf16_to_f32(kbits[p * d + i]);
        if (codec == 1)
            orc_quest_quantize_group(x, d, bits, alpha, kc + p * d, kp + 2 * p, kp + 2 * p + 1);
        else
            orc_quantize_group(x, d, bits, lok, tkf, kc + p * d, kp + 2 * p, kp + 2 * p + 1);
        for (int i = 0; i < d; ++i) x[i] = orc_bf16_to_f32(vbits[p * d + i]);
        if (codec == 1)
            orc_quest_quantize_group(x, d, bits, alpha, vc + p * d, vp + 2 * p, vp + 2 * p + 1);
        else
            orc_quantize_group(x, d, bits, lov, tvf, vc + p * d, vp + 2 * p, vp + 2 * p + 1);
    }
    return q_new;
}

/* ------------------------------------------------------------------------ */
/* Attention, Eq. (2) and Eq. (3).                                           */
/* ------------------------------------------------------------------------ */

/* One query against S keys: l_s = scale * q . k_s, p = softmax(l), out = sum_s p_s v_s.
 * K and V are [S][d].  S == 0 gives a zero output. */
void orc_attend(int d, int64_t S, const double *q, const double *K, const double *V,
                double scale, double *out)
{
    for (int j = 0; j < d; ++j) out[j] = 0.0;
    if (S <= 0) return;
    double *l = (double *)malloc((size_t)S * sizeof(double));
    double m = -INFINITY;
    for (int64_t s = 0; s < S; ++s) {
        double dot = 0.0;
        for (int j = 0; j < d; ++j) dot += q[j] * K[s * d + j];
        l[s] = scale * dot;
        if (l[s] > m) m = l[s];
    }
    double z = 0.0;
    for (int64_t s = 0; s < S; ++s) { l[s] = exp(l[s] - m); z += l[s]; }
    for (int64_t s = 0; s < S; ++s)
        for (int j = 0; j < d; ++j) out[j] += l[s] * V[s * d + j];
    for (int j = 0; j < d; ++j) out[j] /= z;
    free(l);
}

/* Key or value of position p as the cache holds it: the bf16 entry for the
 * sink window (p < S_sink) and the recent window (p >= max(S_quant, S_sink)),
 * the exact reconstruction scale * code + zero for the quantised middle. */
static void cached_row(int d, int s_sink, int32_t q_end, int64_t p,
                       const uint16_t *bits16, const uint8_t *codes, const uint16_t *params,
                       double *row)
{
    int32_t qe = q_end > s_sink ? q_end : s_sink;
    if (p >= s_sink && p < qe) {
        double s = (double)orc_f16_to_f32(params[2 * p]);
        double z = (double)orc_f16_to_f32(params[2 * p + 1]);
        for (int j = 0; j < d; ++j) row[j] = s * (double)codes[p * d + j] + z;
    } else {
        for (int j = 0; j < d; ++j) row[j] = (double)orc_bf16_to_f32(bits16[p * d + j]);
    }
}

/* Decode attention of one (sequence, kv-head): G query heads (h, g) read this
 * kv head.  The query of head g is compensated as q~ = q^T T_K^{-1} (fp64 from
 * the bf16 query and the fp32 inverse), then attends to all S cached positions
 * (the decode query sits at position S-1 and sees itself).  out is [G][d] in
 * transformed value coordinates. */
void orc_decode_head(int d, int G, int s_sink, int32_t S, int32_t q_end,
                     const uint16_t *kbits, const uint16_t *vbits,
                     const uint8_t *kc, const uint16_t *kp,
                     const uint8_t *vc, const uint16_t *vp,
                     const uint16_t *q, const float *tinv, float sm_scale,
                     double *out)
{
    double *K = (double *)malloc((size_t)(S > 0 ? S : 1) * d * sizeof(double));
    double *V = (double *)malloc((size_t)(S > 0 ? S : 1) * d * sizeof(double));
    for (int64_t p = 0; p < S; ++p) {
        cached_row(d, s_sink, q_end, p, kbits, kc, kp, K + p * d);
        cached_row(d, s_sink, q_end, p, vbits, vc, vp, V + p * d);
    }
    double qt[512];
    for (int g = 0; g < G; ++g) {
        for (int j = 0; j < d; ++j) {
            double acc = 0.0;
            for (int i = 0; i < d; ++i)
                acc += (double)orc_bf16_to_f32(q[(int64_t)g * d + i]) * (double)tinv[(int64_t)i * d + j];
            qt[j] = acc;
        }
        orc_attend(d, S, qt, K, V, (double)sm_scale, out + (int64_t)g * d);
    }
    free(K);
    free(V);
}

/* ------------------------------------------------------------------------ */
/* Many (sequence, kv-head) pairs at once, for the benchmark's CPU baseline.  */
/* ------------------------------------------------------------------------ */

/* The pairs are independent (Eq. (2) attends within one kv head of one
 * sequence), so they are spread over `threads` host threads (OpenMP,
 * threads <= 0: the runtime's default); each pair is exactly
 * orc_decode_head, so the arithmetic is unchanged.  Array arguments hold one
 * pointer per pair, laid out as orc_decode_head takes them.  Returns the
 * number of threads that ran. */
int orc_decode_heads_parallel(int n_pairs, int threads, int d, int G, int s_sink,
                              const int32_t *S, const int32_t *q_end,
                              const uint16_t *const *kbits, const uint16_t *const *vbits,
                              const uint8_t *const *kc, const uint16_t *const *kp,
                              const uint8_t *const *vc, const uint16_t *const *vp,
                              const uint16_t *const *q, const float *const *tinv,
                              float sm_scale, double *const *out)
{
    int used = 1;
    int nt = threads > 0 ? threads : omp_get_max_threads();
#pragma omp parallel num_threads(nt)
    {
#pragma omp single
        used = omp_get_num_threads();
#pragma omp for schedule(dynamic, 1)
        for (int i = 0; i < n_pairs; ++i)
            orc_decode_head(d, G, s_sink, S[i], q_end[i], kbits[i], vbits[i], kc[i], kp[i],
                            vc[i], vp[i], q[i], tinv[i], sm_scale, out[i]);
    }
    return used;
}

/* orc_append_head for many pairs, in parallel over the pairs (each pair's
 * own arguments as orc_append_head takes them; n_new[i] keys at k_new[i]
 * with row stride d).  q_new[i] receives the pair's new S_quant. */
int orc_append_heads_parallel(int n_pairs, int threads, int d, int bits, int s_sink, int s_keep,
                              int s_flush, int codec, float kappa_k, float kappa_v, float alpha,
                              const int32_t *s_old, const int32_t *q_old, const int32_t *n_new,
                              const uint16_t *const *k_new, const uint16_t *const *v_new,
                              const uint16_t *const *tk,
                              uint16_t *const *kbits, uint16_t *const *vbits,
                              uint8_t *const *kc, uint16_t *const *kp,
                              uint8_t *const *vc, uint16_t *const *vp, int32_t *q_new)
{
    int used = 1;
    int nt = threads > 0 ? threads : omp_get_max_threads();
#pragma omp parallel num_threads(nt)
    {
#pragma omp single
        used = omp_get_num_threads();
#pragma omp for schedule(dynamic, 1)
        for (int i = 0; i < n_pairs; ++i)
            q_new[i] = orc_append_head(d, bits, s_sink, s_keep, s_flush, codec, kappa_k, kappa_v,
                                       alpha, s_old[i], q_old[i], n_new[i], k_new[i], d, v_new[i],
                                       d, tk[i], kbits[i], vbits[i], kc[i], kp[i], vc[i], vp[i]);
    }
    return used;
}
