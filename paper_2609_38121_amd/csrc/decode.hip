// wushkv_decode_attention: split-K GQA decode attention over the mixed
// bf16 / packed-code cache (Alg. 2 step 5, Eq. (2)), with the query-side
// compensation q~ = q^T T_K^{-1} of Eq. (3).
//
// Launches on the caller's stream:
//   decode_qt_kernel       (only when the main grid runs in several
//                          residency rounds) q~ and its limbs per (kv head,
//                          row), into the workspace; otherwise each main
//                          workgroup forms them itself in LDS.
//   decode_main_kernel     grid (kv heads, splits, rows: a row is a sequence,
//                          or a sequence's token group for chunks), four
//                          waves per workgroup; the kv head on x deals each
//                          head to one XCD.  q~ is scaled by sm_scale log2(e)
//                          so that the softmax runs in base 2, and comes with
//                          the form the quantised-key product consumes: q~ in
//                          24-bit fixed point as six fp8 digit "limbs" with
//                          one power-of-two scale each, and sum(q~).
//                          Workgroups 0 .. n_page_splits - 1 scan the
//                          quantised pages, each wave a contiguous run; the
//                          others scan the bf16 sink + ring slots: one
//                          64-slot unit per workgroup, 16 slots per wave, or,
//                          when the grid runs in rounds, one workgroup per
//                          row whose waves walk all the units.  Each
//                          workgroup writes one partial (m, l, o) per query
//                          head.
//   decode_combine_kernel  log-sum-exp merge of the splits.
// Chunks at d = 128 run chunk_qt_kernel, chunk_pages_kernel and
// chunk_window_kernel instead (below).
//
// Quantised pages.  A stored key is k = s c + z per token, so
//   q~ . k = s (q~ . c) + z sum(q~).
// q~ . c comes from one 16x16x128 scaled matrix instruction per 16 tokens:
// (two of them: limbs 0-3, then limbs 4-5) the rows are (query head, limb)
// pairs of fp8 limbs with their E8M0 scales,
// the columns are tokens whose 2-bit codes read as fp4 e2m1 (a code c in the
// low two bits of a nibble is the value c / 2, exactly) or whose 4-bit codes
// read as fp8 e4m3 (c in the low nibble of a byte is c 2^-9); a column scale
// of 2 or 2^9 restores c.  Each lane then owns one query head and four
// tokens: it adds its four limb rows, forms the logits, and updates the
// online softmax.  The weights p s, split into fp16 hi + lo parts, go through
// a small per-wave LDS buffer to become the A operand rows (head, part) of
// the P V product (16x16x32 fp16), whose B operand is the value codes
// widened to fp16 subnormals with the code near the top of the fraction (see
// widen_word_f16); a slot's power-of-two factor is folded into the exponent
// of p.
//
// Window slots.  bf16 keys and values: q~ in bf16 hi + lo parts forms the A
// rows (head, part) of 16x16x32 bf16 products against the key slots; the
// probabilities, again split hi + lo, go through LDS into a 16x16x16 bf16
// P V product against the channel-major value slots.
#include <atomic>
#include <cfloat>
#include <mutex>

#include "common.h"
#include "merge.h"

namespace wushkv {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kLimbs = 6;

typedef __attribute__((ext_vector_type(8))) int i32x8;

struct DecodeArgs {
    const uint8_t *pages;
    const int32_t *page_table;
    const uint16_t *win_k;
    const uint16_t *win_v;
    const int32_t *seq_len;
    const int32_t *quant_end;
    int32_t n_kv, s_sink, win_slots, max_pages, n_pages;
    int32_t n_q;
    int32_t units_per_wave, n_page_splits, n_splits;
    int32_t win_units;     // SHARE: 64-slot window units per window workgroup
    const uint16_t *q;     // bf16 queries (decode [batch][n_q][D]; chunks [batch][max_tok][n_q][D])
    const float *tinv;     // [n_kv][D][D] T_K^{-1}, row-major
    float scale;           // sm_scale log2(e)
    float *part;           // [batch][n_kv][n_splits][G][D + 2]
    // formed by decode_qt_kernel when the main kernel does not form q~
    // itself (rows (grid row, kv head, query head of the group)):
    float *qt;             // [rows][D], scaled q~
    uint8_t *qlimb;        // [rows][6][128] fp8 limbs in operand order
    uint32_t *qaux;        // [rows][4]: limb scales (E8M0 bytes, limbs 0-3 then 4-5),
                           // sum(q~) (fp32 bits), unused
    // query rows: G is the number of virtual query heads per kv head, each
    // a (chunk token, query head) pair; grid z runs over (sequence, token
    // group) pairs bz = b n_groups + tg, token group tg holding chunk tokens
    // tg tpg .. tg tpg + tpg - 1 (virtual head v: token tg tpg + v / g_real,
    // head v % g_real).  Decode is the case max_tok = tpg = n_groups = 1.
    int32_t n_groups, tpg, g_real, max_tok;
    const int32_t *n_tok;  // [batch] chunk tokens per sequence, or null (max_tok)
    // fused step (wushkv_decode_step; null otherwise): sequence b's new token
    // (n_new[b], clamped to 0 or 1) joins the attention at position
    // seq_len[b]; the workgroup owning its window slot forms k~ = T_K k,
    // writes the slot and uses the token from LDS
    const int32_t *n_new;   // [batch]
    const uint16_t *k_new;  // bf16 [batch][n_kv][D]
    const uint16_t *v_new;  // bf16 [batch][n_kv][D]
    const uint16_t *t_k;    // bf16 [n_kv][D][D]
    uint16_t *win_kw, *win_vw;  // the windows, written
};

// Tokens of sequence b's chunk: n_tok[b] (or max_tok), at most max_tok and
// at most seq_len; the chunk is the last that many positions.
__device__ __forceinline__ int32_t chunk_tokens(const int32_t *n_tok, int32_t max_tok, int32_t b,
                                                int32_t S)
{
    int32_t n = n_tok != nullptr ? n_tok[b] : max_tok;
    n = n < max_tok ? n : max_tok;
    n = n < S ? n : S;
    return n < 0 ? 0 : n;
}

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Byte position, inside a limb's 128 operand bytes, of query channel ch: the
// A operand lane group j' element i' of the scaled product meets the key
// operand at the position the key codes' format dictates.  With fp4 keys
// (2-bit) the fp8 element (j', i') meets fp4 lane group 2 (i' / 16) + j' / 2,
// element 16 (j' % 2) + i' % 16, and the key codes put channel 32 j + i at
// fp4 element (j, i); with fp8 keys (4-bit) elements meet one to one.
template <int BITS>
__host__ __device__ constexpr int limb_pos(int ch)
{
    if (BITS == 4) return ch;
    const int j = ch >> 5, i = ch & 31;  // key lane group and element
    // solve 2 (i' / 16) + j' / 2 = j and 16 (j' % 2) + i' % 16 = i
    const int jp = 2 * (j & 1) + (i >> 4);
    const int ip = 16 * (j >> 1) + (i & 15);
    return 32 * jp + ip;
}

// ------------------------------------------------------------------ q~

// LDS of a workgroup's query rows.  One region holds, in turn, the raw bf16
// queries, q~ (fp32, scaled) and the digit limbs in operand order; the limb
// scale bytes and sum(q~) of each head follow it.
template <int D, int G>
struct QueryLds {
    // the raw queries' row pitch in bf16 elements: rows 16 bytes apart in
    // the LDS banks, so that a column read across rows does not conflict
    static constexpr int kQPitch = D + 8;
    static constexpr int kRegion = G * D * 4 > G * kLimbs * 128 ? G * D * 4 : G * kLimbs * 128;
    static constexpr int kAux = kRegion;  // uint32 [G][4]: limb scales (E8M0 bytes, limbs
                                          // 0-3 then 4-5), sum(q~) (fp32 bits), unused
    static constexpr int kBytes = kRegion + G * 16;
};

// What a thread loads for query_rows, requested before any page so that
// the pages' in-order completion cannot hold it back: its T^{-1} entries
// (wave w covers columns D/4 w .. D/4 w + D/4 - 1 as kQuads groups of four;
// lane (cq, part), cq = lane % kQuads, reads columns D/4 w + 4 cq .. + 3 of
// rows part kRr .. part kRr + kRr - 1, one 16-byte load per row) and its
// share of the raw queries (elements tid + 256 k of the G x D rows; rows of
// tokens beyond a sequence's chunk are zero).
template <int D, int G>
struct QueryIn {
    static constexpr int kQuads = D / 16;       // column quads per wave: 8 or 4
    static constexpr int kParts = 64 / kQuads;  // row parts per wave: 8 or 16
    static constexpr int kRr = D / kParts;      // rows per part: 16 or 4
    static constexpr int kPer = (G * D + 255) / 256;
    f32x4 t[kRr];
    uint16_t q[kPer];
    __device__ __forceinline__ void load(const DecodeArgs &a, int b, int tg, int h, int32_t S, int tid)
    {
        const int lane = tid & 63, wave = tid >> 6;
        const float *T = a.tinv + (int64_t)h * D * D + (int64_t)(lane / kQuads) * kRr * D +
                         (D / 4) * wave + 4 * (lane % kQuads);
#pragma unroll
        for (int r = 0; r < kRr; ++r) t[r] = *reinterpret_cast<const f32x4 *>(T + (int64_t)r * D);
        load_q(a, b, tg, h, S, tid);
    }
    // the raw queries only
    __device__ __forceinline__ void load_q(const DecodeArgs &a, int b, int tg, int h, int32_t S, int tid)
    {
        // one load per element, its address chosen first (a load in each of
        // two branches would leave the compiler waiting on both)
        const bool decode = a.max_tok == 1 && a.n_tok == nullptr;
        const int32_t nb = decode ? 1 : chunk_tokens(a.n_tok, a.max_tok, b, S);
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = tid + 256 * k;
            int64_t at = -1;
            if (i < G * D) {
                if (decode) {
                    // one token per sequence, always a valid row (an empty
                    // sequence's output is zero anyway)
                    at = ((int64_t)b * a.n_kv * G + h * G) * D + i;
                } else {
                    const int v = i / D, c = i % D;
                    const int t = tg * a.tpg + v / a.g_real, g = v % a.g_real;
                    if (t < nb)
                        at = (((int64_t)b * a.max_tok + t) * a.n_kv * a.g_real + h * a.g_real + g) * D + c;
                }
            }
            q[k] = at >= 0 ? a.q[at] : (uint16_t)0;
        }
    }
};

// The raw queries into the region R (no barrier).
template <int D, int G>
__device__ __forceinline__ void stage_queries(const QueryIn<D, G> &in, uint8_t *R, int tid)
{
    uint16_t *qs = reinterpret_cast<uint16_t *>(R);  // bf16 [G][kQPitch]
    constexpr int kP = QueryLds<D, G>::kQPitch;
#pragma unroll
    for (int k = 0; k < QueryIn<D, G>::kPer; ++k) {
        const int i = tid + 256 * k;
        if (i < G * D) qs[(i / D) * kP + i % D] = in.q[k];
    }
}

// q~ = q^T T^{-1} for the workgroup's G query rows (Alg. 2 step 3, Eq. (3)),
// scaled by sm_scale log2(e), over the staged queries in R (QueryLds).  Each
// lane forms its columns' partial products over its rows from the T^{-1}
// entries it loaded (in); the row parts of a column are summed by lane
// exchanges in a fixed order, so every workgroup of a (sequence, kv head)
// forms the same q~.  Every thread of the workgroup calls it after
// stage_queries; it starts and ends with a barrier.
template <int D, int G>
__device__ void form_qt(const DecodeArgs &a, const QueryIn<D, G> &in, uint8_t *R, int tid)
{
    using C = QueryIn<D, G>;
    const uint16_t *qs = reinterpret_cast<const uint16_t *>(R);
    __syncthreads();
    const int lane = tid & 63, wave = tid >> 6;
    const int part = lane / C::kQuads;
    float acc[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[g][e] = 0.0f;
    constexpr int kRv = C::kRr < 8 ? C::kRr : 8;  // rows per LDS read of the queries
#pragma unroll
    for (int r0 = 0; r0 < C::kRr; r0 += kRv)
#pragma unroll
        for (int g = 0; g < G; ++g) {
            uint32_t ww[4];
            if constexpr (kRv == 8) {
                const uint4 w = *reinterpret_cast<const uint4 *>(qs + g * QueryLds<D, G>::kQPitch + part * C::kRr + r0);
                ww[0] = w.x; ww[1] = w.y; ww[2] = w.z; ww[3] = w.w;
            } else {
                const uint2 w = *reinterpret_cast<const uint2 *>(qs + g * QueryLds<D, G>::kQPitch + part * C::kRr + r0);
                ww[0] = w.x; ww[1] = w.y;
            }
#pragma unroll
            for (int e = 0; e < kRv; ++e) {
                const float qi = bf16_bits_to_f32((e & 1) ? (ww[e >> 1] >> 16) : (ww[e >> 1] & 0xFFFFu));
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[g][c] = fmaf(qi, in.t[r0 + e][c], acc[g][c]);
            }
        }
    // the row parts of the wave's columns: lanes cq + kQuads m
#pragma unroll
    for (int off = C::kQuads; off < 64; off <<= 1)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[g][c] += __shfl_xor(acc[g][c], off);
    __syncthreads();  // the raw queries are read
    float *qt = reinterpret_cast<float *>(R);
    if (lane < C::kQuads) {
#pragma unroll
        for (int g = 0; g < G; ++g)
            *reinterpret_cast<f32x4 *>(qt + g * D + (D / 4) * wave + 4 * lane) =
                f32x4{acc[g][0] * a.scale, acc[g][1] * a.scale, acc[g][2] * a.scale, acc[g][3] * a.scale};
    }
    __syncthreads();
}

// The T^{-1} entries lane l of wave w supplies to form_qt_mfma: column
// D/4 w + 16 t + l % 16 at rows 4 st + l / 16.  Loaded on their own so that
// a kernel can request them together with the raw queries (one round trip).
template <int D>
struct TColumns {
    static constexpr int kTiles = D / 64;  // 16-column tiles per wave
    static constexpr int kSteps = D / 4;   // k steps of 4
    float bv[kTiles][kSteps];
    __device__ __forceinline__ void load(const DecodeArgs &a, int h, int tid)
    {
        const int lane = tid & 63, wave = tid >> 6;
        const float *T = a.tinv + (int64_t)h * D * D + (D / 4) * wave + (lane & 15);
#pragma unroll
        for (int t = 0; t < kTiles; ++t)
#pragma unroll
            for (int st = 0; st < kSteps; ++st) bv[t][st] = T[(int64_t)(4 * st + (lane >> 4)) * D + 16 * t];
    }
};

// form_qt on the fp32 matrix instructions, for decode_qt_kernel (which has
// no pages to overlap and is bound by the products): q~ = q^T T^{-1} as a
// (16 x D) x (D x D) product of 16x16x4 fp32 tiles, the G query rows padded
// to 16 with zeros.  Wave w takes the output columns D/4 w .. D/4 w + D/4 - 1
// (D/64 tiles of 16); lane l supplies A = q[l % 16][k0 + l / 16] and
// B = T^{-1}[k0 + l / 16][n0 + l % 16] and holds the result rows
// 4 (l / 16) .. + 3 of column n0 + l % 16.  The T^{-1} column entries of
// all steps come loaded in tc.  Same contract as form_qt (q~ scaled,
// fp32, into R; starts and ends with a barrier); the products are summed in
// the matrix unit's order, so q~ may differ from form_qt's in the last bits.
template <int D, int G>
__device__ void form_qt_mfma(const DecodeArgs &a, const TColumns<D> &tc, uint8_t *R, int tid)
{
    constexpr int kTiles = TColumns<D>::kTiles;
    constexpr int kSteps = TColumns<D>::kSteps;
    const uint16_t *qs = reinterpret_cast<const uint16_t *>(R);
    const int lane = tid & 63, wave = tid >> 6;
    const int m = lane & 15, kk = lane >> 4;
    const auto &bv = tc.bv;
    __syncthreads();  // the staged queries
    f32x4 acc[kTiles];
#pragma unroll
    for (int t = 0; t < kTiles; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
        const float av = m < G ? bf16_bits_to_f32(qs[m * QueryLds<D, G>::kQPitch + 4 * st + kk]) : 0.0f;
#pragma unroll
        for (int t = 0; t < kTiles; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[t][st], acc[t], 0, 0, 0);
    }
    __syncthreads();  // the raw queries are read
    float *qt = reinterpret_cast<float *>(R);
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = 4 * kk + i;
            if (row < G) qt[row * D + (D / 4) * wave + 16 * t + m] = acc[t][i] * a.scale;
        }
    __syncthreads();
}

// Rewrites q~ in R (form_qt) as the operands of the quantised-key product:
// one wave per query head writes q~ in fixed point, N = rne(q~ 2^F) with F
// the largest exponent that keeps |N| <= 7829367, as six balanced base-16
// digits d_l in [-8, 7] (N = sum_l d_l 16^(5 - l)).  Each digit is an fp8
// integer and limb l carries the E8M0 scale 16^(5 - l) 2^-F, so every
// product the matrix instruction forms is an integer times a power of two:
// its block sums, which it does not accumulate at full fp32 precision in
// general, are exact.  Also sum(q~) per head.  Every thread of the
// workgroup calls it; it ends with a barrier.
template <int D, int BITS, int G>
__device__ void form_limbs(uint8_t *R, int tid)
{
    using Q = QueryLds<D, G>;
    const int lane = tid & 63, wave = tid >> 6;
    const float *qt = reinterpret_cast<const float *>(R);
    // wave w handles query heads w, w + 4; the rows are read before the
    // region is rewritten
    constexpr int kPer = D / 64;  // channels per lane
    constexpr int kMine = (G + 3) / 4;
    float r[kMine][kPer];
#pragma unroll
    for (int k = 0; k < kMine; ++k)
#pragma unroll
        for (int e = 0; e < kPer; ++e)
            r[k][e] = (wave + 4 * k < G) ? qt[(wave + 4 * k) * D + 64 * e + lane] : 0.0f;
    __syncthreads();
    uint8_t *qlimb = R;
    uint32_t *qaux = reinterpret_cast<uint32_t *>(R + Q::kAux);
#pragma unroll
    for (int k = 0; k < kMine; ++k) {
        const int g = wave + 4 * k;
        if (g >= G) break;
        float zs = 0.0f;
#pragma unroll
        for (int e = 0; e < kPer; ++e) zs += r[k][e];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) zs += __shfl_xor(zs, off);
        uint8_t *out = qlimb + g * (kLimbs * 128);
        float mx = 0.0f;
#pragma unroll
        for (int e = 0; e < kPer; ++e) mx = fmaxf(mx, fabsf(r[k][e]));
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        // fixed point N = rne(q~ 2^F) with |N| <= 7829367 (< 2^23, exact
        // in fp32), the largest value six balanced base-16 digits reach
        constexpr float kNMax = 7829367.0f;
        int F = 0;
        if (mx > 0.0f) {
            int ex;
            (void)frexpf(kNMax / mx, &ex);
            F = ex - 1;
            if (ldexpf(mx, F) > kNMax) F -= 1;
            if (ldexpf(mx, F + 1) <= kNMax) F += 1;
            F = F < -100 ? -100 : (F > 100 ? 100 : F);
        }
        uint32_t scales[2] = {0u, 0u};
#pragma unroll
        for (int l = 0; l < kLimbs; ++l)
            scales[l >> 2] |= (uint32_t)(127 + 4 * (kLimbs - 1 - l) - F) << (8 * (l & 3));
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            const int ch = 64 * e + lane;
            int N = (int)rintf(ldexpf(r[k][e], F));
#pragma unroll
            for (int l = kLimbs - 1; l >= 0; --l) {
                const int d = ((N + 8) & 15) - 8;  // balanced digit
                N = (N - d) >> 4;
                // fp8 e4m3 of the integer d: exponent and top mantissa bits
                // of its fp32 form
                const uint32_t fb = __float_as_uint((float)(d < 0 ? -d : d));
                const uint32_t code = (d == 0 ? 0u : ((((fb >> 23) - 120u) << 3) | ((fb >> 20) & 7u))) |
                                      (d < 0 ? 0x80u : 0u);
                out[l * 128 + limb_pos<BITS>(ch)] = (uint8_t)code;
            }
        }
        if (D == 64) {
            // operand positions no channel maps to are zero: with fp4 keys
            // the elements 16 .. 31 of each lane group, with fp8 keys 64 ..
            for (int l = 0; l < kLimbs; ++l)
                for (int p = lane; p < 128; p += 64)
                    if (BITS == 2 ? (p & 16) != 0 : p >= 64) out[l * 128 + p] = 0;
        }
        if (lane == 0) {
            qaux[4 * g] = scales[0];
            qaux[4 * g + 1] = scales[1];
            qaux[4 * g + 2] = __float_as_uint(zs);
            qaux[4 * g + 3] = 0u;
        }
    }
    __syncthreads();
}

// One workgroup per (kv head, grid row): q~ and its limbs for that kv
// head's G query rows, written to the workspace for the main kernel.  Used
// when the main grid does not fit on the device at once: its workgroups
// then run in several rounds, and each forming q~ itself would read T^{-1}
// from L2 once per workgroup.
template <int D, int BITS, int G>
__global__ void __launch_bounds__(256) decode_qt_kernel(DecodeArgs a)
{
    using Q = QueryLds<D, G>;
    __shared__ __attribute__((aligned(16))) uint8_t R[Q::kBytes];
    const int tid = threadIdx.x;
    const int h = blockIdx.x, bz = blockIdx.y;
    const int b = bz / a.n_groups, tg = bz % a.n_groups;
    const int32_t S = (a.max_tok == 1 && a.n_tok == nullptr) ? 0 : a.seq_len[b];
    TColumns<D> tc;
    tc.load(a, h, tid);
    QueryIn<D, G> in;
    in.load_q(a, b, tg, h, S, tid);
    stage_queries<D, G>(in, R, tid);
    form_qt_mfma<D, G>(a, tc, R, tid);
    const int64_t row0 = ((int64_t)bz * a.n_kv + h) * G;  // first (virtual) query head
    for (int i = tid; i < G * D / 4; i += 256)
        reinterpret_cast<f32x4 *>(a.qt + row0 * D)[i] = reinterpret_cast<const f32x4 *>(R)[i];
    form_limbs<D, BITS, G>(R, tid);
    for (int i = tid; i < G * kLimbs * 128 / 16; i += 256)
        reinterpret_cast<u32x4 *>(a.qlimb + row0 * kLimbs * 128)[i] = reinterpret_cast<const u32x4 *>(R)[i];
    if (tid < G * 4) a.qaux[row0 * 4 + tid] = reinterpret_cast<const uint32_t *>(R + Q::kAux)[tid];
}

// Chunks at d = 128 (eight virtual heads per token group): one workgroup
// per (kv head, sequence, pair of token groups) forms the 16 rows of both
// groups at once, which fills the 16-row products of form_qt_mfma and reads
// T^{-1} once per pair; each group's rows go where decode_qt_kernel puts
// them.
template <int BITS>
__global__ void __launch_bounds__(256) chunk_qt_kernel(DecodeArgs a)
{
    constexpr int D = 128, G = 8, G2 = 16;
    using Q = QueryLds<D, G2>;
    __shared__ __attribute__((aligned(16))) uint8_t R[Q::kBytes];
    const int tid = threadIdx.x;
    const int h = blockIdx.x;
    const int n_pairs = (a.n_groups + 1) / 2;
    const int b = (int)blockIdx.y / n_pairs, tg = 2 * ((int)blockIdx.y % n_pairs);
    const int32_t S = a.seq_len[b];
    // virtual head v of the pair: token tg tpg + v / g_real, which is token
    // group tg + v / 8, virtual head v % 8 of that group
    TColumns<D> tc;
    tc.load(a, h, tid);
    QueryIn<D, G2> in;
    in.load_q(a, b, tg, h, S, tid);
    stage_queries<D, G2>(in, R, tid);
    form_qt_mfma<D, G2>(a, tc, R, tid);
    const int n_mine = tg + 1 < a.n_groups ? 2 : 1;
    for (int e = 0; e < n_mine; ++e) {
        const int64_t row0 = (((int64_t)b * a.n_groups + tg + e) * a.n_kv + h) * G;
        for (int i = tid; i < G * D / 4; i += 256)
            reinterpret_cast<f32x4 *>(a.qt + row0 * D)[i] = reinterpret_cast<const f32x4 *>(R)[e * G * D / 4 + i];
    }
    form_limbs<D, BITS, G2>(R, tid);
    for (int e = 0; e < n_mine; ++e) {
        const int64_t row0 = (((int64_t)b * a.n_groups + tg + e) * a.n_kv + h) * G;
        for (int i = tid; i < G * kLimbs * 128 / 16; i += 256)
            reinterpret_cast<u32x4 *>(a.qlimb + row0 * kLimbs * 128)[i] =
                reinterpret_cast<const u32x4 *>(R)[e * G * kLimbs * 128 / 16 + i];
        if (tid < G * 4) a.qaux[row0 * 4 + tid] = reinterpret_cast<const uint32_t *>(R + Q::kAux)[e * G * 4 + tid];
    }
}

// ------------------------------------------------------------------ main

template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                                  CTRL, 0xF, 0xF, false));
}
// max / sum over the 16 lanes of a row (quad butterflies, then rotations).
// The max is four DPP-operand maxima in one assembly block; each is preceded
// by the two wait states a DPP read of a just-written register needs.  The
// inputs are finite or -inf.
__device__ __forceinline__ float row_max16(float x)
{
    float y;
    asm volatile(
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %1, %1 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_f32_dpp %0, %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf"
        : "=&v"(y)
        : "v"(x));
    return y;
}
__device__ __forceinline__ float row_sum16(float x)
{
    x += dpp<0xB1>(x);
    x += dpp<0x4E>(x);
    x += dpp<0x124>(x);
    x += dpp<0x128>(x);
    return x;
}

__device__ __forceinline__ void __attribute__((address_space(3))) *lds_ptr(void *p)
{
    return (void __attribute__((address_space(3))) *)p;
}
__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)lds_ptr(const_cast<void *>(p));
}

// LDS reads and writes are ordinary loads and stores, so the compiler tracks
// their completion (and any register copies of their results) itself.  The
// direct-to-LDS page loads are not visible to it (dma16 below): it would
// otherwise wait for every one of them before any LDS access, since it
// cannot tell the staging slots apart from the rest of LDS.  Ordering
// against those loads is explicit: wait_vmcnt_at_most before a slot is read,
// lds_drain before a slot is refilled; both are compiler barriers.
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) uint16_t lds_u16;

__device__ __forceinline__ u32x4 lds_read16(uint32_t addr)
{
    return *(const lds_u32x4 *)(uintptr_t)addr;
}
__device__ __forceinline__ u32x2 lds_read8(uint32_t addr)
{
    return *(const lds_u32x2 *)(uintptr_t)addr;
}
__device__ __forceinline__ void lds_write8(uint32_t addr, uint32_t lo, uint32_t hi)
{
    *(lds_u32x2 *)(uintptr_t)addr = u32x2{lo, hi};
}
__device__ __forceinline__ void lds_write2(uint32_t addr, uint32_t v)
{
    *(lds_u16 *)(uintptr_t)addr = (uint16_t)v;
}
// Every LDS access issued so far has completed.  The assembly form is the
// compiler barrier (no memory access moves across it); the builtin form
// tells the compiler's wait bookkeeping that nothing is outstanding, so it
// adds no waits of its own for those accesses later.  (Encoding: vmcnt 63,
// expcnt 7, lgkmcnt 0.)
__device__ __forceinline__ void lds_drain()
{
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);
}

// One 16-byte direct-to-LDS load per lane: lane L's bytes src .. src + 15
// land at LDS byte lds_base + 16 L.  lds_base must be wave-uniform.  M0
// carries the LDS base; its previous value is restored, so code the
// compiler generates around this block sees M0 unchanged.  Not tracked by
// the compiler: completion is waited for with wait_vmcnt_at_most.
__device__ __forceinline__ void dma16(const void *src, uint32_t lds_base)
{
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %2\n\t"
                 "s_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, off\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(lds_base)
                 : "memory");
}

// Wait until at most `after` direct-to-LDS loads are outstanding.  `after`
// is a multiple of kDma between 0 and kMaxAhead * kDma; the count must be an
// immediate, hence the cases.  The memory clobber keeps LDS reads below it.
// The compiler's own vector-memory loads, if any are in flight, only make
// the wait stricter (loads complete in issue order).
template <int kMaxAhead, int kDma>
__device__ __forceinline__ void wait_vmcnt_at_most(int after)
{
    static_assert(kMaxAhead * kDma <= 63, "vmcnt immediate");
    if (after <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if (after <= kDma) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kDma) : "memory");
    else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kMaxAhead * kDma) : "memory");
}

__device__ __forceinline__ f32x4 mfma_scaled(const i32x8 &a, const i32x8 &b, int fmt_b, int scale_a,
                                             int scale_b, f32x4 c)
{
    if (fmt_b == 4)
        return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 4, 0, scale_a, 0, scale_b);
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, scale_a, 0, scale_b);
}

// LDS per wave: page stages (also the merge buffer) and the weight buffer.
template <int D, int BITS, int G>
struct MainLds {
    using L = Layout<D, BITS>;
    static constexpr int kStages = 2;
    static constexpr int kDma = (L::kPageBytes + 1023) / 1024;  // direct-to-LDS loads per page
    static constexpr int kSlot = kDma * 1024;
    static constexpr int kStageBytes = kStages * kSlot > G * D * 4 ? kStages * kSlot : G * D * 4;
    // weight buffer: 2G rows of 64 tokens (fp16 or bf16; row part G + g
    // holds part `part` of head g), then a zero row.  The 144-byte pitch
    // spreads the rows one reads together over distinct LDS banks.
    static constexpr int kTRows = 2 * G;
    static constexpr int kTPitch = 144;
    static constexpr int kTBytes = kTRows * kTPitch + 64;
    static constexpr int kWave = kStageBytes + kTBytes;
    // Workgroups a compute unit keeps resident, as the variants' register
    // counts allow (three waves per SIMD at most; fewer for the 4-bit and
    // the eight-head ones: the 2-bit eight-head decode kernel at d = 128 and
    // the 4-bit eight-head kernels at d = 64 are given two, and the
    // registers of a third, so that their page loops do not spill); it only
    // decides the query rows' placement.
    static constexpr int kResident = D == 128 ? (BITS == 2 ? (G == 8 ? 2 : 3) : (G == 8 ? 1 : 2))
                                              : (BITS == 2 ? (G == 8 ? 3 : 4) : (G == 8 ? 2 : 3));
    // The query rows get LDS of their own when that keeps the residency:
    // the pages can then be in flight while the rows are formed.  Otherwise
    // they borrow the start of the page stages, and the pages wait for them.
    static constexpr int kOwnBytes = 4 * kWave + QueryLds<D, G>::kBytes + 2 * 4 * G * 4;
    static constexpr bool kEarly = kOwnBytes <= 163840 / kResident;
    static constexpr int kRowsAt = kEarly ? 4 * kWave : 0;
    static constexpr int kBytes = kEarly ? 4 * kWave + QueryLds<D, G>::kBytes : 4 * kWave;
    static_assert(QueryLds<D, G>::kBytes <= 4 * kWave, "the query rows fit the page stages");
};

// Fused step: the new token of (sequence b, kv head h) into window slot
// `slot`.  k~ = T_K k is formed as the appends form it (KeyTile, the key in
// operand row 0; wave w takes output channels w D/4 .. w D/4 + D/4 - 1), so
// the stored key does not depend on the path that formed it; k~ and v go to
// the windows and to tok (LDS: bf16 k~ [D], then v [D]).  Every thread of
// the workgroup calls it; it ends with a barrier.
template <int D>
__device__ void step_token(const DecodeArgs &a, int b, int h, int32_t slot, uint16_t *tok, int tid)
{
    constexpr int kNtW = D / 64;
    constexpr int kC = D / 32;
    const int lane = tid & 63, wave = tid >> 6, j = lane >> 4, n = lane & 15;
    KeyTile<D, kNtW> xf;
    xf.load(a.t_k, h, wave * kNtW, lane);
    const int64_t row = ((int64_t)b * a.n_kv + h) * D;
    bf16x8 aop[kC];
#pragma unroll
    for (int c = 0; c < kC; ++c) {
        u32x4 av = {0u, 0u, 0u, 0u};
        if (n == 0) av = *reinterpret_cast<const u32x4 *>(a.k_new + row + 32 * c + 8 * j);
        aop[c] = __builtin_bit_cast(bf16x8, av);
    }
    uint16_t v = 0;
    if (tid < D) v = a.v_new[row + tid];
    f32x4 acc[kNtW];
    xf.apply(aop, acc);
    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;
    if (j == 0) {  // row 0, output channel 16 (w kNtW + nt) + n
#pragma unroll
        for (int nt = 0; nt < kNtW; ++nt) {
            const int o = (wave * kNtW + nt) * 16 + n;
            const uint16_t kb = (uint16_t)(pack_bf16_rne(acc[nt][0], 0.0f) & 0xFFFFu);
            tok[o] = kb;
            a.win_kw[(head_win + slot) * D + o] = kb;
        }
    }
    if (tid < D) {
        tok[D + tid] = v;
        a.win_vw[head_win * D + (int64_t)tid * a.win_slots + slot] = v;  // channel-major
    }
    __syncthreads();
}

// FORM: the workgroup forms q~ and its limbs itself (the grid fits on the
// device at once); otherwise decode_qt_kernel has written them.
// SHARE (chunks, with decode_qt_kernel): the four waves of a workgroup take
// four consecutive token groups of one sequence and the same work items
// (one run of pages, or one 64-slot window unit), so that the cache leaves
// HBM once per four token groups; grid z runs over (sequence, group of four
// token groups) and every wave writes its own partials.
template <int D, int BITS, int G, bool FORM, bool SHARE>
__global__ void __launch_bounds__(256, ((D == 128 && BITS == 2 && G == 8 && !SHARE) || (D == 64 && BITS == 4 && G == 8)) ? 2 : 3)
decode_main_kernel(DecodeArgs a)
{
    static_assert(!(FORM && SHARE), "shared work items take q~ from decode_qt_kernel");
    using L = Layout<D, BITS>;
    using M = MainLds<D, BITS, G>;
    constexpr bool kEarly = FORM && M::kEarly;
    constexpr int kStages = M::kStages;
    constexpr int kDma = M::kDma;
    constexpr int kSlot = M::kSlot;
    constexpr int kNT = L::kNTiles;   // D / 16
    constexpr int kC = L::kChunks;    // D / 32
    constexpr int kNw = L::kNw;
    constexpr int kOpw = L::kOpsPerWord;
    constexpr int kHG = G > 4 ? 2 : 1;          // score products per 16 tokens
    constexpr int kRowsPerHead = G > 4 ? 2 : 4; // P V rows per head (pages): hi, lo, [zero, zero]
    constexpr int kFmtB = BITS == 2 ? 4 : 0;    // fp4 or fp8 key codes
    constexpr int kScaleB = BITS == 2 ? 128 : 136;  // 2^1 or 2^9

    __shared__ __attribute__((aligned(16))) uint8_t lds[FORM ? M::kBytes : 4 * M::kWave];
    __shared__ float sM[4][G], sL[4][G];

    // the wave index is uniform across the wave: keep it (and the page range
    // derived from it) in scalar registers
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j = lane >> 4, n = lane & 15;
    // grid z: (sequence, token group) pairs; see DecodeArgs
    // grid x is the kv head: workgroups are handed to the eight XCDs in
    // turn, so with eight kv heads each XCD's L2 holds one head's T_K^-1
    const int h = blockIdx.x, split = blockIdx.y;
    const int n_quads = (a.n_groups + 3) / 4;  // SHARE: groups of four token groups
    const int b = SHARE ? (int)blockIdx.z / n_quads : (int)blockIdx.z / a.n_groups;
    const int tg = SHARE ? 4 * ((int)blockIdx.z % n_quads) + wave : (int)blockIdx.z % a.n_groups;
    const bool rows_live = !SHARE || tg < a.n_groups;   // SHARE: this wave has rows
    const int bz = b * a.n_groups + (rows_live ? tg : 0);  // grid row of this wave's rows
    uint8_t *stage = lds + wave * M::kWave;
    uint8_t *tbuf = stage + M::kStageBytes;
    constexpr int kTP = M::kTPitch;
    const uint32_t zero_row = lds_addr(tbuf + M::kTRows * kTP);

    // fused step: the new token is position seq_len[b] and is attended to
    const int32_t s_old = a.seq_len[b];
    int32_t nn = a.n_new != nullptr ? a.n_new[b] : 0;
    nn = nn < 0 ? 0 : (nn > 1 ? 1 : nn);
    const int32_t S = s_old + nn;
    int32_t qend = a.quant_end[b];
    qend = qend < S ? qend : S;
    const int32_t q_hi = qend > a.s_sink ? qend : a.s_sink;  // quantised: [s_sink, q_hi)
    const int32_t n_qpages = (q_hi - a.s_sink + kPage - 1) / kPage;

    // per-wave results for the merge: o (unnormalised, relative to m), m, l
    float(*sC)[D] = reinterpret_cast<float(*)[D]>(stage);

    // the page run of this wave and its page-table entries, then the T^{-1}
    // entries of q~, all requested before any page
    const bool page_wg = split < a.n_page_splits;
    const int upw = a.units_per_wave;
    const int w0 = page_wg ? (SHARE ? split : split * 4 + wave) * upw : 0;
    const int w1 = page_wg && rows_live ? min(w0 + upw, n_qpages) : 0;
    int32_t tbl = -1;
    if (w0 + lane < w1 && w0 + lane < a.max_pages)
        tbl = a.page_table[(int64_t)b * a.max_pages + w0 + lane];
    QueryIn<D, G> qin;
    if constexpr (FORM) qin.load(a, b, tg, h, S, tid);
    using Q = QueryLds<D, G>;
    uint8_t *qrows = lds + M::kRowsAt;
    const int64_t row0 = ((int64_t)bz * a.n_kv + h) * G;  // first (virtual) query head

    if (page_wg) {
        // ================================================ quantised pages
        auto phys_of = [&](int u) -> int32_t { return __builtin_amdgcn_readlane(tbl, u - w0); };
        // Every page of the run issues exactly kDma loads; an entry outside
        // the pool loads physical page 0 instead (its data is never used),
        // which keeps the count of outstanding loads a closed form.
        auto issue = [&](int u, int s) {
            int32_t phys = phys_of(u);
            if (phys < 0 || phys >= a.n_pages) phys = 0;
            const uint8_t *src = a.pages + ((int64_t)phys * a.n_kv + h) * L::kPageBytes + 16 * lane;
            const uint32_t dst = __builtin_amdgcn_readfirstlane(lds_addr(stage + s * kSlot));
#pragma unroll
            for (int i = 0; i < kDma; ++i) {
                if (i + 1 < kDma || 1024 * i + 16 * lane < L::kPageBytes)
                    dma16(src + 1024 * i, dst + 1024 * i);
            }
        };
        const bool run = a.n_pages > 0 && w0 < w1;
        const uint8_t *qlimb;
        const uint32_t *qaux;
        if constexpr (FORM) {
            // When the rows have LDS of their own, the first two pages of the
            // run go in flight while q~ is formed.  Every load made so far
            // completes first, so that no later wait of the rows' arithmetic
            // can be held up by the pages (loads complete in issue order).
            stage_queries<D, G>(qin, qrows, tid);
            if (kEarly) {
                // vmcnt(0) as the compiler's own wait: it then counts the
                // rows' loads complete and sets no wait on them behind the pages
                __builtin_amdgcn_s_waitcnt(0x0F70);
                if (run) {
                    issue(w0, 0);
                    if (w0 + 1 < w1) issue(w0 + 1, 1);
                }
            }
            form_qt<D, G>(a, qin, qrows, tid);
            form_limbs<D, BITS, G>(qrows, tid);
            qlimb = qrows;
            qaux = reinterpret_cast<const uint32_t *>(qrows + Q::kAux);
        } else {
            qlimb = a.qlimb + row0 * kLimbs * 128;
            qaux = a.qaux + row0 * 4;
        }

        // score A operands, two per head group: row m = 4 g' + r holds limb
        // r (first) or limb 4 + r for r < 2 (second; rows r >= 2 zero) of
        // head hd = g' (G <= 4) or 2 g' + hg (G = 8); heads >= G give zero rows
        i32x8 qa[kHG][2];
        int qsc[kHG][2];
        float zs[kHG];  // sum(q~) of the head this lane's scores belong to
#pragma unroll
        for (int hg = 0; hg < kHG; ++hg) {
            const int hd = G > 4 ? 2 * (n >> 2) + hg : (n >> 2);
#pragma unroll
            for (int part = 0; part < 2; ++part) {
                const int limb = 4 * part + (n & 3);
                u32x4 x0 = {0u, 0u, 0u, 0u}, x1 = x0;
                qsc[hg][part] = 127;
                if (hd < G && limb < kLimbs) {
                    const uint8_t *src = qlimb + (hd * kLimbs + limb) * 128 + 32 * j;
                    x0 = *reinterpret_cast<const u32x4 *>(src);
                    x1 = *reinterpret_cast<const u32x4 *>(src + 16);
                    qsc[hg][part] = (qaux[4 * hd + part] >> (8 * (n & 3))) & 0xFFu;
                }
                qa[hg][part] = i32x8{(int)x0[0], (int)x0[1], (int)x0[2], (int)x0[3],
                                     (int)x1[0], (int)x1[1], (int)x1[2], (int)x1[3]};
            }
            const int hs = G > 4 ? 2 * j + hg : j;
            zs[hg] = hs < G ? __uint_as_float(qaux[4 * hs + 2]) : 0.0f;
        }
        if constexpr (!kEarly) {
            // every wave has its operands: the pages may now land over the
            // rows (LDS), or (memory) the operands have arrived, so that the
            // compiler's wait for them cannot include the pages
            if constexpr (FORM) __syncthreads();
            else __builtin_amdgcn_s_waitcnt(0x0F70);
            if (run) {
                issue(w0, 0);
                if (w0 + 1 < w1) issue(w0 + 1, 1);
            }
        }
        if (lane < 16) reinterpret_cast<uint32_t *>(tbuf + M::kTRows * kTP)[lane] = 0u;
        // this lane's heads in the score layout, and whether they exist
        bool hvalid[kHG];
#pragma unroll
        for (int hg = 0; hg < kHG; ++hg) hvalid[hg] = (G > 4 ? 2 * j + hg : j) < G;

        // online-softmax state per head of this lane (l and z in units of
        // 2^-off, below)
        f32x4 acc[kNT];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        float m_run[kHG], lc[kHG], zc[kHG];
#pragma unroll
        for (int hg = 0; hg < kHG; ++hg) {
            m_run[hg] = -INFINITY;
            lc[hg] = zc[hg] = 0.0f;
        }
        // token 4 n + t is slot i = 4 (n % 2) + t of the value operand, in
        // register i / 2 = 2 (n % 2) + t / 2; the value widening puts 2-bit
        // codes of registers 2-3 two bits higher (2^8 instead of 2^6), so this
        // lane's weights carry 2^-off, off = 2 (n % 2); 4-bit codes all sit
        // at 2^4.  The products are p s c 2^-18 (2-bit) or 2^-20 (4-bit).
        const float off = BITS == 2 ? 2.0f * (n & 1) : 0.0f;
        constexpr float kOutScale = BITS == 2 ? 262144.0f : 1048576.0f;

        // P V A operand rows: row m is part m % kRowsPerHead (0: fp16 hi
        // of the weight, 1: the fp16 rest, others zero) of head
        // m / kRowsPerHead; weight rows sit at 2 g + part in the buffer
        const int ahead = n / kRowsPerHead, apart = n % kRowsPerHead;
        const bool arow_ok = ahead < G && apart < 2;
        const uint32_t a_addr = arow_ok ? lds_addr(tbuf + (apart * G + ahead) * kTP + 16 * j) : zero_row;
        const uint32_t a_step = arow_ok ? 64u : 0u;  // second 32-token chunk

        // Per page: the value words are read at the top (they are needed only
        // by the P V products at the end); the key words and parameters of
        // page u were read at the end of iteration u - 1, while its P V
        // products ran.  A page's stage is refilled (page u + 2) as soon as
        // its value reads have completed, right after the score products are
        // issued.
        constexpr int kKX = L::kKWordsPerLane / 4;  // key chunks per lane
        constexpr int kVX = L::kWordsPerLane / 4;   // value chunks per lane
        auto read_keys = [&](uint32_t pg, u32x4 (&kx)[kKX + 2]) {
#pragma unroll
            for (int q4 = 0; q4 < kKX; ++q4) kx[q4] = lds_read16(pg + 4 * L::k_word(lane, 4 * q4));
            kx[kKX] = lds_read16(pg + L::kParamOffset + 16 * n);
            kx[kKX + 1] = lds_read16(pg + L::kParamOffset + 4 * kPage + 16 * n);
        };
        auto read_values = [&](uint32_t pg, u32x4 (&vx)[kVX]) {
#pragma unroll
            for (int q4 = 0; q4 < kVX; ++q4) vx[q4] = lds_read16(pg + L::kRegionBytes + 4 * L::v_word(lane, 4 * q4));
        };
        if (run) {
            // Three stages: page u in registers, pages u + 1 and u + 2 in
            // flight to the two LDS slots (the first two issued above).  A
            // slot is emptied into registers as soon as its page has landed
            // and refilled right away, so both slots stay in flight while a
            // page is computed.
            static_assert(kStages == 2, "two slots per wave");
            wait_vmcnt_at_most<1, kDma>(w0 + 1 < w1 ? kDma : 0);
            u32x4 kx[kKX + 2], vv[kVX];
            read_keys(lds_addr(stage), kx);
            read_values(lds_addr(stage), vv);
            lds_drain();
            if (w0 + 2 < w1) issue(w0 + 2, 0);
            for (int u = w0; u < w1; ++u) {
                const int s = (u - w0) & 1;
                const int32_t phys = phys_of(u);
                // a page outside the pool contributes nothing (its stage holds page 0)
                const int32_t nvalid = (phys < 0 || phys >= a.n_pages)
                                           ? 0 : min(kPage, q_hi - (a.s_sink + u * kPage));
                const u32x4 kp = kx[kKX], vp = kx[kKX + 1];

                // scores: one product per 16 tokens, head group and limb group;
                // all issued before any result is used
                i32x8 bop[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    uint32_t w[BITS];
#pragma unroll
                    for (int i = 0; i < BITS; ++i) w[i] = kx[(BITS * t + i) / 4][(BITS * t + i) % 4];
                    if constexpr (BITS == 2) {
                        bop[t] = i32x8{(int)(w[0] & 0x33333333u), (int)((w[0] >> 2) & 0x33333333u),
                                       (int)(w[1] & 0x33333333u), (int)((w[1] >> 2) & 0x33333333u),
                                       0, 0, 0, 0};
                    } else {
                        bop[t] = i32x8{(int)(w[0] & 0x0F0F0F0Fu), (int)((w[0] >> 4) & 0x0F0F0F0Fu),
                                       (int)(w[1] & 0x0F0F0F0Fu), (int)((w[1] >> 4) & 0x0F0F0F0Fu),
                                       (int)(w[2] & 0x0F0F0F0Fu), (int)((w[2] >> 4) & 0x0F0F0F0Fu),
                                       (int)(w[3] & 0x0F0F0F0Fu), (int)((w[3] >> 4) & 0x0F0F0F0Fu)};
                    }
                }
                // limbs 4-5 (rows 4 g' + 0, 1 of the second product) are
                // accumulated onto limbs 0-1 of the first, so each head's six
                // limbs end up in its four rows
                f32x4 c[kHG][4];
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int hg = 0; hg < kHG; ++hg)
                        c[hg][t] = mfma_scaled(qa[hg][0], bop[t], kFmtB, qsc[hg][0], kScaleB, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int hg = 0; hg < kHG; ++hg)
                        c[hg][t] = mfma_scaled(qa[hg][1], bop[t], kFmtB, qsc[hg][1], kScaleB, c[hg][t]);
                float lg[kHG][4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const float ks = f16_bits_to_f32(kp[t] & 0xFFFFu);
                    const float kz = f16_bits_to_f32(kp[t] >> 16);
#pragma unroll
                    for (int hg = 0; hg < kHG; ++hg) {
                        const f32x4 &c0 = c[hg][t];
                        const float dot = (c0[0] + c0[1]) + (c0[2] + c0[3]);
                        lg[hg][t] = fmaf(ks, dot, kz * zs[hg]);
                    }
                }
                if (nvalid < kPage) {
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        if (4 * n + t >= nvalid)
#pragma unroll
                            for (int hg = 0; hg < kHG; ++hg) lg[hg][t] = -INFINITY;
                }
                // running max per head (every lane of a row holds its head's)
                float m_new[kHG];
                bool grow = false;
#pragma unroll
                for (int hg = 0; hg < kHG; ++hg) {
                    const float mx = row_max16(fmaxf(fmaxf(lg[hg][0], lg[hg][1]), fmaxf(lg[hg][2], lg[hg][3])));
                    m_new[hg] = fmaxf(m_run[hg], mx);
                    grow |= hvalid[hg] && m_new[hg] > m_run[hg];
                }
                if (__any(grow)) {
                    // rescale: P V rows of lane (j, n) register r belong to
                    // head j (G <= 4) or 2 j + r / 2 (G = 8), this lane's own
                    float al[kHG];
#pragma unroll
                    for (int hg = 0; hg < kHG; ++hg) {
                        al[hg] = m_new[hg] == -INFINITY ? 1.0f : fexp2(m_run[hg] - m_new[hg]);
                        lc[hg] *= al[hg];
                        zc[hg] *= al[hg];
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float ar = al[G > 4 ? (r >> 1) : 0];
#pragma unroll
                        for (int nt = 0; nt < kNT; ++nt) acc[nt][r] *= ar;
                    }
                }
#pragma unroll
                for (int hg = 0; hg < kHG; ++hg) m_run[hg] = m_new[hg];

                // weights p s 2^-off as fp16 hi + lo (about 22 significant
                // bits), through LDS into the A operand rows
#pragma unroll
                for (int hg = 0; hg < kHG; ++hg) {
                    // (no valid token yet: every weight is exp2(-inf) = 0)
                    const float mo = m_run[hg] == -INFINITY ? 0.0f : m_run[hg] + off;
                    float wgt[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const float pw = fexp2(lg[hg][t] - mo);
                        lc[hg] += pw;
                        zc[hg] = fmaf(pw, f16_bits_to_f32(vp[t] >> 16), zc[hg]);
                        // one mixed-precision product, rounded once like pw * s
                        wgt[t] = fmaf(pw, f16_bits_to_f32(vp[t] & 0xFFFFu), 0.0f);
                    }
                    const int hs = G > 4 ? 2 * j + hg : j;
                    if (hs < G) {
                        const uint32_t h01 = pack_f16_rne(wgt[0], wgt[1]);
                        const uint32_t h23 = pack_f16_rne(wgt[2], wgt[3]);
                        // the rest w - hi is exact in fp32 (one fused step each)
                        const uint32_t l01 = pack_f16_rne(fmaf(-1.0f, f16_bits_to_f32(h01 & 0xFFFFu), wgt[0]),
                                                          fmaf(-1.0f, f16_bits_to_f32(h01 >> 16), wgt[1]));
                        const uint32_t l23 = pack_f16_rne(fmaf(-1.0f, f16_bits_to_f32(h23 & 0xFFFFu), wgt[2]),
                                                          fmaf(-1.0f, f16_bits_to_f32(h23 >> 16), wgt[3]));
                        lds_write8(lds_addr(tbuf + hs * kTP + 8 * n), h01, h23);
                        lds_write8(lds_addr(tbuf + (G + hs) * kTP + 8 * n), l01, l23);
                    }
                }
                // A operands (two 32-token chunks)
                u32x4 ax[2];
                ax[0] = lds_read16(a_addr);
                ax[1] = lds_read16(a_addr + a_step);
                // page u + 1 (slot s ^ 1) into registers: it has landed once at
                // most page u + 2's loads remain
                u32x4 vn[kVX];
                if (u + 1 < w1) {
                    wait_vmcnt_at_most<1, kDma>(u + 2 < w1 ? kDma : 0);
                    read_keys(lds_addr(stage + (s ^ 1) * kSlot), kx);
                    read_values(lds_addr(stage + (s ^ 1) * kSlot), vn);
                }
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    const f16x8 A = __builtin_bit_cast(f16x8, ax[kc]);
#pragma unroll
                    for (int uu = 0; uu < 2 * kNw; ++uu) {
                        const int widx = kc * 2 * kNw + uu;
                        uint32_t op[L::kCodesPerWord / 2];
                        widen_word_f16<BITS>(vv[widx / 4][widx % 4], op);
#pragma unroll
                        for (int o = 0; o < kOpw; ++o) {
                            const int nt = uu * kOpw + o;
                            acc[nt] = mfma16h(A, as_op_h(op + 4 * o), acc[nt]);
                        }
                    }
                }
                if (u + 1 < w1) {
                    // slot s ^ 1 has been read out: refill it with page u + 3
                    lds_drain();
                    if (u + 3 < w1) issue(u + 3, s ^ 1);
#pragma unroll
                    for (int q4 = 0; q4 < kVX; ++q4) vv[q4] = vn[q4];
                }
            }
        }

        // ---- this wave's result per head: o = acc 2^18 (or 2^20) + z (rows of
        // lane (j, n) register r: head j, or 2 j + r / 2 for G = 8)
        float zt[kHG], lt[kHG];
#pragma unroll
        for (int hg = 0; hg < kHG; ++hg) {
            const float f = ldexpf(1.0f, (int)off);
            zt[hg] = row_sum16(zc[hg] * f);
            lt[hg] = row_sum16(lc[hg] * f);
        }
#pragma unroll
        for (int hg = 0; hg < kHG; ++hg) {
            const int hs = G > 4 ? 2 * j + hg : j;
            const int r = G > 4 ? 2 * hg : 0;  // the hi row; the lo row follows
            if (hs < G) {
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt)
                    sC[hs][16 * nt + n] = fmaf(acc[nt][r] + acc[nt][r + 1], kOutScale, zt[hg]);
                if (n == 0) {
                    sM[wave][hs] = m_run[hg];
                    sL[wave][hs] = lt[hg];
                }
            }
        }
    } else {
        // ================================================ window slots
        // Workgroup n_page_splits + u owns window unit u (slots 64 u ..
        // 64 u + 63), wave w its 16 slots 64 u + 16 w .. + 15 (SHARE: the
        // workgroup owns win_units consecutive units and every wave all their
        // 16-slot tiles, for its own rows, with an online softmax across
        // them).  All of a tile's loads are issued together.
        const int32_t ring = a.win_slots - a.s_sink;
        // the ring holds positions [q_hi, S); the oldest sits at ring index a0
        const int32_t a0 = S > q_hi ? (q_hi - a.s_sink) % ring : 0;
        const int32_t ring_live = S > q_hi ? S - q_hi : 0;
        const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;
        const int32_t unit0 = (split - a.n_page_splits) * kPage * a.win_units;
        // fused step: the workgroup whose unit holds the new token's slot
        // writes the token and keeps it in LDS, at the end of wave 3's page
        // stage (its merge rows, written last, sit at the start)
        int32_t new_slot = -1;
        uint16_t *tok = reinterpret_cast<uint16_t *>(lds + 3 * M::kWave + M::kStageBytes - 4 * D);
        static_assert(G * D * 4 + 8 * D <= M::kStageBytes, "the new token fits the page stage");
        if (a.n_new != nullptr && nn > 0) {
            const int32_t slot = s_old < a.s_sink ? s_old : ring_slot(s_old, a.s_sink, ring);
            if (slot >= unit0 && slot < unit0 + kPage * a.win_units) {
                new_slot = slot;
                step_token<D>(a, b, h, slot, tok, tid);
            }
        }

        const float *qtl;
        if constexpr (FORM) {
            stage_queries<D, G>(qin, qrows, tid);
            form_qt<D, G>(a, qin, qrows, tid);
            qtl = reinterpret_cast<const float *>(qrows);
        } else {
            qtl = a.qt + row0 * D;
        }
        // A operands: row m = 2 g + part (hi, lo) of q~, chunk c.  From LDS
        // they are formed at once; from memory only after the slot loads are
        // issued, so that the latencies overlap.
        bf16x8 qa[kC];
        auto form_qa = [&]() {
            const int g = n >> 1, part = n & 1;
#pragma unroll
            for (int c = 0; c < kC; ++c) {
                uint32_t u[4] = {0u, 0u, 0u, 0u};
                if (g < G) {
                    const float *src = qtl + g * D + 32 * c + 8 * j;
                    const f32x4 x0 = *reinterpret_cast<const f32x4 *>(src);
                    const f32x4 x1 = *reinterpret_cast<const f32x4 *>(src + 4);
                    const float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
#pragma unroll
                    for (int pp = 0; pp < 4; ++pp) {
                        const uint32_t hi = pack_bf16_rne(x[2 * pp], x[2 * pp + 1]);
                        const uint32_t lo = pack_bf16_rne(x[2 * pp] - bf16_bits_to_f32(hi & 0xFFFFu),
                                                          x[2 * pp + 1] - bf16_bits_to_f32(hi >> 16));
                        u[pp] = part ? lo : hi;
                    }
                }
                qa[c] = __builtin_bit_cast(bf16x8, u32x4{u[0], u[1], u[2], u[3]});
            }
        };
        if constexpr (FORM) form_qa();
        if constexpr (FORM && !kEarly) __syncthreads();  // the rows may now be overwritten
        if (lane < 16) reinterpret_cast<uint32_t *>(tbuf + M::kTRows * kTP)[lane] = 0u;

        f32x4 acc[kNT];
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        float m_run[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f};
        bool formed = FORM;
        // SHARE: every wave all 16-slot tiles of the workgroup's units, with
        // an online softmax across them
        // (otherwise wave w takes tile w of each of the workgroup's units)
        // (the query-forming variant runs only plans of one unit per window
        // workgroup: its loop is a single tile, kept compile-time so that it
        // costs no registers)
        const int kSub = SHARE ? 4 * a.win_units : (FORM ? 1 : a.win_units);
        for (int st = 0; st < (rows_live ? kSub : 0); ++st) {
            const int32_t slot0 = unit0 + 16 * (SHARE ? st : wave + 4 * st);
            // this tile's live slots, one bit per slot (lanes 0..15)
            bool mine;
            {
                const int32_t sl = slot0 + n;
                if (sl < a.s_sink) mine = sl < S;
                else mine = ((sl - a.s_sink - a0 + ring) % ring) < ring_live;
            }
            const uint32_t vmask = (uint32_t)(__ballot(mine) & 0xFFFFu);
            if (vmask == 0) continue;
            // key slots (token slot0 + n, channels 32 c + 8 j ..) and value
            // slots (channel 16 nt + n, tokens slot0 + 4 j .. + 3)
            const uint16_t *krow = a.win_k + (head_win + slot0 + n) * D + 8 * j;
            u32x4 kx[kC];
#pragma unroll
            for (int c = 0; c < kC; ++c) kx[c] = *reinterpret_cast<const u32x4 *>(krow + 32 * c);
            const uint16_t *vrow = a.win_v + head_win * D + slot0 + 4 * j;
            u32x2 vx[kNT];
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
                vx[nt] = *reinterpret_cast<const u32x2 *>(vrow + (int64_t)(16 * nt + n) * a.win_slots);
            if (new_slot >= slot0 && new_slot < slot0 + 16) {
                // the new token's slot: its key row (lanes n = t) and its
                // values (element t % 4 of lanes j = t / 4) from LDS
                const int t = new_slot - slot0;
                if (n == t) {
#pragma unroll
                    for (int c = 0; c < kC; ++c) kx[c] = *reinterpret_cast<const u32x4 *>(tok + 32 * c + 8 * j);
                }
                if (j == (t >> 2)) {
                    const int e = t & 3;
#pragma unroll
                    for (int nt = 0; nt < kNT; ++nt) {
                        const uint32_t v = tok[D + 16 * nt + n];
                        const uint32_t w = vx[nt][e >> 1];
                        vx[nt][e >> 1] = (e & 1) ? ((w & 0xFFFFu) | (v << 16)) : ((w & 0xFFFF0000u) | v);
                    }
                }
            }
            if (!formed) {
                form_qa();
                formed = true;
            }

            // scores: lane (j, n) gets rows 4 j + r = (head 2 j + r / 2,
            // part r % 2) of token slot0 + n
            f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < kC; ++c) sc = mfma16(qa[c], __builtin_bit_cast(bf16x8, kx[c]), sc);
            const bool ok = (vmask >> n) & 1u;
            // causal visibility of this slot's position to the query rows
            // 2 j and 2 j + 1: a chunk token at position p sees [0, p] (the
            // quantised pages all lie before the chunk, so only the windows
            // need this)
            bool vis[2] = {ok, ok};  // decode: the query sees every live slot
            if (a.max_tok > 1 || a.n_tok != nullptr) {
                const int32_t sl = slot0 + n;
                const int32_t pos = sl < a.s_sink ? sl : q_hi + ((sl - a.s_sink - a0 + ring) % ring);
                const int32_t nb = chunk_tokens(a.n_tok, a.max_tok, b, S);
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const int32_t t = tg * a.tpg + (2 * j + e) / a.g_real;  // chunk token of the row
                    vis[e] = ok && t < nb && pos <= S - nb + t;
                }
            }
            float lg[2];
            lg[0] = vis[0] ? sc[0] + sc[1] : -INFINITY;
            lg[1] = vis[1] ? sc[2] + sc[3] : -INFINITY;
            float pr[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                // online softmax over the tiles: the running sums are scaled
                // to the new maximum (a first tile scales zeros)
                const float m_new = fmaxf(m_run[e], row_max16(lg[e]));
                const float f_old = m_run[e] == -INFINITY ? 0.0f : fexp2(m_run[e] - m_new);
                pr[e] = m_new == -INFINITY ? 0.0f : fexp2(lg[e] - m_new);
                lsum[e] = fmaf(lsum[e], f_old, pr[e]);
                m_run[e] = m_new;
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt) {
                    acc[nt][2 * e] *= f_old;
                    acc[nt][2 * e + 1] *= f_old;
                }
                const int g = 2 * j + e;
                if (g < G) {
                    const uint32_t hl = pack_bf16_rne(pr[e], 0.0f) & 0xFFFFu;
                    const uint32_t ll = pack_bf16_rne(pr[e] - bf16_bits_to_f32(hl), 0.0f) & 0xFFFFu;
                    lds_write2(lds_addr(tbuf + g * kTP + 2 * n), hl);
                    lds_write2(lds_addr(tbuf + (G + g) * kTP + 2 * n), ll);
                }
            }
            // A operand of the 16x16x16 product: row m = 2 g + part, tokens
            // 4 j .. 4 j + 3
            const uint32_t pa_addr = n < 2 * G ? lds_addr(tbuf + ((n & 1) * G + (n >> 1)) * kTP + 8 * j) : zero_row;
            const u32x2 pa = lds_read8(pa_addr);
            // dead slots' values are zeroed, whatever bits they hold
            const uint32_t bits4 = (vmask >> (4 * j)) & 0xFu;
            const uint32_t msk0 = ((bits4 & 1u) ? 0x0000FFFFu : 0u) | ((bits4 & 2u) ? 0xFFFF0000u : 0u);
            const uint32_t msk1 = ((bits4 & 4u) ? 0x0000FFFFu : 0u) | ((bits4 & 8u) ? 0xFFFF0000u : 0u);
            typedef __attribute__((ext_vector_type(4))) short s16x4;
            const s16x4 A = __builtin_bit_cast(s16x4, pa);
#pragma unroll
            for (int nt = 0; nt < kNT; ++nt) {
                const u32x2 y = {vx[nt][0] & msk0, vx[nt][1] & msk1};
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(A, __builtin_bit_cast(s16x4, y), acc[nt], 0, 0, 0);
            }
        }
        // result per head g = 2 j + e: rows 4 j + 2 e (hi) and + 1 (lo)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int g = 2 * j + e;
            const float lt = row_sum16(lsum[e]);
            if (g < G) {
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt) sC[g][16 * nt + n] = acc[nt][2 * e] + acc[nt][2 * e + 1];
                if (n == 0) {
                    sM[wave][g] = m_run[e];
                    sL[wave][g] = lt;
                }
            }
        }
    }
    __syncthreads();

    if constexpr (SHARE) {
        // every wave's own rows: its result is that split's partial
        for (int idx = tid; idx < 4 * G * D; idx += 256) {
            const int rb = idx / (G * D), gg = (idx / D) % G, ch = idx % D;
            const int tgr = 4 * ((int)blockIdx.z % n_quads) + rb;
            if (tgr >= a.n_groups) continue;
            const int64_t bzr = (int64_t)b * a.n_groups + tgr;
            float *pr = a.part + ((bzr * a.n_kv + h) * a.n_splits + split) * G * (D + 2);
            const float mx = sM[rb][gg];
            pr[gg * (D + 2) + ch] =
                mx == -INFINITY ? 0.0f : reinterpret_cast<const float(*)[D]>(lds + rb * M::kWave)[gg][ch];
            if (ch == 0) {
                pr[gg * (D + 2) + D] = mx;
                pr[gg * (D + 2) + D + 1] = sL[rb][gg];
            }
        }
        return;
    }

    // ---- merge the four waves
    float *part = a.part + (((int64_t)bz * a.n_kv + h) * a.n_splits + split) * G * (D + 2);
    for (int idx = tid; idx < G * D; idx += 256) {
        const int gg = idx / D, ch = idx % D;
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) mx = fmaxf(mx, sM[w][gg]);
        float o = 0.0f, l = 0.0f;
        if (mx != -INFINITY) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                if (sM[w][gg] == -INFINITY) continue;
                const float f = fexp2(sM[w][gg] - mx);
                o += f * reinterpret_cast<const float(*)[D]>(lds + w * M::kWave)[gg][ch];
                l += f * sL[w][gg];
            }
        }
        part[gg * (D + 2) + ch] = o;
        if (ch == 0) {
            part[gg * (D + 2) + D] = mx;
            part[gg * (D + 2) + D + 1] = l;
        }
    }
}

// ------------------------------------------------------------------ chunk pages

// The quantised pages of chunk attention (Alg. 2 step 5 with S' > 1) at
// d = 128.  One workgroup per (kv head, run of pages, sequence, block of
// eight token groups) takes all 64 query rows of the block -- (chunk token,
// query head) pairs, eight token groups of G = 8 rows, row r of the block in
// token group r / 8 -- so that each page leaves HBM once and its codes are
// unpacked once.  Pages stream through three LDS slots that the four waves
// share (each wave loads its part of every page).  Per page:
//   scores  wave w takes rows 16 w .. 16 w + 15: one scaled product per
//           limb and 16 tokens, whose A rows are the 16 query rows' fp8
//           digits of that limb (held in registers for the whole run, each
//           row with its own E8M0 scale) and whose B columns are the fp4 /
//           fp8 key codes, accumulated over the six limbs; lane (j, n) then
//           holds rows 16 w + 4 j + r of tokens 4 n .. 4 n + 3, runs their
//           online softmax and writes their weights (fp16 hi + lo) and
//           rescale factors to LDS;
//   P V     wave w takes channel tiles 2 w, 2 w + 1 of all 64 rows: the
//           weights times its value codes widened to fp16 subnormals.
// The chunk lies in the recent window (every quantised position precedes
// it), so no mask applies.  Each row's partial (o, m, l) goes where the
// decode kernel writes it; the window slots are left to that kernel.
// Byte offset of byte `byte` of a 128-byte weight row `row`: the 16-byte
// chunks of row r are stored in the order chunk ^ (r % 8), so that the rows
// one instruction reads together fall in distinct LDS banks.
__device__ __forceinline__ uint32_t tbuf_at(int row, int byte)
{
    return (uint32_t)(row * 128 + ((((byte >> 4) ^ (row & 7)) << 4) | (byte & 15)));
}

template <int BITS>
struct ChunkLds {
    using L = Layout<128, BITS>;
    static constexpr int kRows = 64;
    static constexpr int kSlots = 4;
    static constexpr int kSlot = (L::kPageBytes + 15) / 16 * 16;
    static constexpr int kWBytes = 2 * kRows * 128;          // weights: hi plane, lo plane
    static constexpr int kWAt = 0;                           // two buffers (page parity)
    static constexpr int kAlphaAt = kWAt + 2 * kWBytes;      // per row: rescale factors, two buffers
    static constexpr int kZAt = kAlphaAt + 2 * kRows * 4;    // per row at the end: z term, m, l
    static constexpr int kMAt = kZAt + kRows * 4;
    static constexpr int kLAt = kMAt + kRows * 4;
    static constexpr int kSlotAt = kLAt + kRows * 4;
    static constexpr int kBytes = kSlotAt + kSlots * kSlot;
};

// One limb's scaled product: A = limb L of 16 query rows, whose E8M0 scale
// is byte L % 4 of the lane's packed scale word (the instruction's byte
// select), B = 16 tokens' key codes.
template <int L, int FMT_B, int SCALE_B>
__device__ __forceinline__ f32x4 limb_product(const i32x8 &a, const i32x8 &b, int scales, f32x4 c)
{
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, FMT_B, L % 4, scales, 0, SCALE_B);
}

template <int BITS>
__global__ void __launch_bounds__(256, 2) chunk_pages_kernel(DecodeArgs a)
{
    constexpr int D = 128, G = 8;
    using L = Layout<D, BITS>;
    using C = ChunkLds<BITS>;
    constexpr int kDma = (L::kPageBytes + 1023) / 1024;  // direct-to-LDS loads per page
    constexpr int kNTw = L::kNTiles / 4;                  // channel tiles per wave
    constexpr int kFmtB = BITS == 2 ? 4 : 0;
    constexpr int kScaleB = BITS == 2 ? 128 : 136;
    constexpr int kKX = L::kKWordsPerLane / 4;            // key chunks per lane
    constexpr int kOpw = L::kOpsPerWord;
    constexpr float kOutScale = BITS == 2 ? 262144.0f : 1048576.0f;
    __shared__ __attribute__((aligned(16))) uint8_t lds[C::kBytes];

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j = lane >> 4, n = lane & 15;
    const int h = blockIdx.x, split = blockIdx.y;
    const int n_blocks = (a.n_groups + 7) / 8;
    const int b = (int)blockIdx.z / n_blocks, tg0 = 8 * ((int)blockIdx.z % n_blocks);
    const int32_t S = a.seq_len[b];
    int32_t qend = a.quant_end[b];
    qend = qend < S ? qend : S;
    const int32_t q_hi = qend > a.s_sink ? qend : a.s_sink;  // quantised: [s_sink, q_hi)
    const int32_t n_qpages = (q_hi - a.s_sink + kPage - 1) / kPage;
    const int upw = a.units_per_wave;  // pages of a workgroup's run (at most 64)
    const int w0 = split * upw;
    const int w1 = min(w0 + upw, n_qpages);
    int32_t tbl = -1;
    if (w0 + lane < w1 && w0 + lane < a.max_pages) tbl = a.page_table[(int64_t)b * a.max_pages + w0 + lane];

    // The wave's 16 query rows 16 w .. 16 w + 15 of the block's 64 (rows
    // past the chunk's token groups have zero limbs).  Lane (j, n) holds the
    // A operands of row 16 w + n, K bytes 32 j .., one per limb, and that
    // row's packed limb scales; its scores are rows 16 w + 4 j + r (r < 4),
    // whose sums of q~ it keeps.
    auto row_of = [&](int r64) -> int64_t {
        const int tg = tg0 + r64 / G;
        return tg < a.n_groups ? (((int64_t)b * a.n_groups + tg) * a.n_kv + h) * G + r64 % G : -1;
    };
    i32x8 qa[kLimbs];
    int sc03 = 0, sc45 = 0;
    {
        const int64_t row = row_of(16 * wave + n);
#pragma unroll
        for (int l = 0; l < kLimbs; ++l) {
            u32x4 x0 = {0u, 0u, 0u, 0u}, x1 = x0;
            if (row >= 0) {
                const uint8_t *src = a.qlimb + row * (kLimbs * 128) + l * 128 + 32 * j;
                x0 = *reinterpret_cast<const u32x4 *>(src);
                x1 = *reinterpret_cast<const u32x4 *>(src + 16);
            }
            qa[l] = i32x8{(int)x0[0], (int)x0[1], (int)x0[2], (int)x0[3],
                          (int)x1[0], (int)x1[1], (int)x1[2], (int)x1[3]};
        }
        if (row >= 0) {
            sc03 = (int)a.qaux[4 * row];
            sc45 = (int)a.qaux[4 * row + 1];
        }
    }
    float zs[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int64_t row = row_of(16 * wave + 4 * j + r);
        zs[r] = row >= 0 ? __uint_as_float(a.qaux[4 * row + 2]) : 0.0f;
    }

    const uint32_t lbase = lds_addr(lds);
    // This wave's share of each page's loads: loads i = wave, wave + 4, ..
    constexpr int kMine0 = (kDma + 3) / 4;  // (wave 0 takes the most)
    const int n_mine = (kDma - wave + 3) / 4;
    auto issue = [&](int u, int slot) {
        int32_t phys = __builtin_amdgcn_readlane(tbl, u - w0);
        if (phys < 0 || phys >= a.n_pages) phys = 0;  // (its data is never used)
        const uint8_t *src = a.pages + ((int64_t)phys * a.n_kv + h) * L::kPageBytes + 16 * lane;
        const uint32_t dst = __builtin_amdgcn_readfirstlane(lbase + C::kSlotAt + slot * C::kSlot);
#pragma unroll
        for (int i0 = 0; i0 < kMine0; ++i0) {
            const int i = wave + 4 * i0;
            if (i < kDma && (i + 1 < kDma || 1024 * i + 16 * lane < L::kPageBytes))
                dma16(src + 1024 * i, dst + 1024 * i);
        }
    };
    // at most `pages` of this wave's page loads still in flight
    auto wait_pages = [&](int pages) {
        const int after = pages * n_mine;
        if (after <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        else if (after == 1) asm volatile("s_waitcnt vmcnt(1)" ::: "memory");
        else if (after == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(3)" ::: "memory");
    };
    static_assert(kMine0 <= 3, "at most three loads per wave and page");

    // per-row state of the lane's score rows 16 w + 4 j + r, in units of
    // 2^-off (the value widening's field offset, as in decode)
    const float off = BITS == 2 ? 2.0f * (n & 1) : 0.0f;
    float m_run[4], lc[4], zc[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        m_run[r] = -FLT_MAX;
        lc[r] = zc[r] = 0.0f;
    }
    float one;
    asm("v_mov_b32 %0, 1.0" : "=v"(one));
    f32x4 acc[4][kNTw];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int c = 0; c < kNTw; ++c) acc[rt][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Page u sits in slot (u - w0) % 4 and writes its weights and rescale
    // factors to buffer (u - w0) % 2; its P V runs in the next iteration.
    auto slot_at = [&](int u) -> uint32_t { return lbase + C::kSlotAt + ((u - w0) & 3) * C::kSlot; };
    auto wbuf_at = [&](int u) -> uint32_t { return lbase + C::kWAt + ((u - w0) & 1) * C::kWBytes; };
    auto alpha_at = [&](int u) -> float * {
        return reinterpret_cast<float *>(lds + C::kAlphaAt) + ((u - w0) & 1) * C::kRows;
    };
    // tokens of page u that hold keys (0 for an entry outside the pool)
    auto page_valid = [&](int u) -> int32_t {
        const int32_t phys = __builtin_amdgcn_readlane(tbl, u - w0);
        return (phys < 0 || phys >= a.n_pages) ? 0 : min(kPage, q_hi - (a.s_sink + u * kPage));
    };
    // the score products of page u: c[t][r] = q~ . codes of row 16 w + 4 j
    // + r and token 4 n + t, the limbs accumulated in order (each product's
    // block sums are exact); kp, vp the key and value parameters of the
    // lane's tokens
    auto score_products = [&](int u, f32x4 (&c)[4], u32x4 &kp, u32x4 &vp) {
        const uint32_t pg = slot_at(u);
        u32x4 kx[kKX];
#pragma unroll
        for (int q4 = 0; q4 < kKX; ++q4) kx[q4] = lds_read16(pg + 4 * L::k_word(lane, 4 * q4));
        kp = lds_read16(pg + L::kParamOffset + 16 * n);
        vp = lds_read16(pg + L::kParamOffset + 4 * kPage + 16 * n);
        i32x8 bop[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            uint32_t w[BITS];
#pragma unroll
            for (int i = 0; i < BITS; ++i) w[i] = kx[(BITS * t + i) / 4][(BITS * t + i) % 4];
            if constexpr (BITS == 2) {
                bop[t] = i32x8{(int)(w[0] & 0x33333333u), (int)((w[0] >> 2) & 0x33333333u),
                               (int)(w[1] & 0x33333333u), (int)((w[1] >> 2) & 0x33333333u), 0, 0, 0, 0};
            } else {
                bop[t] = i32x8{(int)(w[0] & 0x0F0F0F0Fu), (int)((w[0] >> 4) & 0x0F0F0F0Fu),
                               (int)(w[1] & 0x0F0F0F0Fu), (int)((w[1] >> 4) & 0x0F0F0F0Fu),
                               (int)(w[2] & 0x0F0F0F0Fu), (int)((w[2] >> 4) & 0x0F0F0F0Fu),
                               (int)(w[3] & 0x0F0F0F0Fu), (int)((w[3] >> 4) & 0x0F0F0F0Fu)};
            }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) c[t] = limb_product<0, kFmtB, kScaleB>(qa[0], bop[t], sc03, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
        for (int t = 0; t < 4; ++t) c[t] = limb_product<1, kFmtB, kScaleB>(qa[1], bop[t], sc03, c[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) c[t] = limb_product<2, kFmtB, kScaleB>(qa[2], bop[t], sc03, c[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) c[t] = limb_product<3, kFmtB, kScaleB>(qa[3], bop[t], sc03, c[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) c[t] = limb_product<4, kFmtB, kScaleB>(qa[4], bop[t], sc45, c[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) c[t] = limb_product<5, kFmtB, kScaleB>(qa[5], bop[t], sc45, c[t]);
    };
    // the online softmax of page u over the products: the weights (fp16
    // hi + lo) and rescale factors of the wave's rows into LDS; tail: mask
    // the tokens past nvalid
    auto softmax = [&](int u, const f32x4 (&c)[4], const u32x4 &kp, const u32x4 &vp, bool tail,
                       int32_t nvalid) {
        const uint32_t wbase = wbuf_at(u);
        float *alpha = alpha_at(u);
        float ks[4], kz[4], vs[4], vz[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            ks[t] = f16_bits_to_f32(kp[t] & 0xFFFFu);
            kz[t] = f16_bits_to_f32(kp[t] >> 16);
            vs[t] = f16_bits_to_f32(vp[t] & 0xFFFFu);
            vz[t] = f16_bits_to_f32(vp[t] >> 16);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int rz = 16 * wave + 4 * j + r;  // the row, in the block's 64
            float lg[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) lg[t] = fmaf(ks[t], c[t][r], kz[t] * zs[r]);
            if (tail) {
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    if (4 * n + t >= nvalid) lg[t] = -INFINITY;
            }
            // online softmax of row rz over this page's tokens 4 n .. 4 n + 3
            const float mx = row_max16(fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3])));
            // (m_run starts at -FLT_MAX, so m_new is finite: a first page
            // scales zeros by exp2(-huge) = 0, and a row with no key yet
            // keeps weights exp2(-inf) = 0)
            const float m_new = fmaxf(m_run[r], mx);
            const float al = fexp2(m_run[r] - m_new);
            lc[r] *= al;
            zc[r] *= al;
            m_run[r] = m_new;
            alpha[rz] = al;  // (the row's 16 lanes store the same value)
            const float mo = m_new + off;
            float wgt[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const float pw = fexp2(lg[t] - mo);
                lc[r] += pw;
                zc[r] = fmaf(pw, vz[t], zc[r]);
                wgt[t] = fmaf(pw, vs[t], 0.0f);
            }
            // fp16 hi parts, then the lo parts w - hi in one rounding each
            // (one mixed-precision fma per weight: `one` is opaque to the
            // compiler, which would otherwise fold the product away)
            const uint32_t h01 = pack_f16_rne(wgt[0], wgt[1]);
            const uint32_t h23 = pack_f16_rne(wgt[2], wgt[3]);
            const uint32_t l01 = pack_f16_rne(fmaf(-f16_bits_to_f32(h01 & 0xFFFFu), one, wgt[0]),
                                              fmaf(-f16_bits_to_f32(h01 >> 16), one, wgt[1]));
            const uint32_t l23 = pack_f16_rne(fmaf(-f16_bits_to_f32(h23 & 0xFFFFu), one, wgt[2]),
                                              fmaf(-f16_bits_to_f32(h23 >> 16), one, wgt[3]));
            lds_write8(wbase + tbuf_at(rz, 8 * n), h01, h23);
            lds_write8(wbase + C::kRows * 128 + tbuf_at(rz, 8 * n), l01, l23);
        }
    };
    // P V of page u: all 64 rows, this wave's channel tiles
    auto pv = [&](int u) {
        // lane (j, n) holds query rows 16 rt + 4 j + i (i < 4) of row tile
        // rt; the hi and lo weights are two products into the same sums
        const uint32_t pg = slot_at(u);
        const uint32_t wbase = wbuf_at(u);
        const float *alpha = alpha_at(u);
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            const f32x4 al = *reinterpret_cast<const f32x4 *>(alpha + 16 * rt + 4 * j);
#pragma unroll
            for (int c = 0; c < kNTw; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[rt][c][i] *= al[i];
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
            // this wave's value codes for tokens 32 kc .., channel tiles
            // kNTw w .. (words vw = nt / kOpw of the lane)
            uint32_t op[kNTw][4];
#pragma unroll
            for (int cw = 0; cw < kNTw / kOpw; ++cw) {
                const int vw = (kNTw * wave) / kOpw + cw;
                const uint32_t word = *(const __attribute__((address_space(3))) uint32_t *)(uintptr_t)(
                    pg + L::kRegionBytes + 4 * L::v_word(lane, kc * 2 * L::kNw + vw));
                uint32_t wide[L::kCodesPerWord / 2];
                widen_word_f16<BITS>(word, wide);
#pragma unroll
                for (int o = 0; o < kOpw; ++o)
#pragma unroll
                    for (int q = 0; q < 4; ++q) op[cw * kOpw + o][q] = wide[4 * o + q];
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                for (int part = 0; part < 2; ++part) {
                    const f16x8 A = __builtin_bit_cast(
                        f16x8, lds_read16(wbase + part * C::kRows * 128 + tbuf_at(16 * rt + n, 64 * kc + 16 * j)));
#pragma unroll
                    for (int c = 0; c < kNTw; ++c) acc[rt][c] = mfma16h(A, as_op_h(op[c]), acc[rt][c]);
                }
        }
    };

    // Software pipeline over the run, one barrier per page: iteration u
    // waits for page u's loads, then (barrier) issues page u + 2 into the
    // slot page u - 2 has left, runs the P V of page u - 1 (its weights
    // complete) and the scores of page u.
    const bool run = a.n_pages > 0 && w0 < w1;
    if (run) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // the page table and query reads have returned
        issue(w0, 0);
        if (w0 + 1 < w1) issue(w0 + 1, 1);
        wait_pages(w0 + 1 < w1 ? 1 : 0);
        __syncthreads();
        if (w0 + 2 < w1) issue(w0 + 2, 2);
        {
            f32x4 c[4];
            u32x4 kp, vp;
            const int32_t nv = page_valid(w0);
            score_products(w0, c, kp, vp);
            softmax(w0, c, kp, vp, nv < kPage, nv);
        }
        for (int u = w0 + 1; u < w1; ++u) {
            wait_pages(u + 1 < w1 ? 1 : 0);
            __syncthreads();  // page u is in; page u - 1's weights are written
            if (u + 2 < w1) issue(u + 2, (u + 2 - w0) & 3);
            const int32_t nv = page_valid(u);
            f32x4 c[4];
            u32x4 kp, vp;
            if (nv == kPage) {
                // a full page: one branch-free region, page u's products and
                // page u - 1's P V interleaved with the softmax arithmetic
                score_products(u, c, kp, vp);
                pv(u - 1);
                softmax(u, c, kp, vp, false, kPage);
#pragma unroll
                for (int i = 0; i < 24; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // a score product
                    __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // vector arithmetic
                }
#pragma unroll
                for (int i = 0; i < 32; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // a P V product
                    __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
                }
            } else {
                pv(u - 1);
                score_products(u, c, kp, vp);
                softmax(u, c, kp, vp, true, nv);
            }
        }
        __syncthreads();
        pv(w1 - 1);
    }

    // ---- partials: each row's m, l and z term from its owner wave, then
    // every wave its channel tiles of o
    float *zrow = reinterpret_cast<float *>(lds + C::kZAt);
    float *mrow = reinterpret_cast<float *>(lds + C::kMAt);
    float *lrow = reinterpret_cast<float *>(lds + C::kLAt);
    {
        const float f = ldexpf(1.0f, (int)off);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float zt = row_sum16(zc[r] * f);
            const float lt = row_sum16(lc[r] * f);
            if (n == 0) {
                const int rz = 16 * wave + 4 * j + r;
                zrow[rz] = zt;
                mrow[rz] = m_run[r] == -FLT_MAX ? -INFINITY : m_run[r];  // no key: -inf
                lrow[rz] = lt;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 16 * rt + 4 * j + i;
            const int tg = tg0 + r / G;
            if (tg >= a.n_groups) continue;
            const int64_t bzr = (int64_t)b * a.n_groups + tg;
            float *pr = a.part + ((bzr * a.n_kv + h) * a.n_splits + split) * G * (D + 2) + (r % G) * (D + 2);
            const float mx = mrow[r];
#pragma unroll
            for (int c = 0; c < kNTw; ++c) {
                const int ch = 16 * (kNTw * wave + c) + n;
                pr[ch] = mx == -INFINITY ? 0.0f : fmaf(acc[rt][c][i], kOutScale, zrow[r]);
            }
            if (wave == 0 && n == 0) {
                pr[D] = mx;
                pr[D + 1] = lrow[r];
            }
        }
}

// ------------------------------------------------------------------ chunk windows

// The bf16 window slots of chunk attention at d = 128, merged with the page
// runs of chunk_pages_kernel into the output (so no combine launch follows).
// One workgroup per (kv head, sequence, block of eight token groups, quarter
// of the block's 64 query rows): its 16 rows, the rows of chunk_pages_kernel's
// wave of the same index.  Wave w takes the 64-slot window units w, w + 4,
// .., each staged whole in the wave's own LDS buffer (keys and channel-major
// values, direct-to-LDS loads).  Per unit:
//   scores  q~ in bf16 hi + lo parts (A, the 16 rows) times the keys, tile t
//           column n the slot 4 n + t, so that lane (j, n) holds rows 4 j + r
//           of slots 4 n .. 4 n + 3; causal and live-slot masks;
//   softmax online across the wave's units; the lane's rows are its P V
//           rows, so the rescale stays in the lane;
//   P V     weights (bf16 hi, lo: two products) through a per-wave LDS
//           buffer, times the values (dead slots' values zeroed).
// Then the four waves' results and the row's page-run partials merge by
// log-sum-exp (as decode_combine_kernel does), eight splits' loads at a time.
struct ChunkWinLds {
    static constexpr int kUnitK = 64 * 256;                 // [slot][16 chunks of 16 B]
    static constexpr int kUnitV = 128 * 128;                // [channel][8 chunks of 16 B]
    static constexpr int kUnit = kUnitK + kUnitV;           // one per wave
    static constexpr int kPWave = 2 * 16 * 128;             // [part][16 rows][64 slots] bf16
    static constexpr int kPAt = 4 * kUnit;
    static constexpr int kBytes = kPAt + 4 * kPWave;
};

__global__ void __launch_bounds__(256, 1) chunk_window_kernel(DecodeArgs a, float *out)
{
    constexpr int D = 128, G = 8;
    using W = ChunkWinLds;
    __shared__ __attribute__((aligned(16))) uint8_t lds[W::kBytes];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j = lane >> 4, n = lane & 15;
    const int h = blockIdx.x;
    const int n_blocks = (a.n_groups + 7) / 8;
    const int blk = (int)blockIdx.y >> 2, r0 = 16 * ((int)blockIdx.y & 3);
    const int b = blk / n_blocks, tg0 = 8 * (blk % n_blocks);
    const int32_t S = a.seq_len[b];
    int32_t qend = a.quant_end[b];
    qend = qend < S ? qend : S;
    const int32_t q_hi = qend > a.s_sink ? qend : a.s_sink;
    const int32_t ring = a.win_slots - a.s_sink;
    // the ring holds positions [q_hi, S); the oldest sits at ring index a0
    const int32_t a0 = S > q_hi ? (q_hi - a.s_sink) % ring : 0;
    const int32_t ring_live = S > q_hi ? S - q_hi : 0;
    const int32_t nb = chunk_tokens(a.n_tok, a.max_tok, b, S);
    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;
    const int n_units = a.win_slots / kPage;
    const uint32_t lbase = lds_addr(lds);

    // row rr of the block (0 .. 63): its q~ row (-1: past the token groups)
    // and chunk token
    auto qt_row = [&](int rr) -> int64_t {
        const int tg = tg0 + rr / G;
        return tg < a.n_groups ? (((int64_t)b * a.n_groups + tg) * a.n_kv + h) * G + rr % G : -1;
    };
    auto chunk_tok = [&](int rr) -> int32_t { return (tg0 + rr / G) * a.tpg + (rr % G) / a.g_real; };

    // unit u's keys and values into the wave's buffer: LDS chunk p of the
    // keys is slot p / 16, chunk (p % 16) ^ ((slot / 4) % 16); of the values
    // channel p / 8, chunk (p % 8) ^ (channel % 8) (the readers' bank
    // swizzles)
    const uint32_t kb = lbase + wave * W::kUnit, vb = kb + W::kUnitK;
    auto issue = [&](int u) {
        const int32_t unit0 = u * kPage;
#pragma unroll 4
        for (int i = 0; i < 16; ++i) {
            const int pk = 64 * i + lane;
            const int slot = pk >> 4, ck = (pk & 15) ^ ((slot >> 2) & 15);
            dma16(a.win_k + (head_win + unit0 + slot) * D + 8 * ck, __builtin_amdgcn_readfirstlane(kb + 1024 * i));
            const int ch = pk >> 3, cv = (pk & 7) ^ (ch & 7);
            dma16(a.win_v + head_win * D + (int64_t)ch * a.win_slots + unit0 + 8 * cv,
                  __builtin_amdgcn_readfirstlane(vb + 1024 * i));
        }
    };
    if (wave < n_units) issue(wave);

    // A operands: q~ of row r0 + n (lane n), channels 32 c + 8 j .., as
    // bf16 hi and lo parts
    bf16x8 qh[4], ql[4];
    {
        const int64_t row = qt_row(r0 + n);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
            if (row >= 0) {
                const float *src = a.qt + row * D + 32 * c + 8 * j;
                const f32x4 x0 = *reinterpret_cast<const f32x4 *>(src);
                const f32x4 x1 = *reinterpret_cast<const f32x4 *>(src + 4);
                const float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
#pragma unroll
                for (int pp = 0; pp < 4; ++pp) {
                    hi[pp] = pack_bf16_rne(x[2 * pp], x[2 * pp + 1]);
                    lo[pp] = pack_bf16_rne(x[2 * pp] - bf16_bits_to_f32(hi[pp] & 0xFFFFu),
                                           x[2 * pp + 1] - bf16_bits_to_f32(hi[pp] >> 16));
                }
            }
            qh[c] = __builtin_bit_cast(bf16x8, u32x4{hi[0], hi[1], hi[2], hi[3]});
            ql[c] = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], lo[2], lo[3]});
        }
    }
    // the lane's rows r0 + 4 j + r: chunk token (or -1: no such row)
    int32_t trow[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int rr = r0 + 4 * j + r;
        trow[r] = qt_row(rr) >= 0 ? chunk_tok(rr) : -1;
    }

    float m_run[4], lsum[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        m_run[r] = -INFINITY;
        lsum[r] = 0.0f;
    }
    f32x4 acc[8];  // P V: lane (j, n) rows 4 j + i, channel 16 nt + n
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const uint32_t pbuf = lbase + W::kPAt + wave * W::kPWave;

    for (int u = wave; u < n_units; u += 4) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the wave's loads of unit u
        const int32_t unit0 = u * kPage;
        // slots of the unit that hold a position (bit s: slot unit0 + s,
        // lane s answers), and the lane's slots 4 n + t with their positions
        uint64_t live_mask;
        {
            const int32_t sl = unit0 + lane;
            const int32_t ri = (sl - a.s_sink - a0 + ring) % ring;
            live_mask = __ballot(sl < a.s_sink ? sl < S : ri < ring_live);
        }
        int32_t pos[4];
        bool live[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int32_t sl = unit0 + 4 * n + t;
            const int32_t ri = (sl - a.s_sink - a0 + ring) % ring;
            live[t] = sl < a.s_sink ? sl < S : ri < ring_live;
            pos[t] = sl < a.s_sink ? sl : q_hi + ri;
        }
        if (live_mask != 0) {
            // ---- scores
            f32x4 sc[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                sc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
                const uint32_t krow = kb + (4 * n + t) * 256;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const bf16x8 kk = __builtin_bit_cast(bf16x8, lds_read16(krow + 16 * ((4 * c + j) ^ n)));
                    sc[t] = mfma16(qh[c], kk, sc[t]);
                    sc[t] = mfma16(ql[c], kk, sc[t]);
                }
            }
            // ---- online softmax of the lane's rows over the unit
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float lg[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const bool vis = live[t] && trow[r] >= 0 && trow[r] < nb && pos[t] <= S - nb + trow[r];
                    lg[t] = vis ? sc[t][r] : -INFINITY;
                }
                const float mx = row_max16(fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3])));
                const float m_new = fmaxf(m_run[r], mx);
                const float al = m_new == -INFINITY ? 1.0f : fexp2(m_run[r] - m_new);
                m_run[r] = m_new;
                lsum[r] *= al;
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) acc[nt][r] *= al;
                uint32_t hw[2], lw[2];
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const float p0 = m_new == -INFINITY ? 0.0f : fexp2(lg[2 * e] - m_new);
                    const float p1 = m_new == -INFINITY ? 0.0f : fexp2(lg[2 * e + 1] - m_new);
                    lsum[r] += p0 + p1;
                    hw[e] = pack_bf16_rne(p0, p1);
                    lw[e] = pack_bf16_rne(p0 - bf16_bits_to_f32(hw[e] & 0xFFFFu),
                                          p1 - bf16_bits_to_f32(hw[e] >> 16));
                }
                lds_write8(pbuf + tbuf_at(4 * j + r, 8 * n), hw[0], hw[1]);
                lds_write8(pbuf + 16 * 128 + tbuf_at(4 * j + r, 8 * n), lw[0], lw[1]);
            }
            // ---- P V (the weight buffer is the wave's own: no barrier)
            const bool dead = ~live_mask != 0;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const bf16x8 ph = __builtin_bit_cast(bf16x8, lds_read16(pbuf + tbuf_at(n, 64 * kc + 16 * j)));
                const bf16x8 pl =
                    __builtin_bit_cast(bf16x8, lds_read16(pbuf + 16 * 128 + tbuf_at(n, 64 * kc + 16 * j)));
                // dead slots 32 kc + 8 j + e: their values are zeroed
                uint32_t msk[4] = {~0u, ~0u, ~0u, ~0u};
                if (dead) {
                    const uint32_t bits8 = (uint32_t)(live_mask >> (32 * kc + 8 * j)) & 0xFFu;
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        msk[q] = ((bits8 >> (2 * q)) & 1u ? 0x0000FFFFu : 0u) |
                                 ((bits8 >> (2 * q + 1)) & 1u ? 0xFFFF0000u : 0u);
                }
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) {
                    const int ch = 16 * nt + n;
                    u32x4 v = lds_read16(vb + ch * 128 + 16 * ((4 * kc + j) ^ (ch & 7)));
#pragma unroll
                    for (int q = 0; q < 4; ++q) v[q] &= msk[q];
                    const bf16x8 vv = __builtin_bit_cast(bf16x8, v);
                    acc[nt] = mfma16(ph, vv, acc[nt]);
                    acc[nt] = mfma16(pl, vv, acc[nt]);
                }
            }
        }
        if (u + 4 < n_units) {
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the unit's reads are done
            issue(u + 4);
        }
    }

    // ---- merge: the four waves' results through LDS (the unit buffers are
    // free once every wave is past its units), then thread (row tid / 16,
    // channels 8 (tid % 16) ..) adds its row's page-run partials
#pragma unroll
    for (int r = 0; r < 4; ++r) lsum[r] = row_sum16(lsum[r]);
    __syncthreads();
    float *wo = reinterpret_cast<float *>(lds);  // [wave][16 rows][D]
    float *wml = wo + 4 * 16 * D;                // [wave][16 rows][m, l]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ri = 4 * j + i;
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) wo[(wave * 16 + ri) * D + 16 * nt + n] = acc[nt][i];
        if (n == 0) {
            wml[2 * (wave * 16 + ri)] = m_run[i];
            wml[2 * (wave * 16 + ri) + 1] = lsum[i];
        }
    }
    __syncthreads();
    const int ri = tid >> 4, c0 = 8 * (tid & 15), rr = r0 + ri;
    if (qt_row(rr) < 0) return;
    const int32_t t = chunk_tok(rr);
    if (t >= a.max_tok) return;
    float *dst = out + (((int64_t)b * a.max_tok + t) * a.n_kv * a.g_real + h * a.g_real + (rr % G) % a.g_real) * D + c0;
    f32x4 o[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    float l = 0.0f, M = -INFINITY;
    if (t < nb) {
        // running (M, o, l); a batch of partials joins with the new maximum
        auto join = [&](float mb) -> float {
            const float m_new = fmaxf(M, mb);
            const float f = (M == -INFINITY) ? 0.0f : fexp2(M - m_new);
            o[0] = f32x4{f * o[0][0], f * o[0][1], f * o[0][2], f * o[0][3]};
            o[1] = f32x4{f * o[1][0], f * o[1][1], f * o[1][2], f * o[1][3]};
            l *= f;
            M = m_new;
            return m_new;
        };
        auto add = [&](float ms, float ls, const f32x4 &x0, const f32x4 &x1) {
            const float f = (ms == -INFINITY) ? 0.0f : fexp2(ms - M);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                o[0][k] = fmaf(f, x0[k], o[0][k]);
                o[1][k] = fmaf(f, x1[k], o[1][k]);
            }
            l = fmaf(f, ls, l);
        };
        float mw[4];
#pragma unroll
        for (int w = 0; w < 4; ++w) mw[w] = wml[2 * (w * 16 + ri)];
        join(fmaxf(fmaxf(mw[0], mw[1]), fmaxf(mw[2], mw[3])));
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float *src = wo + (w * 16 + ri) * D + c0;
            add(mw[w], wml[2 * (w * 16 + ri) + 1], *reinterpret_cast<const f32x4 *>(src),
                *reinterpret_cast<const f32x4 *>(src + 4));
        }
        const int64_t bzr = (int64_t)b * a.n_groups + tg0 + rr / G;
        const float *pp = a.part + ((bzr * a.n_kv + h) * a.n_splits) * G * (D + 2) + (rr % G) * (D + 2);
        const int64_t stride = (int64_t)G * (D + 2);
        for (int s0 = 0; s0 < a.n_page_splits; s0 += 8) {
            float ms[8], ls[8];
            f32x4 x[8][2];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const bool in = s0 + e < a.n_page_splits;
                const float *src = pp + (in ? s0 + e : s0) * stride;  // (a repeat weighs 0)
                ms[e] = in ? src[D] : -INFINITY;
                ls[e] = src[D + 1];
                x[e][0] = *reinterpret_cast<const f32x4 *>(src + c0);
                x[e][1] = *reinterpret_cast<const f32x4 *>(src + c0 + 4);
            }
            float mb = ms[0];
#pragma unroll
            for (int e = 1; e < 8; ++e) mb = fmaxf(mb, ms[e]);
            join(mb);
#pragma unroll
            for (int e = 0; e < 8; ++e) add(ms[e], ls[e], x[e][0], x[e][1]);
        }
    }
#pragma unroll
    for (int q = 0; q < 2; ++q)
        reinterpret_cast<f32x4 *>(dst)[q] = l > 0.0f ? f32x4{o[q][0] / l, o[q][1] / l, o[q][2] / l, o[q][3] / l}
                                                  : f32x4{0.f, 0.f, 0.f, 0.f};
}

// ------------------------------------------------------------------ combine

// One workgroup per (query head, sequence): the split maxima and weights go
// through LDS, then every channel thread sums its column with the loads
// unrolled so they are in flight together.
template <int D>
__global__ void __launch_bounds__(D) decode_combine_kernel(const float *part, float *out,
                                                           int32_t n_kv, int32_t G,
                                                           int32_t n_splits, DecodeArgs a)
{
    __shared__ float fw[kMaxSplits];
    __shared__ float red[D];
    // virtual head qh = (h, v) of grid row bz = (b, token group tg): chunk
    // token tg tpg + v / g_real, query head h g_real + v % g_real
    const int qh = blockIdx.x, bz = blockIdx.y;
    const int h = qh / G, g = qh % G;
    const int ch = threadIdx.x;
    float *dst;
    if (a.max_tok == 1 && a.n_tok == nullptr) {
        dst = out + ((int64_t)bz * n_kv * G + qh) * D;  // decode: row bz = b, head qh
    } else {
        const int b = bz / a.n_groups, tg = bz % a.n_groups;
        const int t = tg * a.tpg + g / a.g_real;
        if (t >= a.max_tok) return;
        dst = out + (((int64_t)b * a.max_tok + t) * n_kv * a.g_real + h * a.g_real + g % a.g_real) * D;
        if (t >= chunk_tokens(a.n_tok, a.max_tok, b, a.seq_len[b])) {
            dst[ch] = 0.0f;  // beyond this sequence's chunk
            return;
        }
    }
    const int64_t stride = (int64_t)G * (D + 2);
    const float *pp = part + (((int64_t)bz * n_kv + h) * n_splits) * stride + g * (D + 2);
    merge_splits<D>(pp, stride, n_splits, dst, ch, fw, red);
}

// ------------------------------------------------------------------ host

struct DecodePlan {
    int32_t units_per_wave, n_page_splits, n_splits, win_units;
    size_t qt_bytes, limb_bytes, aux_bytes, part_bytes;
};

template <int D, int BITS, int G>
static void main_kernel_ptr(const void *&f, bool share)
{
    if (share) f = reinterpret_cast<const void *>(&decode_main_kernel<D, BITS, G, false, true>);
    else f = reinterpret_cast<const void *>(&decode_main_kernel<D, BITS, G, true, false>);
}

// Waves of decode_main_kernel the device keeps resident at once (its
// occupancy from registers and LDS, times the compute units), cached per
// variant: the query-forming one, or with share the shared-items one;
// 256 compute units at three workgroups each when no device answers.  The
// cache entries are atomics: concurrent first calls compute the same value
// and store it, so the cache is safe to fill from any thread.
static int64_t resident_waves(int D, int bits, int G, bool share)
{
    static std::atomic<int64_t> cache[2][2][2][4] = {};
    const int di = D == 128, bi = bits == 4, gi = G == 1 ? 0 : G == 2 ? 1 : G == 4 ? 2 : 3;
    std::atomic<int64_t> &slot = cache[share][di][bi][gi];
    const int64_t known = slot.load(std::memory_order_relaxed);
    if (known > 0) return known;
    const void *f = nullptr;
    const int key = D * 100 + bits * 10 + gi;
    switch (key) {
        case 12820: main_kernel_ptr<128, 2, 1>(f, share); break;
        case 12821: main_kernel_ptr<128, 2, 2>(f, share); break;
        case 12822: main_kernel_ptr<128, 2, 4>(f, share); break;
        case 12823: main_kernel_ptr<128, 2, 8>(f, share); break;
        case 12840: main_kernel_ptr<128, 4, 1>(f, share); break;
        case 12841: main_kernel_ptr<128, 4, 2>(f, share); break;
        case 12842: main_kernel_ptr<128, 4, 4>(f, share); break;
        case 12843: main_kernel_ptr<128, 4, 8>(f, share); break;
        case 6420: main_kernel_ptr<64, 2, 1>(f, share); break;
        case 6421: main_kernel_ptr<64, 2, 2>(f, share); break;
        case 6422: main_kernel_ptr<64, 2, 4>(f, share); break;
        case 6423: main_kernel_ptr<64, 2, 8>(f, share); break;
        case 6440: main_kernel_ptr<64, 4, 1>(f, share); break;
        case 6441: main_kernel_ptr<64, 4, 2>(f, share); break;
        case 6442: main_kernel_ptr<64, 4, 4>(f, share); break;
        default: main_kernel_ptr<64, 4, 8>(f, share); break;
    }
    int dev = 0, ncu = 0, blocks = 0;
    int64_t waves = 256 * 3 * 4;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, f, 256, 0) == hipSuccess && ncu > 0 &&
        blocks > 0)
        waves = (int64_t)ncu * blocks * 4;
    else
        (void)hipGetLastError();
    slot.store(waves, std::memory_order_relaxed);
    return waves;
}

// Compute units of the current device (256 when no device answers),
// cached like resident_waves.
static int64_t device_cus()
{
    static std::atomic<int64_t> cache{0};
    const int64_t known = cache.load(std::memory_order_relaxed);
    if (known > 0) return known;
    int dev = 0, ncu = 0;
    int64_t v = 256;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && ncu > 0)
        v = ncu;
    else
        (void)hipGetLastError();
    cache.store(v, std::memory_order_relaxed);
    return v;
}

// Query rows of a call: G virtual heads per kv head, each a (chunk token,
// query head) pair, and n_groups token groups per sequence (see DecodeArgs).
struct RowShape {
    int32_t g_real, tpg, G, n_groups, max_tok;
    bool share;  // several token groups: four waves share each work item
};

static RowShape row_shape(const wushkv_cache *c, int32_t n_q, int32_t max_tok)
{
    RowShape r;
    r.g_real = n_q / c->n_kv_heads;
    r.max_tok = max_tok;
    r.tpg = 1;
    while (r.g_real * r.tpg * 2 <= 8 && r.tpg < max_tok) r.tpg *= 2;
    r.G = r.g_real * r.tpg;
    r.n_groups = (max_tok + r.tpg - 1) / r.tpg;
    r.share = r.n_groups > 1;
    return r;
}

// Longest page run of one wave: its page-table entries sit one per lane.
constexpr int64_t kMaxRunPages = 64;

static bool make_plan(const wushkv_cache *c, const RowShape &rs, int32_t max_seq_len, DecodePlan &p,
                      bool one_window_wg = false)
{
    const int32_t G = rs.G;
    const int64_t qpages = max_seq_len > c->s_sink ? (max_seq_len - c->s_sink + kPage - 1) / kPage : 0;
    const int64_t rows_z = (int64_t)c->batch * rs.n_groups;  // grid z
    const int64_t heads = rows_z * c->n_kv_heads;
    const int64_t n_q = (int64_t)c->n_kv_heads * G;          // virtual query heads per row
    // One residency round if it can be had: the page waves get what the
    // window workgroups leave of the resident waves; at least 2 and at most
    // 16 pages per wave (when the work cannot fit one round, shorter waves
    // balance the last round better).
    const int64_t wunits = c->win_slots / kPage;
    // Window workgroups: one per 64-slot unit, four waves on its four tiles;
    // with shared work items (share) one per row for all units, since there
    // every wave walks all the tiles anyway and the page runs then get the
    // resident slots the other window workgroups would hold.
    int64_t win_units = (rs.share || one_window_wg) ? wunits : 1;
    int64_t wwgs = (wunits + win_units - 1) / win_units;
    // With shared work items (share_items) the four waves of a workgroup
    // walk one run together, each for another token group: a workgroup row
    // is then a (sequence, four token groups, kv head) triple and a split
    // covers upw pages instead of 4 upw.
    const int64_t per_split = rs.share ? 1 : 4;
    const int64_t wg_rows = rs.share ? (int64_t)c->batch * ((rs.n_groups + 3) / 4) * c->n_kv_heads : heads;
    const int64_t budget = resident_waves(c->head_dim, storage_bits(c->bits), G, rs.share) - 4 * wg_rows * wwgs;
    const int64_t upw_max = rs.share ? 64 : 16;
    int64_t upw = 2;
    while (upw < upw_max && wg_rows * ((qpages + per_split * upw - 1) / (per_split * upw)) * 4 > budget) ++upw;
    int64_t psplits = (qpages + per_split * upw - 1) / (per_split * upw);
    // the same number of runs, evened out (the last one is not left short)
    if (psplits > 0) {
        upw = (qpages + per_split * psplits - 1) / (per_split * psplits);
        psplits = (qpages + per_split * upw - 1) / (per_split * upw);
    }
    // Chunks at d = 128 run their pages in chunk_pages_kernel: a workgroup
    // per run of upw pages takes the 64 rows of eight token groups; the
    // runs are sized for about two such workgroups per compute unit, one
    // round.  The window slots and the merge follow in chunk_window_kernel,
    // so the splits are the page runs alone.
    if (rs.share && c->head_dim == 128 && G == 8) {
        const int64_t per_cu = 2;
        const int64_t crows = (int64_t)c->batch * ((rs.n_groups + 7) / 8) * c->n_kv_heads;
        int64_t runs = (per_cu * device_cus() + crows - 1) / crows;
        runs = runs < 1 ? 1 : (runs > qpages ? qpages : runs);
        upw = qpages > 0 ? (qpages + runs - 1) / runs : 1;
        if (upw > kMaxRunPages) upw = kMaxRunPages;
        psplits = (qpages + upw - 1) / upw;
        win_units = 1;
        wwgs = 0;
    }
    // A decode grid that cannot be resident at once (it runs in rounds)
    // takes one window workgroup per row, its waves on every unit's tiles:
    // a third as many workgroups, each with an online softmax over its
    // tiles, instead of one per 64-slot unit.
    if (!rs.share && !one_window_wg && wunits > 1 &&
        (psplits + wwgs) * heads * 4 > resident_waves(c->head_dim, storage_bits(c->bits), G, false))
        return make_plan(c, rs, max_seq_len, p, true);
    if (psplits + wwgs > kMaxSplits) {
        const int64_t room = kMaxSplits - wwgs;
        if (room < 1) return false;
        upw = (qpages + per_split * room - 1) / (per_split * room);
        psplits = (qpages + per_split * upw - 1) / (per_split * upw);
    }
    const int64_t splits = psplits + wwgs;  // and the window workgroups
    // a wave keeps the page-table entries of its run in its 64 lanes, one
    // each (the run's k-th page is lane k's entry), so a run is at most 64
    // pages long: longer contexts than kMaxSplits runs of 64 cover are not
    // planned (the caller gets WUSHKV_EUNSUPPORTED)
    if (splits > kMaxSplits || upw > kMaxRunPages) return false;
    p.units_per_wave = (int32_t)upw;
    p.win_units = (int32_t)win_units;
    p.n_page_splits = (int32_t)psplits;
    p.n_splits = (int32_t)splits;
    p.qt_bytes = ((size_t)rows_z * n_q * c->head_dim * 4 + 255) / 256 * 256;
    p.limb_bytes = (size_t)rows_z * n_q * kLimbs * 128;
    p.aux_bytes = ((size_t)rows_z * n_q * 16 + 255) / 256 * 256;
    p.part_bytes = (size_t)heads * splits * G * (c->head_dim + 2) * 4;
    return true;
}

// The main kernel, preceded by decode_qt_kernel unless it forms q~ itself
// (rows_z: grid rows of the query rows, one per (sequence, token group)).
template <int D, int BITS, int G>
static void launch_main(bool form, bool share, dim3 grid, unsigned rows_z, hipStream_t s,
                        const DecodeArgs &a)
{
    if (form) {
        launch("decode_main_kernel", decode_main_kernel<D, BITS, G, true, false>, grid, dim3(256), s, a);
        return;
    }
    launch("decode_qt_kernel", decode_qt_kernel<D, BITS, G>, dim3(grid.x, rows_z), dim3(256), s, a);
    if (share)
        launch("decode_main_kernel", decode_main_kernel<D, BITS, G, false, true>, grid, dim3(256), s, a);
    else
        launch("decode_main_kernel", decode_main_kernel<D, BITS, G, false, false>, grid, dim3(256), s, a);
}

template <int D, int BITS>
static void launch_main_g(int G, bool form, bool share, dim3 grid, unsigned rows_z, hipStream_t s,
                          const DecodeArgs &a)
{
    switch (G) {
        case 1: launch_main<D, BITS, 1>(form, share, grid, rows_z, s, a); break;
        case 2: launch_main<D, BITS, 2>(form, share, grid, rows_z, s, a); break;
        case 4: launch_main<D, BITS, 4>(form, share, grid, rows_z, s, a); break;
        default: launch_main<D, BITS, 8>(form, share, grid, rows_z, s, a); break;
    }
}

}  // namespace wushkv

using namespace wushkv;

int wushkv_validate_cache(const wushkv_cache *c);  // api.hip

static int check_decode_args(const wushkv_cache *c, int32_t n_q, int32_t max_seq_len)
{
    int st = wushkv_validate_cache(c);
    if (st != WUSHKV_OK) return st;
    if (n_q <= 0 || max_seq_len < 0 || n_q % c->n_kv_heads != 0) return WUSHKV_EINVAL;
    const int32_t G = n_q / c->n_kv_heads;
    if (G > 8 || (G & (G - 1)) != 0) return WUSHKV_EUNSUPPORTED;
    return WUSHKV_OK;
}

// A chunk must lie inside the recent window (at most s_keep tokens): every
// quantised position then precedes it.
static int check_chunk(const wushkv_cache *c, int32_t max_tok)
{
    if (max_tok < 1 || max_tok > c->s_keep) return WUSHKV_EINVAL;
    return WUSHKV_OK;
}

static size_t workspace_bytes(const wushkv_cache *c, int32_t n_q, int32_t max_tok, int32_t max_seq_len)
{
    if (check_decode_args(c, n_q, max_seq_len) != WUSHKV_OK) return 0;
    DecodePlan p;
    if (!make_plan(c, row_shape(c, n_q, max_tok), max_seq_len, p)) return 0;
    return p.qt_bytes + p.limb_bytes + p.aux_bytes + p.part_bytes;
}

// The new tokens of a fused step (wushkv_decode_step).
struct StepIn {
    const int32_t *n_new;
    const uint16_t *k_new, *v_new, *t_k;
};

int wushkv_step_finish(const wushkv_cache *c, const int32_t *n_new, const float *part, float *out,
                       int32_t G, int32_t n_splits, hipStream_t s);  // append.hip

static int attend(const wushkv_cache *c, const uint16_t *q, const int32_t *n_tok, int32_t max_tok,
                  int32_t n_q_heads, int32_t max_seq_len, const float *t_k_inv, float sm_scale,
                  float *out, void *workspace, size_t workspace_bytes, wushkv_stream_t stream,
                  const StepIn *step = nullptr)
{
    int st = check_decode_args(c, n_q_heads, max_seq_len);
    if (st != WUSHKV_OK) return st;
    if (!q || !t_k_inv || !out || !workspace) return WUSHKV_EINVAL;
    if (((uintptr_t)q | (uintptr_t)t_k_inv | (uintptr_t)out | (uintptr_t)workspace) & 15u)
        return WUSHKV_EINVAL;
    if (!(sm_scale > 0.0f) || sm_scale == INFINITY) return WUSHKV_EINVAL;
    const RowShape rs = row_shape(c, n_q_heads, max_tok);
    DecodePlan p;
    if (!make_plan(c, rs, max_seq_len, p)) return WUSHKV_EUNSUPPORTED;
    if (workspace_bytes < p.qt_bytes + p.limb_bytes + p.aux_bytes + p.part_bytes) return WUSHKV_EWORKSPACE;

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int32_t G = rs.G;
    uint8_t *ws = reinterpret_cast<uint8_t *>(workspace);
    float *part = reinterpret_cast<float *>(ws);
    float *qt = reinterpret_cast<float *>(ws + p.part_bytes);
    uint8_t *qlimb = ws + p.part_bytes + p.qt_bytes;
    uint32_t *qaux = reinterpret_cast<uint32_t *>(ws + p.part_bytes + p.qt_bytes + p.limb_bytes);

    DecodeArgs a{};
    a.pages = c->pages;
    a.page_table = c->page_table;
    a.win_k = c->win_k;
    a.win_v = c->win_v;
    a.seq_len = c->seq_len;
    a.quant_end = c->quant_end;
    a.n_kv = c->n_kv_heads;
    a.s_sink = c->s_sink;
    a.win_slots = c->win_slots;
    a.max_pages = c->max_pages_per_seq;
    a.n_pages = c->n_pages;
    a.n_q = c->n_kv_heads * G;
    a.units_per_wave = p.units_per_wave;
    a.n_page_splits = p.n_page_splits;
    a.n_splits = p.n_splits;
    a.win_units = p.win_units;
    a.q = q;
    a.tinv = t_k_inv;
    a.scale = sm_scale * kLog2e;
    a.part = part;
    a.qt = qt;
    a.qlimb = qlimb;
    a.qaux = qaux;
    a.n_groups = rs.n_groups;
    a.tpg = rs.tpg;
    a.g_real = rs.g_real;
    a.max_tok = rs.max_tok;
    a.n_tok = n_tok;
    if (step != nullptr) {
        a.n_new = step->n_new;
        a.k_new = step->k_new;
        a.v_new = step->v_new;
        a.t_k = step->t_k;
        a.win_kw = c->win_k;
        a.win_vw = c->win_v;
    }

    const unsigned rows_z = (unsigned)(c->batch * rs.n_groups);
    // several token groups (a chunk of more tokens than one group holds):
    // the four waves of a workgroup take four of them over the same items
    const unsigned grid_z = rs.share ? (unsigned)(c->batch * ((rs.n_groups + 3) / 4)) : rows_z;
    const dim3 gm(c->n_kv_heads, p.n_splits, grid_z);
    const dim3 gc(c->n_kv_heads * G, rows_z);
    // Each workgroup forms q~ itself when the whole grid is resident at
    // once (one round: the rows cost each workgroup an L2 read of T^{-1}
    // that overlaps its first pages).  A grid that runs in rounds would pay
    // that read once per workgroup, so a small kernel forms q~ first; so do
    // grids of shared work items.
    const int64_t wgs = (int64_t)p.n_splits * c->n_kv_heads * grid_z;
    const bool form = !rs.share && p.win_units == 1 &&
                      wgs * 4 <= resident_waves(c->head_dim, storage_bits(c->bits), G, false);
    const int key = c->head_dim * 10 + storage_bits(c->bits);
    if (rs.share && c->head_dim == 128 && G == 8) {
        // chunks: q~ rows (chunk_qt_kernel), the pages (chunk_pages_kernel, splits 0 ..
        // n_page_splits - 1), then the window slots merged with the page
        // runs into the output (chunk_window_kernel)
        const unsigned blocks = (unsigned)(c->batch * ((rs.n_groups + 7) / 8));
        const dim3 gp(c->n_kv_heads, p.n_page_splits, blocks);
        const dim3 gw(c->n_kv_heads, 4 * blocks);
        const dim3 gq(c->n_kv_heads, (unsigned)(c->batch * ((rs.n_groups + 1) / 2)));
        if (key == 1282) {
            launch("chunk_qt_kernel", chunk_qt_kernel<2>, gq, dim3(256), s, a);
            if (p.n_page_splits > 0) launch("chunk_pages_kernel", chunk_pages_kernel<2>, gp, dim3(256), s, a);
        } else {
            launch("chunk_qt_kernel", chunk_qt_kernel<4>, gq, dim3(256), s, a);
            if (p.n_page_splits > 0) launch("chunk_pages_kernel", chunk_pages_kernel<4>, gp, dim3(256), s, a);
        }
        launch("chunk_window_kernel", chunk_window_kernel, gw, dim3(256), s, a, out);
        if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
        return WUSHKV_OK;
    } else switch (key) {
        case 1282: launch_main_g<128, 2>(G, form, rs.share, gm, rows_z, s, a); break;
        case 1284: launch_main_g<128, 4>(G, form, rs.share, gm, rows_z, s, a); break;
        case 642: launch_main_g<64, 2>(G, form, rs.share, gm, rows_z, s, a); break;
        case 644: launch_main_g<64, 4>(G, form, rs.share, gm, rows_z, s, a); break;
    }
    if (step != nullptr) {
        if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
        return wushkv_step_finish(c, step->n_new, part, out, G, p.n_splits, s);
    }
    if (c->head_dim == 128) launch("decode_combine_kernel", decode_combine_kernel<128>, gc, dim3(128), s, (const float *)part, out, c->n_kv_heads, G, p.n_splits, a);
    else launch("decode_combine_kernel", decode_combine_kernel<64>, gc, dim3(64), s, (const float *)part, out, c->n_kv_heads, G, p.n_splits, a);
    if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
    return WUSHKV_OK;
}

extern "C" size_t wushkv_decode_workspace_bytes(const wushkv_cache *c, int32_t n_q_heads,
                                                int32_t max_seq_len)
{
    return workspace_bytes(c, n_q_heads, 1, max_seq_len);
}

extern "C" int wushkv_decode_attention(const wushkv_cache *c, const uint16_t *q, int32_t n_q_heads,
                                       int32_t max_seq_len, const float *t_k_inv, float sm_scale,
                                       float *out, void *workspace, size_t workspace_bytes,
                                       wushkv_stream_t stream)
{
    return attend(c, q, nullptr, 1, n_q_heads, max_seq_len, t_k_inv, sm_scale, out, workspace,
                  workspace_bytes, stream);
}

// ------------------------------------------------------- no-allocation call

// The workspace of wushkv_decode_attention_noalloc: a file-scope device
// array, one copy per GPU the library runs on, held until the process ends.
// Host code never uses its name as an address (on the host it stands for a
// host-side shadow); it takes the device address from hipGetSymbolAddress,
// once per device, with that device current.
static __device__ __align__(256) uint8_t scratch[WUSHKV_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of the current device's copy of scratch (looked up on the
// first call on that device), or null when there is no usable device.
static void *scratch_on_current_device()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        (void)hipGetLastError();
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

extern "C" int wushkv_decode_attention_noalloc(const wushkv_cache *c, const uint16_t *q,
                                               int32_t n_q_heads, int32_t max_seq_len,
                                               const float *t_k_inv, float sm_scale, float *out,
                                               wushkv_stream_t stream)
{
    // the plan's size first: a call that needs more than the array holds is
    // refused before anything else happens
    const size_t need = workspace_bytes(c, n_q_heads, 1, max_seq_len);
    if (need == 0) {
        const int st = check_decode_args(c, n_q_heads, max_seq_len);
        return st != WUSHKV_OK ? st : WUSHKV_EUNSUPPORTED;
    }
    if (need > (size_t)WUSHKV_NOALLOC_SCRATCH_BYTES) return WUSHKV_EWORKSPACE;
    void *ws = scratch_on_current_device();
    if (ws == nullptr) return WUSHKV_ENODEVICE;
    return attend(c, q, nullptr, 1, n_q_heads, max_seq_len, t_k_inv, sm_scale, out, ws,
                  (size_t)WUSHKV_NOALLOC_SCRATCH_BYTES, stream);
}

extern "C" size_t wushkv_chunk_workspace_bytes(const wushkv_cache *c, int32_t n_q_heads,
                                               int32_t max_tok, int32_t max_seq_len)
{
    if (wushkv_validate_cache(c) != WUSHKV_OK || check_chunk(c, max_tok) != WUSHKV_OK) return 0;
    return workspace_bytes(c, n_q_heads, max_tok, max_seq_len);
}

extern "C" int wushkv_chunk_attention(const wushkv_cache *c, const uint16_t *q,
                                      const int32_t *n_tok, int32_t max_tok, int32_t n_q_heads,
                                      int32_t max_seq_len, const float *t_k_inv, float sm_scale,
                                      float *out, void *workspace, size_t workspace_bytes,
                                      wushkv_stream_t stream)
{
    int st = wushkv_validate_cache(c);
    if (st != WUSHKV_OK) return st;
    st = check_chunk(c, max_tok);
    if (st != WUSHKV_OK) return st;
    return attend(c, q, n_tok, max_tok, n_q_heads, max_seq_len, t_k_inv, sm_scale, out, workspace,
                  workspace_bytes, stream);
}

extern "C" int wushkv_decode_step(const wushkv_cache *c, const uint16_t *k_new, const uint16_t *v_new,
                                  const int32_t *n_new, const uint16_t *t_k, const uint16_t *q,
                                  int32_t n_q_heads, int32_t max_seq_len, const float *t_k_inv,
                                  float sm_scale, float *out, void *workspace,
                                  size_t workspace_bytes, wushkv_stream_t stream)
{
    int st = wushkv_validate_cache(c);
    if (st != WUSHKV_OK) return st;
    if (!k_new || !v_new || !n_new || !t_k) return WUSHKV_EINVAL;
    if (((uintptr_t)t_k & 15u) || ((uintptr_t)k_new | (uintptr_t)v_new) & 1u || ((uintptr_t)n_new & 3u))
        return WUSHKV_EINVAL;
    // the new token's ring slot must be free: the ring holds at most
    // s_keep + s_flush - 1 live entries before the step
    if ((int64_t)c->win_slots - c->s_sink < (int64_t)c->s_keep + c->s_flush) return WUSHKV_EUNSUPPORTED;
    const StepIn in{n_new, k_new, v_new, t_k};
    return attend(c, q, nullptr, 1, n_q_heads, max_seq_len, t_k_inv, sm_scale, out, workspace,
                  workspace_bytes, stream, &in);
}
