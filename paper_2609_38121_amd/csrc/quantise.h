// The quantiser shared by the append kernels and the fused decode step:
// kernel arguments of the append path, the per-token clip-range selection
// and parameters of Eq. (7) (and the QuEST projection of Eq. (5)), the
// tile quantiser writing codes and parameters into a page, and the flush of
// a range of positions from the recent ring (Alg. 2 steps 7-11).
#pragma once
#include <type_traits>

#include "common.h"

namespace wushkv {

enum { kModeFlush = 1, kModeNew = 2 };

struct AppendArgs {
    uint8_t *pages;
    const int32_t *page_table;
    uint16_t *win_k;
    uint16_t *win_v;
    int32_t *seq_len;
    int32_t *quant_end;
    int32_t *commit;     // [batch] arrivals of this launch's workgroups (zero between calls)
    int32_t arrivals;    // workgroups per sequence that report; 0: this launch does not commit
    int32_t n_kv, s_sink, s_keep, s_flush, win_slots, max_pages, n_pages;
    int32_t lo_k, lo_v;  // quantile positions: lo = floor(kappa (d-1))
    float t_k, t_v;      // and t = kappa (d-1) - lo
    int32_t codec;       // WUSHKV_CODEC_PCLIP (Eq. (7)) or WUSHKV_CODEC_QUEST (Eq. (5))
    int32_t levels;      // 2^b - 1 for b-bit codes (b = 3 codes sit in 4-bit fields)
    double quest_coef;   // QuEST: 2 alpha_b / (2^bits - 1)
    const uint16_t *k_new;
    const uint16_t *v_new;
    const int32_t *n_new;
    int32_t max_new;
    const uint16_t *tk;
    uint16_t *k_tilde_out;
    int32_t mode;
    int32_t sink_tiles;  // ceil(s_sink / 64)
    // headwise RMS normalisation + rotary embedding of the new keys (Alg. 2
    // step 1), applied when rope is not null
    const float *gain;   // [D] or null (one)
    float eps;
    const float *rope;   // [positions][D]: cos(s w_j) | sin(s w_j)
};

// RoPE(Norm(x)) of one key row held by four lanes (the lanes n + 16 j,
// j = 0..3 of a 16-lane column group): lane j holds channels 32 c + 8 j + e
// (c = 0..3, e = 0..7) in x[c][e].  The rotary partner of channel i < D/2
// is i + D/2, chunk c + D/64 of the same lane, so the rotation is local.
// Each step is a separately rounded fp32 operation.  The rotary table's
// entries for this lane (cos in rt[c][0..7], sin in rt[c][8..15] for the
// chunks c < D/64 of position pos) come from load_rope, so that their load
// can be issued with the row's own.
template <int D>
__device__ __forceinline__ void load_rope(const AppendArgs &a, int j, int32_t pos, float (&rt)[D / 64][16])
{
    const float *row = a.rope + (int64_t)pos * D;
#pragma unroll
    for (int c = 0; c < D / 64; ++c) {
        const float *cs = row + 32 * c + 8 * j;
        const float4 c0 = *reinterpret_cast<const float4 *>(cs);
        const float4 c1 = *reinterpret_cast<const float4 *>(cs + 4);
        const float4 s0 = *reinterpret_cast<const float4 *>(cs + D / 2);
        const float4 s1 = *reinterpret_cast<const float4 *>(cs + D / 2 + 4);
        const float v[16] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w,
                             s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
        for (int e = 0; e < 16; ++e) rt[c][e] = v[e];
    }
}

template <int D>
__device__ __forceinline__ void norm_rope_row(float (&x)[D / 32][8], int j, const float (&rt)[D / 64][16],
                                              const AppendArgs &a)
{
    constexpr int kC = D / 32;
    float ss = 0.0f;
#pragma unroll
    for (int c = 0; c < kC; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) ss = fmaf(x[c][e], x[c][e], ss);
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    const float r = 1.0f / sqrtf(ss / (float)D + a.eps);
    // (x r) g, or x r with no gain (a product by 1 is exact)
#pragma unroll
    for (int c = 0; c < kC; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[c][e] = x[c][e] * r;
    if (a.gain != nullptr) {
#pragma unroll
        for (int c = 0; c < kC; ++c) {
            const float4 g0 = *reinterpret_cast<const float4 *>(a.gain + 32 * c + 8 * j);
            const float4 g1 = *reinterpret_cast<const float4 *>(a.gain + 32 * c + 8 * j + 4);
            const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) x[c][e] = x[c][e] * g[e];
        }
    }
#pragma unroll
    for (int c = 0; c < kC / 2; ++c) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float lo = x[c][e], hi = x[c + kC / 2][e];
            x[c][e] = lo * rt[c][e] - hi * rt[c][8 + e];
            x[c + kC / 2][e] = hi * rt[c][e] + lo * rt[c][8 + e];
        }
    }
}

template <int D>
__device__ __forceinline__ void norm_rope_row(float (&x)[D / 32][8], int j, int32_t pos, const AppendArgs &a)
{
    float rt[D / 64][16];
    load_rope<D>(a, j, pos, rt);
    norm_rope_row<D>(x, j, rt, a);
}

// Sequence b's counters as they stand before this launch: thread 0 reads
// S, S_quant and the new-token count and hands them to the whole workgroup
// through LDS (sh: three int32 of the caller's), so that every wave works
// with the very values thread 0's arrival is tied to (commit_arrive).  The
// count is clamped to [0, max_nn].  Every thread of the workgroup calls it;
// it contains a barrier.
struct SeqCounters {
    int32_t s_old, q_old, nn;
};
__device__ __forceinline__ SeqCounters read_counters(const AppendArgs &a, int b, int32_t max_nn,
                                                     int32_t *sh, int tid)
{
    if (tid == 0) {
        sh[0] = a.seq_len[b];
        sh[1] = a.quant_end[b];
        sh[2] = a.n_new[b];
    }
    __syncthreads();
    SeqCounters c{sh[0], sh[1], sh[2]};
    c.nn = c.nn < 0 ? 0 : (c.nn > max_nn ? max_nn : c.nn);
    return c;
}

// Sequence b's counters advance from inside the launch that last reads
// them.  Each workgroup reports once, after its reads of seq_len and
// quant_end have returned (the values are tied to the report's operand), to
// the sequence's arrival count (commit_arrive, early in the workgroup's
// work); the workgroup that was last of a.arrivals writes S_new and
// S_quant_new and clears the count for the next call (commit_finish, at its
// end, so that the count's round trip overlaps its work).  Every workgroup
// of the sequence has read the old values before the last one arrives, so
// none can see the new ones: the other waves of a workgroup use thread 0's
// reads (read_counters).  Thread 0 only; a launch with a.arrivals = 0 leaves
// the counters alone (a launch of many workgroups per sequence does, and
// append_commit_kernel advances them after it).
__device__ __forceinline__ int32_t commit_arrive(const AppendArgs &a, int b, int32_t s_old, int32_t q_old,
                                                 int32_t nn, int tid)
{
    if (a.arrivals <= 0 || tid != 0) return -1;
    int32_t one = 1;
    asm volatile("" : "+v"(one) : "v"(s_old), "v"(q_old), "v"(nn));
    return __hip_atomic_fetch_add(a.commit + b, one, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void commit_finish(const AppendArgs &a, int b, int32_t arrived, int32_t s_new,
                                              int32_t q_new, int tid)
{
    if (a.arrivals <= 0 || tid != 0 || arrived != a.arrivals - 1) return;
    a.seq_len[b] = s_new;
    a.quant_end[b] = q_new;
    __hip_atomic_store(a.commit + b, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// max and min of two values as medians of three against an infinity held in
// a register (inf: +inf for the max, -inf for the min): one instruction
// each, where fmaxf / fminf first quiet an operand that might be a
// signalling NaN, a second instruction per call.  Equal to fmaxf / fminf for
// every non-NaN operand.  The infinity comes from opaque_inf: a literal one
// would be folded back into fmaxf / fminf.
__device__ __forceinline__ float opaque_inf(bool negative)
{
    float v = negative ? -INFINITY : INFINITY;
    asm volatile("" : "+v"(v));
    return v;
}
__device__ __forceinline__ float max_m3(float x, float y, float pinf) { return __builtin_amdgcn_fmed3f(x, y, pinf); }
__device__ __forceinline__ float min_m3(float x, float y, float ninf) { return __builtin_amdgcn_fmed3f(x, y, ninf); }

// Descending top-KMAX of the values pushed so far; t[0] is the largest.
// Inserting a into a sorted list is one median-of-three per slot:
// new t[i] = med3(t[i-1], t[i], a), and new t[0] = max(t[0], a).
template <int KMAX>
struct TopK {
    float t[KMAX];
    float pinf;
    __device__ __forceinline__ void init()
    {
#pragma unroll
        for (int i = 0; i < KMAX; ++i) t[i] = -1.0f;
        pinf = opaque_inf(false);
    }
    __device__ __forceinline__ void push(float a)
    {
#pragma unroll
        for (int i = KMAX - 1; i >= 1; --i) t[i] = __builtin_amdgcn_fmed3f(t[i - 1], t[i], a);
        t[0] = max_m3(t[0], a, pinf);
    }
    // t[k] for a runtime k, as a chain of selects.  The empty assembly step
    // keeps the chain in registers: without it the compiler turns the chain
    // into an indexed load from a private (scratch) copy of the list.
    __device__ __forceinline__ float get(int k) const
    {
        float r = t[0];
#pragma unroll
        for (int i = 1; i < KMAX; ++i) {
            r = (k == i) ? t[i] : r;
            asm volatile("" : "+v"(r));
        }
        return r;
    }
};

// The value of the partner lane (lane ^ 1): the two lanes of a pair share
// one quantisation group, half of its elements each.
__device__ __forceinline__ float pair_swap(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0xB1, 0xF,
                                                              0xF, false));
}

// a_lo and a_{lo+1} of the ascending sort of |x| over a bf16 row in LDS,
// for lo = D - K (a_lo is the K-th largest), with the row's min and max.
// The lane pair (2 r, 2 r + 1) shares row r: each lane keeps the sorted top
// K of |x| over its half of the row.  The top K of the whole row are then
// max(t[i], t'[K-1-i]), i < K, with t' the partner's list (a descending list
// against an ascending one: each pair's larger value is in the top K of the
// union, and each smaller one is not); a_lo and a_{lo+1} are the smallest and
// the second smallest of these.  Both lanes form the same multiset.
template <int D, int K>
__device__ __forceinline__ void order_stats_topk(const uint16_t *row, int hf, float &a_lo, float &a_hi,
                                                 float &mn, float &mx)
{
    TopK<K> tk;
    tk.init();
    mn = INFINITY;
    mx = -INFINITY;
    const uint16_t *half = row + hf * (D / 2);
#pragma unroll 4
    for (int c8 = 0; c8 < D / 16; ++c8) {
        uint4 v = *reinterpret_cast<const uint4 *>(half + 8 * c8);
        uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                float x = bf16_bits_to_f32(hh ? (w[q] >> 16) : (w[q] & 0xFFFFu));
                mn = fminf(mn, x);
                mx = fmaxf(mx, x);
                tk.push(fabsf(x));
            }
        }
    }
    const float ninf = opaque_inf(true);
    float c[K];
#pragma unroll
    for (int i = 0; i < K; ++i) c[i] = max_m3(tk.t[i], pair_swap(tk.t[K - 1 - i]), tk.pinf);
    if constexpr (K == 1) {
        a_lo = a_hi = c[0];
    } else {
        float m1 = min_m3(c[0], c[1], ninf), m2 = max_m3(c[0], c[1], tk.pinf);
#pragma unroll
        for (int i = 2; i < K; ++i) {
            m2 = __builtin_amdgcn_fmed3f(m1, m2, c[i]);  // m1 <= m2: the new second smallest
            m1 = min_m3(m1, c[i], ninf);
        }
        a_lo = m1;
        a_hi = m2;
    }
    mn = fminf(mn, pair_swap(mn));
    mx = fmaxf(mx, pair_swap(mx));
}

// Same order statistics by counting ranks: any lo, O(D^2) work.  Used when
// kappa is small enough that the top-k list would not fit in registers.
// Each lane of the pair ranks the elements of its half against the whole
// row; an order statistic is found in the half (or halves, for equal values)
// that holds it.
template <int D>
__device__ __forceinline__ void order_stats_rank(const uint16_t *row, int hf, int lo, float &a_lo,
                                              float &a_hi, float &mn, float &mx)
{
    mn = INFINITY;
    mx = -INFINITY;
    a_lo = -1.0f;
    a_hi = -1.0f;
    for (int e = hf * (D / 2); e < (hf + 1) * (D / 2); ++e) {
        float xe = bf16_bits_to_f32(row[e]);
        mn = fminf(mn, xe);
        mx = fmaxf(mx, xe);
        float ae = fabsf(xe);
        int less = 0, le = 0;
        for (int f = 0; f < D; ++f) {
            float af = fabsf(bf16_bits_to_f32(row[f]));
            less += (af < ae);
            le += (af <= ae);
        }
        // |x_e| occupies ascending ranks [less, le)
        if (less <= lo && lo < le) a_lo = ae;
        if (less <= lo + 1 && lo + 1 < le) a_hi = ae;
    }
    a_lo = fmaxf(a_lo, pair_swap(a_lo));
    a_hi = fmaxf(a_hi, pair_swap(a_hi));
    mn = fminf(mn, pair_swap(mn));
    mx = fmaxf(mx, pair_swap(mx));
    if (lo + 1 >= D) a_hi = a_lo;
}

// Eq. (7) parameters from the order statistics.  Every operation is a single
// correctly rounded fp32 operation (the file is built without contraction).
__device__ __forceinline__ void quant_params(float a_lo, float a_hi, float t, bool interp,
                                             float mn, float mx, int levels, uint32_t &s16,
                                             uint32_t &z16, float &z, float &inv)
{
    float q = a_lo;
    if (interp) {
        float diff = a_hi - a_lo;
        float prod = t * diff;
        q = a_lo + prod;
    }
    float x_min = (mn > -q) ? mn : -q;
    float x_max = (mx < q) ? mx : q;
    float delta = (x_max - x_min) / (float)levels;
    s16 = f32_to_f16_bits(delta);
    z16 = f32_to_f16_bits(x_min);
    float s = f16_bits_to_f32(s16);
    z = f16_bits_to_f32(z16);
    inv = (s > 0.0f) ? 1.0f / s : 0.0f;
}

// clamp(rne((x - z) inv), 0, levels).  Clamping to [0, levels] before the
// rounding gives the same integer (levels is an integer), and adding 2^23 to
// a value in [0, 2^23) rounds it to an integer in the default
// nearest-even mode, leaving that integer in the low bits of the sum.
__device__ __forceinline__ uint32_t code_of(float x, float z, float inv, float levels)
{
    const float y = (x - z) * inv;
    const float c = __builtin_amdgcn_fmed3f(y, 0.0f, levels);
    return __float_as_uint(c + 8388608.0f) - 0x4B000000u;
}

// Eq. (5) (QuEST) parameters of a group held by a lane pair (this lane's
// half of the channels from hf): the step is 2 alpha_b / (2^bits - 1) times
// the group's RMS, with the sum of squares in fp64 (each square exact, the
// two halves added last; the order does not change the result beyond fp64
// rounding) and the step rounded once to fp32 and then to the fp16 scale.
// The zero is the offset of the lowest bin centre, scale (1/2 - 2^(bits-1)),
// exact in fp32 and rounded to fp16.
// Eq. (5) parameters from the group's sum of squares ss (fp64).
// half = 2^(b-1) for b-bit codes.
template <int D>
__device__ __forceinline__ void quest_finish(double ss, double coef, float half, uint32_t &s16,
                                             uint32_t &z16, float &z, float &inv)
{
    const float step = (float)(coef * sqrt(ss / (double)D));
    s16 = f32_to_f16_bits(step);
    const float s = f16_bits_to_f32(s16);
    z16 = f32_to_f16_bits(s * (0.5f - half));
    z = f16_bits_to_f32(z16);
    inv = (s > 0.0f) ? 1.0f / s : 0.0f;
}

template <int D>
__device__ __forceinline__ void quest_params(const uint16_t *row, int hf, double coef, float h_levels,
                                             uint32_t &s16, uint32_t &z16, float &z, float &inv)
{
    const uint16_t *half = row + hf * (D / 2);
    double ss = 0.0;
#pragma unroll 4
    for (int c8 = 0; c8 < D / 16; ++c8) {
        uint4 v = *reinterpret_cast<const uint4 *>(half + 8 * c8);
        uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const double lo = (double)bf16_bits_to_f32(w[q] & 0xFFFFu);
            const double hi = (double)bf16_bits_to_f32(w[q] >> 16);
            ss = fma(lo, lo, ss);
            ss = fma(hi, hi, ss);
        }
    }
    const uint64_t u = __builtin_bit_cast(uint64_t, ss);
    const uint32_t plo = __builtin_bit_cast(uint32_t, pair_swap(__builtin_bit_cast(float, (uint32_t)u)));
    const uint32_t phi = __builtin_bit_cast(uint32_t, pair_swap(__builtin_bit_cast(float, (uint32_t)(u >> 32))));
    ss += __builtin_bit_cast(double, ((uint64_t)phi << 32) | plo);
    quest_finish<D>(ss, coef, h_levels, s16, z16, z, inv);
}

// clamp(floor(x inv) + 2^(bits-1), 0, levels) of Eq. (5), as code_of.
__device__ __forceinline__ uint32_t quest_code_of(float x, float inv, float h, float levels)
{
    const float c = __builtin_amdgcn_fmed3f(floorf(x * inv) + h, 0.0f, levels);
    return __float_as_uint(c + 8388608.0f) - 0x4B000000u;
}

// The selection for K = D - lo: the top-K lists for K = KC .. 16 (each its
// own exact length), the rank count beyond.
template <int D, int KC = 1>
__device__ __forceinline__ void order_stats(const uint16_t *row, int hf, int lo, float &a_lo, float &a_hi,
                                            float &mn, float &mx)
{
    if (D - lo == KC) order_stats_topk<D, KC>(row, hf, a_lo, a_hi, mn, mx);
    else if constexpr (KC < 16) order_stats<D, KC + 1>(row, hf, lo, a_lo, a_hi, mn, mx);
    else order_stats_rank<D>(row, hf, lo, a_lo, a_hi, mn, mx);
}

// Value codes (one byte each) are written over the value row they come
// from: the lane holding channels [h D / 2, (h + 1) D / 2) of row t writes
// their codes at bytes h D .. h D + D / 2 - 1 of that row, inside the bytes
// it has already read.
template <int D>
__device__ __forceinline__ uint8_t *vcode_row(uint16_t *vt, int t)
{
    return reinterpret_cast<uint8_t *>(vt + t * (D + 8));
}

// Phase C of a tile: the value-code words, from the code bytes that phase
// B left in the value rows (vcode_row).  full: every position of the tile is
// quantised now, so whole words are written without checks; otherwise only
// the codes of positions with quant(p) are merged into what the page holds.
template <int D, int BITS, typename Pred>
__device__ void value_words(uint16_t *vt, int32_t blk_lo, Pred quant, bool full, uint8_t *pg, int tid)
{
    using L = Layout<D, BITS>;
    constexpr int kPitch = D + 8;
    if (full) {
        uint32_t *vreg = reinterpret_cast<uint32_t *>(pg + L::kRegionBytes);
        constexpr int kWords = 64 * L::kWordsPerLane;
        constexpr int kRowBytes = 2 * kPitch;
        for (int idx = tid; idx < kWords; idx += 256) {
            const int Ln = idx / L::kWordsPerLane, rem = idx % L::kWordsPerLane;
            const int kc = rem / (2 * L::kNw), u = rem % (2 * L::kNw);
            const int j = Ln >> 4, m = Ln & 15;
            const uint8_t *base = vcode_row<D>(vt, 32 * kc + 8 * j);  // token i at + i kRowBytes
            uint32_t bits = 0;
#pragma unroll
            for (int e = 0; e < L::kCodesPerWord; ++e) {
                const int o = e >> 3, i = e & 7;
                const int ch = 16 * (u * L::kOpsPerWord + o) + m;
                bits |= (uint32_t)base[i * kRowBytes + ch + (ch >= D / 2 ? D / 2 : 0)] << L::v_bit(o, i);
            }
            vreg[L::v_word(Ln, rem)] = bits;
        }
    } else if (pg != nullptr) {
        uint32_t *vreg = reinterpret_cast<uint32_t *>(pg + L::kRegionBytes);
        constexpr int kWords = 64 * L::kWordsPerLane;
        for (int idx = tid; idx < kWords; idx += 256) {
            const int Ln = idx / L::kWordsPerLane, rem = idx % L::kWordsPerLane;
            const int kc = rem / (2 * L::kNw), u = rem % (2 * L::kNw);
            const int widx = L::v_word(Ln, rem);
            const int j = Ln >> 4, m = Ln & 15;
            uint32_t mask = 0, bits = 0;
#pragma unroll
            for (int e = 0; e < L::kCodesPerWord; ++e) {
                const int o = e >> 3, i = e & 7;
                const int t = 32 * kc + 8 * j + i;
                const int32_t p = blk_lo + t;
                if (quant(p)) {
                    const int ch = 16 * (u * L::kOpsPerWord + o) + m;
                    const int bit = L::v_bit(o, i);
                    mask |= ((1u << BITS) - 1u) << bit;
                    bits |= (uint32_t)vcode_row<D>(vt, t)[ch + (ch >= D / 2 ? D / 2 : 0)] << bit;
                }
            }
            if (mask == 0u) continue;
            if (mask != 0xFFFFFFFFu) bits |= vreg[widx] & ~mask;
            vreg[widx] = bits;
        }
    }
}

// Phases B and C of a tile of up to 64 positions starting at blk_lo, all in
// one page (pg, or null when the page is outside the pool): quantise every
// position p with quant(p) from its bf16 rows in kt / vt (row p - blk_lo),
// write its parameters and key words, then assemble the value words, merging
// words only partly covered with what the page holds.  all_quant: the
// caller's statement that quant(p) holds for every p of [blk_lo, blk_lo +
// 64) (the common case of a prefill); the value words are then assembled
// without per-code checks or merges.  Every thread of the workgroup must
// call it (it synchronises).
template <int D, int BITS, typename Pred>
__device__ void quantise_tile(const AppendArgs &a, const uint16_t *kt, uint16_t *vt,
                              int32_t blk_lo, Pred quant, bool all_quant, uint8_t *pg, int tid)
{
    using L = Layout<D, BITS>;
    constexpr int kPitch = D + 8;
    const bool full = all_quant && pg != nullptr;
    // ---- phase B: quantise.  Lanes 2 r and 2 r + 1 share group r (rows
    // 0-63 keys, 64-127 values), one half of its channels each, so that all
    // four waves take part.
    {
        const int grp = tid >> 1, hf = tid & 1;
        const bool is_v = grp >= kPage;
        const int r = grp & (kPage - 1);
        const int32_t p = blk_lo + r;
        if (quant(p) && pg != nullptr) {  // the same for both lanes of the pair
            const uint16_t *row = (is_v ? vt : kt) + r * kPitch;
            uint32_t s16, z16;
            float z, inv;
            const int kLevels = a.levels;             // 2^b - 1 (b = 3 in 4-bit fields)
            const float kMid = (float)((kLevels + 1) / 2);  // 2^(b-1)
            const bool quest = a.codec == WUSHKV_CODEC_QUEST;
            if (quest) {
                quest_params<D>(row, hf, a.quest_coef, kMid, s16, z16, z, inv);
            } else {
                const int qlo = is_v ? a.lo_v : a.lo_k;
                const float qt = is_v ? a.t_v : a.t_k;
                float a_lo, a_hi, mn, mx;
                order_stats<D>(row, hf, qlo, a_lo, a_hi, mn, mx);
                quant_params(a_lo, a_hi, qt, qlo + 1 < D, mn, mx, kLevels, s16, z16, z, inv);
            }
            if (hf == 0)
                *reinterpret_cast<uint32_t *>(pg + L::kParamOffset + 4 * r + (is_v ? 4 * kPage : 0)) =
                    s16 | (z16 << 16);
            constexpr int kHalf = D / 2;
            const int c0 = hf * kHalf;  // first channel of this lane's half
            // the code loops, instantiated once per codec's code formula
            auto write_codes = [&](auto code_fn) {
                if (!is_v) {
                    // key words of this token: lane group jj = ch / 32 holds
                    // BITS words per token (see Layout::k_pos); this half covers
                    // groups hf D / 64 .. (hf + 1) D / 64 - 1
                    uint32_t kw[D / 64][BITS];
#pragma unroll
                    for (int jl = 0; jl < D / 64; ++jl)
#pragma unroll
                        for (int w = 0; w < BITS; ++w) kw[jl][w] = 0u;
#pragma unroll
                    for (int c8 = 0; c8 < kHalf / 8; ++c8) {
                        uint4 v = *reinterpret_cast<const uint4 *>(row + c0 + 8 * c8);
                        uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            uint32_t hb = (i & 1) ? (wv[i >> 1] >> 16) : (wv[i >> 1] & 0xFFFFu);
                            uint32_t code = code_fn(bf16_bits_to_f32(hb));
                            const int cl = 8 * c8 + i;  // channel c0 + cl
                            int word, bit;
                            L::k_pos(r, c0 + cl, word, bit);
                            kw[cl >> 5][(cl & 31) / (32 / BITS)] |= code << bit;
                        }
                    }
                    uint32_t *kreg = reinterpret_cast<uint32_t *>(pg);
#pragma unroll
                    for (int jl = 0; jl < D / 64; ++jl)
#pragma unroll
                        for (int w = 0; w < BITS; ++w)
                            kreg[L::k_word(16 * (hf * (D / 64) + jl) + (r >> 2), BITS * (r & 3) + w)] = kw[jl][w];
                } else {
#pragma unroll
                    for (int c8 = 0; c8 < kHalf / 8; ++c8) {
                        uint4 v = *reinterpret_cast<const uint4 *>(row + c0 + 8 * c8);
                        uint32_t wv[4] = {v.x, v.y, v.z, v.w};
                        uint32_t lo4 = 0, hi4 = 0;
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            uint32_t hb = (i & 1) ? (wv[i >> 1] >> 16) : (wv[i >> 1] & 0xFFFFu);
                            uint32_t code = code_fn(bf16_bits_to_f32(hb));
                            if (i < 4) lo4 |= code << (8 * i);
                            else hi4 |= code << (8 * (i - 4));
                        }
                        // over bytes of this lane's half of the row that it has read
                        *reinterpret_cast<uint2 *>(vcode_row<D>(vt, r) + hf * D + 8 * c8) = make_uint2(lo4, hi4);
                    }
                }
            };
            const float kLv = (float)kLevels;
            if (quest) {
                // Eq. (5): clamp(floor(x inv) + 2^(bits-1))
                write_codes([&](float x) { return quest_code_of(x, inv, kMid, kLv); });
            } else {
                // Eq. (7): clamp(rne((x - z) inv))
                write_codes([&](float x) { return code_of(x, z, inv, kLv); });
            }
        }
    }
    __syncthreads();

    value_words<D, BITS>(vt, blk_lo, quant, full, pg, tid);
}

// ------------------------------------------------ few positions, wide groups

// Lane exchanges inside each row of 16 lanes (DPP): partner lane ^ 1, ^ 2
// (quad permutations), 7 - lane within 8 and 15 - lane within 16 (the half
// mirror and the mirror).  Applied in that order they combine all 16 lanes,
// as a butterfly does.
template <int kCtrl>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, kCtrl, 0xF, 0xF, false);
}
template <int kStep>
__device__ __forceinline__ uint32_t row16_swap(uint32_t x)
{
    constexpr int kCtrl = kStep == 0 ? 0xB1 : kStep == 1 ? 0x4E : kStep == 2 ? 0x141 : 0x140;
    return dpp_u32<kCtrl>(x);
}
template <int kStep>
__device__ __forceinline__ float row16_swap(float x)
{
    return __builtin_bit_cast(float, row16_swap<kStep>(__builtin_bit_cast(uint32_t, x)));
}

// The exact top-KMAX of |x|, min and max over a group held by 16 lanes,
// kPer elements each: every lane keeps the top KMAX of its elements, then
// inserts its partner's list at each of the four exchange steps, so that
// every lane ends with the top KMAX of the whole group (the same multiset as
// the lane-pair selection finds, hence the same order statistics).
template <int KMAX, int kPer>
__device__ __forceinline__ void few_order_stats(const float (&x)[kPer], int K, float &a_lo, float &a_hi,
                                                float &mn, float &mx)
{
    TopK<KMAX> tk;
    tk.init();
    mn = INFINITY;
    mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        mn = fminf(mn, x[e]);
        mx = fmaxf(mx, x[e]);
        tk.push(fabsf(x[e]));
    }
    auto step = [&](auto st) {
        constexpr int kStep = decltype(st)::value;
        float other[KMAX];
#pragma unroll
        for (int i = 0; i < KMAX; ++i) other[i] = row16_swap<kStep>(tk.t[i]);
#pragma unroll
        for (int i = 0; i < KMAX; ++i) tk.push(other[i]);
        mn = fminf(mn, row16_swap<kStep>(mn));
        mx = fmaxf(mx, row16_swap<kStep>(mx));
    };
    step(std::integral_constant<int, 0>{});
    step(std::integral_constant<int, 1>{});
    step(std::integral_constant<int, 2>{});
    step(std::integral_constant<int, 3>{});
    a_lo = tk.get(K - 1);
    a_hi = (K >= 2) ? tk.get(K - 2) : a_lo;
}

// Phases B and C for at most 8 positions [lo, hi) of the tile at blk_lo (one
// page, pg, or null outside the pool), with 16 lanes per quantisation group:
// group g = tid / 16 is the key row (g < 8) or the value row (g >= 8) of
// position lo + g % 8, lane s = tid % 16 holds its channels kPer s ..
// kPer s + kPer - 1.  The parameters, codes and words are those
// quantise_tile writes (the selection keeps the same multiset; the QuEST sum
// of squares is exact in fp64 for bf16 inputs of the usual range, so its
// order does not matter).  Needs D - lo_k and D - lo_v <= 16 for Eq. (7).
// Every thread of the workgroup calls it.
template <int D, int BITS>
__device__ void quantise_few(const AppendArgs &a, uint16_t *kt, uint16_t *vt, int32_t blk_lo,
                             int32_t lo, int32_t hi, uint8_t *pg, int tid)
{
    using L = Layout<D, BITS>;
    constexpr int kPitch = D + 8;
    constexpr int kPer = D / 16;                 // channels per lane: 8 or 4
    const int kLevels = a.levels;                // 2^b - 1 (b = 3 in 4-bit fields)
    const float kHalf = (float)((kLevels + 1) / 2);  // 2^(b-1)
    constexpr int kPerWord = 32 / BITS;          // key codes per word
    constexpr int kLanesPerWord = kPerWord / kPer;  // 1, 2 or 4
    const int g = tid >> 4, sl = tid & 15;
    const bool is_v = g >= 8;
    const int r = (lo - blk_lo) + (g & 7);
    if ((g & 7) < hi - lo && pg != nullptr) {  // uniform over the group's 16 lanes
        uint16_t *row = (is_v ? vt : kt) + r * kPitch;
        const int ch0 = kPer * sl;
        float x[kPer];
        if constexpr (kPer == 8) {
            const uint4 v = *reinterpret_cast<const uint4 *>(row + ch0);
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = bf16_bits_to_f32((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu));
        } else {
            const uint2 v = *reinterpret_cast<const uint2 *>(row + ch0);
            const uint32_t w[2] = {v.x, v.y};
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = bf16_bits_to_f32((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu));
        }
        uint32_t s16, z16;
        float z, inv;
        const bool quest = a.codec == WUSHKV_CODEC_QUEST;
        if (quest) {
            double ss = 0.0;
#pragma unroll
            for (int e = 0; e < kPer; ++e) ss = fma((double)x[e], (double)x[e], ss);
            auto add = [&](auto st) {
                constexpr int kStep = decltype(st)::value;
                const uint64_t u = __builtin_bit_cast(uint64_t, ss);
                const uint64_t o = ((uint64_t)row16_swap<kStep>((uint32_t)(u >> 32)) << 32) |
                                   row16_swap<kStep>((uint32_t)u);
                ss += __builtin_bit_cast(double, o);
            };
            add(std::integral_constant<int, 0>{});
            add(std::integral_constant<int, 1>{});
            add(std::integral_constant<int, 2>{});
            add(std::integral_constant<int, 3>{});
            quest_finish<D>(ss, a.quest_coef, kHalf, s16, z16, z, inv);
        } else {
            const int qlo = is_v ? a.lo_v : a.lo_k;
            const float qt = is_v ? a.t_v : a.t_k;
            const int K = D - qlo;
            float a_lo, a_hi, mn, mx;
            if (K <= 4) few_order_stats<4, kPer>(x, K, a_lo, a_hi, mn, mx);
            else if (K <= 8) few_order_stats<8, kPer>(x, K, a_lo, a_hi, mn, mx);
            else if (K <= 12) few_order_stats<12, kPer>(x, K, a_lo, a_hi, mn, mx);
            else few_order_stats<16, kPer>(x, K, a_lo, a_hi, mn, mx);
            quant_params(a_lo, a_hi, qt, qlo + 1 < D, mn, mx, kLevels, s16, z16, z, inv);
        }
        if (sl == 0)
            *reinterpret_cast<uint32_t *>(pg + L::kParamOffset + 4 * r + (is_v ? 4 * kPage : 0)) =
                s16 | (z16 << 16);
        uint32_t code[kPer];
        const float kLv = (float)kLevels;
#pragma unroll
        for (int e = 0; e < kPer; ++e)
            code[e] = quest ? quest_code_of(x[e], inv, kHalf, kLv) : code_of(x[e], z, inv, kLv);
        if (!is_v) {
            // this lane's channels lie in one key word: word w of 32-channel
            // chunk jc; the lanes sharing the word OR their bits together
            uint32_t bits = 0;
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
                int word, bit;
                L::k_pos(r, ch0 + e, word, bit);
                bits |= code[e] << bit;
            }
            if constexpr (kLanesPerWord >= 2) bits |= row16_swap<0>(bits);
            if constexpr (kLanesPerWord >= 4) bits |= row16_swap<1>(bits);
            if (sl % kLanesPerWord == 0) {
                const int jc = ch0 >> 5, w = (ch0 & 31) / kPerWord;
                reinterpret_cast<uint32_t *>(pg)[L::k_word(16 * jc + (r >> 2), BITS * (r & 3) + w)] = bits;
            }
        } else {
            // code bytes over the row, where phase C reads them (the whole
            // row was read by this wave's one load above)
            uint8_t *dst = vcode_row<D>(vt, r) + ch0 + (ch0 >= D / 2 ? D / 2 : 0);
            if constexpr (kPer == 8) {
                *reinterpret_cast<uint2 *>(dst) =
                    make_uint2(code[0] | code[1] << 8 | code[2] << 16 | code[3] << 24,
                               code[4] | code[5] << 8 | code[6] << 16 | code[7] << 24);
            } else {
                *reinterpret_cast<uint32_t *>(dst) = code[0] | code[1] << 8 | code[2] << 16 | code[3] << 24;
            }
        }
    }
    __syncthreads();
    value_words<D, BITS>(vt, blk_lo, [&](int32_t p) { return p >= lo && p < hi; }, false, pg, tid);
}

// Quantise positions [start, q_new) of (sequence b, kv head h) into their
// pages, one 64-position block at a time (Alg. 2 steps 7-11).  A position
// before s_ring comes from the windows' ring (keys row-major, values
// channel-major); one at or after it is a new token of this call, its key
// already transformed in kn (LDS, pitch D + 8) and its value in v_new.  kt
// and vt are 64-row LDS tiles, sh one LDS word.  Every thread of the
// 256-thread workgroup calls it.  kNewRows false: every position comes from
// the ring (s_ring and kn unused).
template <int D, int BITS, bool kNewRows>
__device__ void flush_range(const AppendArgs &a, int b, int h, int32_t start, int32_t q_new,
                            int32_t s_ring, const uint16_t *kn, uint16_t *kt, uint16_t *vt,
                            int32_t *sh, int tid)
{
    using L = Layout<D, BITS>;
    constexpr int kPitch = D + 8;
    constexpr int kVec = D / 8;
    const int32_t ring = a.win_slots - a.s_sink;
    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;
    for (int32_t blk = a.s_sink + (start - a.s_sink) / kPage * kPage; blk < q_new; blk += kPage) {
        const int32_t lo = max(blk, start), hi = min(blk + kPage, q_new);
        for (int idx = tid; idx < kPage * kVec; idx += 256) {
            const int r = idx / kVec, cv = idx % kVec;
            const int32_t p = blk + r;
            if (p < lo || p >= hi) continue;
            uint4 kv, vv;
            if (kNewRows && p >= s_ring) {
                kv = *reinterpret_cast<const uint4 *>(kn + (p - s_ring) * kPitch + 8 * cv);
                vv = *reinterpret_cast<const uint4 *>(
                    a.v_new + (((int64_t)b * a.max_new + (p - s_ring)) * a.n_kv + h) * D + 8 * cv);
            } else {
                const int32_t slot = ring_slot(p, a.s_sink, ring);
                kv = *reinterpret_cast<const uint4 *>(a.win_k + (head_win + slot) * D + 8 * cv);
                const uint16_t *vsrc = a.win_v + (head_win * D) + slot;  // channel-major
                uint16_t e[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) e[q] = vsrc[(int64_t)(8 * cv + q) * a.win_slots];
                vv.x = e[0] | ((uint32_t)e[1] << 16);
                vv.y = e[2] | ((uint32_t)e[3] << 16);
                vv.z = e[4] | ((uint32_t)e[5] << 16);
                vv.w = e[6] | ((uint32_t)e[7] << 16);
            }
            *reinterpret_cast<uint4 *>(kt + r * kPitch + 8 * cv) = kv;
            *reinterpret_cast<uint4 *>(vt + r * kPitch + 8 * cv) = vv;
        }
        if (tid == 0) {
            const int32_t lp = (blk - a.s_sink) / kPage;
            int32_t phys = -1;
            if (lp < a.max_pages) {
                phys = a.page_table[(int64_t)b * a.max_pages + lp];
                if (phys < 0 || phys >= a.n_pages) phys = -1;
            }
            sh[0] = phys;
        }
        __syncthreads();
        const int32_t page = sh[0];
        uint8_t *pg = page >= 0 ? a.pages + ((int64_t)page * a.n_kv + h) * L::kPageBytes : nullptr;
        // a short range (a decode step's flush): 16 lanes per group
        const bool few = hi - lo <= 8 &&
                         (a.codec == WUSHKV_CODEC_QUEST || (D - a.lo_k <= 16 && D - a.lo_v <= 16));
        if (few)
            quantise_few<D, BITS>(a, kt, vt, blk, lo, hi, pg, tid);
        else
            quantise_tile<D, BITS>(a, kt, vt, blk, [&](int32_t p) { return p >= lo && p < hi; },
                                   lo <= blk && blk + kPage <= hi, pg, tid);
        __syncthreads();
    }
}

}  // namespace wushkv
