// wushkv_decode_attention: split-K GQA decode attention over the mixed
// bf16 / packed-code cache (Alg. 2 step 5, Eq. (2)), with the query-side
// compensation q~ = q^T T_K^{-1} of Eq. (3).
//
// Three launches on the caller's stream:
//   decode_qt_kernel       q~ for every query head, scaled by sm_scale log2(e)
//                          so that the softmax runs in base 2.
//   decode_main_kernel     grid (splits, kv heads, batch), four waves per
//                          workgroup.  The "units" of a (sequence, head) are
//                          the win_slots / 64 window units (bf16 sink + ring)
//                          followed by the quantised pages.  A split owns a
//                          run of units and each wave a contiguous part of
//                          it; while a wave computes one page it has the next
//                          page's words and parameters in flight.  Per unit
//                          the wave forms 64 scores with the 16x16x32 bf16
//                          matrix instruction (codes as the A operand, the G
//                          query heads as columns), keeps an online softmax
//                          and accumulates P V with a second matrix product.
//                          The four waves merge in LDS; the workgroup writes
//                          one partial (m, l, o) per query head.
//   decode_combine_kernel  log-sum-exp merge of the splits.
//
// Scores against codes.  A stored key is k = s c + z per token, so
//   q~ . k = s (q~ . c) + z sum(q~).
// The codes are widened to bf16 as 128 + c 2^sh (see widen_word), hence
//   q~' . (128 + c 2^sh) = 128 sum(q~') + q~ . c   with q~' = q~ 2^-sh,
// and the correction 128 sum(q~') is subtracted per query head.  Values
// likewise: sum_t p_t (s_t c_t + z_t) = sum_t (p_t s_t) c_t + sum_t p_t z_t;
// value codes are widened to fp16 as 1024 + c 4^p and the weights
// p_t s_t 4^-p enter the fp16 product as one fp16 operand (11 significant
// bits, a relative error below 2.5e-4 per weight); the 1024 offset is removed
// with one more matrix product against a constant-1024 operand, which yields
// 1024 sum_t A_t per row.  q~' is split into bf16 hi + lo parts (about 16
// significant bits), so the scores carry fp32-level accuracy.
#include "common.h"

namespace wushkv {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxSplits = 1024;

struct DecodeArgs {
    const uint8_t *pages;
    const int32_t *page_table;
    const uint16_t *win_k;
    const uint16_t *win_v;
    const int32_t *seq_len;
    const int32_t *quant_end;
    int32_t n_kv, s_sink, win_slots, max_pages, n_pages;
    int32_t G, n_q;
    int32_t units_per_wave, n_splits;
    WidenMasks wk, wv;  // key codes to bf16, value codes to fp16
    const float *qt;  // [batch][n_q][D]
    float *part;      // [batch][n_kv][n_splits][G][D + 2]
};

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------------------ q~

// One workgroup per (kv head, sequence).  Thread (ig, jg) multiplies a block
// of rows i of T^{-1} (kRows of them) by the G queries for 8 output channels
// j; all of a thread's loads are independent and issued together, and the
// row blocks are summed in LDS.
template <int D>
__global__ void __launch_bounds__(256) decode_qt_kernel(const uint16_t *q, const float *tinv,
                                                        float *qt, int32_t n_kv, int32_t G,
                                                        float scale)
{
    constexpr int kJG = D / 8;        // groups of 8 output channels
    constexpr int kIG = 256 / kJG;    // groups of rows
    constexpr int kRows = D / kIG;    // rows per group
    __shared__ float qs[8 * D];
    __shared__ float red[kIG][8][D];
    const int h = blockIdx.x, b = blockIdx.y;
    const int n_q = n_kv * G;
    const uint16_t *qb = q + ((int64_t)b * n_q + h * G) * D;
    for (int i = threadIdx.x; i < G * D; i += 256) qs[i] = bf16_bits_to_f32(qb[i]);
    const int jg = threadIdx.x % kJG, ig = threadIdx.x / kJG;
    const float *T = tinv + (int64_t)h * D * D + (int64_t)ig * kRows * D + 8 * jg;
    f32x4 t[kRows][2];
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        t[r][0] = *reinterpret_cast<const f32x4 *>(T + (int64_t)r * D);
        t[r][1] = *reinterpret_cast<const f32x4 *>(T + (int64_t)r * D + 4);
    }
    __syncthreads();
    for (int g = 0; g < G; ++g) {
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const float qi = qs[g * D + ig * kRows + r];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = fmaf(qi, t[r][e >> 2][e & 3], acc[e]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) red[ig][g][8 * jg + e] = acc[e];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * D; idx += 256) {
        const int g = idx / D, jj = idx % D;
        float s = 0.0f;
#pragma unroll
        for (int k = 0; k < kIG; ++k) s += red[k][g][jj];
        qt[((int64_t)b * n_q + h * G + g) * D + jj] = s * scale;
    }
}

// ------------------------------------------------------------------ main

__device__ __forceinline__ float wave_max_xor_16_32(float x)
{
    x = fmaxf(x, __shfl_xor(x, 16));
    x = fmaxf(x, __shfl_xor(x, 32));
    return x;
}
__device__ __forceinline__ float wave_sum_xor_16_32(float x)
{
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

__device__ __forceinline__ float bf16_hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// hi = bf16(x) (nearest even), lo = bf16(x - hi), for a pair of values.
__device__ __forceinline__ void split_hi_lo(float x0, float x1, uint32_t &hi, uint32_t &lo)
{
    hi = pack_bf16_rne(x0, x1);
    lo = pack_bf16_rne(x0 - bf16_bits_to_f32(hi & 0xFFFFu), x1 - bf16_hi_to_f32(hi));
}

// Token of the page (or window unit) whose score lands in accumulator row
// 4 j + r of score tile tau.
__device__ __forceinline__ int score_token(int tau, int j, int r)
{
    return 32 * (tau >> 1) + 8 * j + 4 * (tau & 1) + r;
}

__device__ __forceinline__ void __attribute__((address_space(3))) *lds_ptr(void *p)
{
    return (void __attribute__((address_space(3))) *)p;
}

// 16-byte LDS read of page data staged by the direct-to-LDS loads.  Written
// as inline assembly because the compiler, unable to tell the staging slots
// apart, would otherwise wait for every outstanding load before any LDS read
// and undo the pipelining.  The caller waits for the data with
// lds_reads_done() before using it; stage_ready() has already ensured the
// page itself has arrived.
__device__ __forceinline__ u32x4 lds_read16(const uint8_t *p)
{
    u32x4 r;
    const uint32_t addr = (uint32_t)(uintptr_t)lds_ptr(const_cast<uint8_t *>(p));
    asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr) : "memory");
    return r;
}

// Wait for the LDS reads above.  The read results pass through the asm as
// read-write operands, so nothing that uses them can be scheduled before it.
template <int NX>
__device__ __forceinline__ void lds_reads_done(u32x4 (&x)[NX], u32x4 (&y)[2][2])
{
    static_assert(NX == 1 || NX == 2 || NX == 4, "words per lane");
    if constexpr (NX == 1)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(x[0]), "+v"(y[0][0]), "+v"(y[0][1]), "+v"(y[1][0]), "+v"(y[1][1])::"memory");
    else if constexpr (NX == 2)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(x[0]), "+v"(x[1]), "+v"(y[0][0]), "+v"(y[0][1]), "+v"(y[1][0]),
                       "+v"(y[1][1])::"memory");
    else
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(y[0][0]),
                       "+v"(y[0][1]), "+v"(y[1][0]), "+v"(y[1][1])::"memory");
}

// Wait until at most `after` direct-to-LDS loads are outstanding.  `after`
// is a multiple of kDma between 0 and kMaxAhead * kDma; the count must be an
// immediate, hence the cases.  The memory clobber keeps LDS reads below it.
template <int kMaxAhead, int kDma>
__device__ __forceinline__ void wait_vmcnt_at_most(int after)
{
    static_assert(kMaxAhead * kDma <= 63, "vmcnt immediate");
    if (after <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if (after <= kDma) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kDma) : "memory");
    else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kMaxAhead * kDma) : "memory");
}

// Packed operands and parameters of one page, as one lane holds them.
template <int D, int BITS>
struct PageRegs {
    using L = Layout<D, BITS>;
    uint32_t kw[L::kWordsPerLane];
    uint32_t vw[L::kWordsPerLane];
    uint32_t kp[2][8];  // (scale, zero) of tokens 32 kc + 8 j + i
    uint32_t vp[2][8];

    __device__ __forceinline__ void load(const uint8_t *pgb, int lane, int j)
    {
        constexpr int kQ = L::kWordsPerLane / 4;
        const u32x4 *kr = reinterpret_cast<const u32x4 *>(pgb) + lane * kQ;
        const u32x4 *vr = reinterpret_cast<const u32x4 *>(pgb + L::kRegionBytes) + lane * kQ;
#pragma unroll
        for (int q4 = 0; q4 < kQ; ++q4) {
            const u32x4 x = kr[q4], y = vr[q4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                kw[4 * q4 + e] = x[e];
                vw[4 * q4 + e] = y[e];
            }
        }
        const u32x4 *kpr = reinterpret_cast<const u32x4 *>(pgb + L::kParamOffset);
        const u32x4 *vpr = reinterpret_cast<const u32x4 *>(pgb + L::kParamOffset + 4 * kPage);
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const u32x4 x = kpr[(32 * kc + 8 * j) / 4 + h2];
                const u32x4 y = vpr[(32 * kc + 8 * j) / 4 + h2];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    kp[kc][4 * h2 + e] = x[e];
                    vp[kc][4 * h2 + e] = y[e];
                }
            }
    }
};

// One wave's online softmax and output accumulators.
template <int D>
struct WaveState {
    static constexpr int kNT = D / 16;
    f32x4 acc[kNT];  // P V accumulators, rows 4 j + r (head g: hi row g, lo row g + G)
    f32x4 accb;      // 128 sum_t A_t per row (offset of the widened value codes)
    float m_lane;    // running max of this lane's column
    float l_lane;    // sum of p over this lane's tokens
    float z_lane;    // sum of p * value zero over this lane's tokens

    __device__ __forceinline__ void init()
    {
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        accb = f32x4{0.f, 0.f, 0.f, 0.f};
        m_lane = -INFINITY;
        l_lane = 0.0f;
        z_lane = 0.0f;
    }

    // Fold a unit's column max into the running max; rescale on change.
    // Accumulator row 4 j + r belongs to head (4 j + r) mod G, whose factor
    // lane (4 j + r) mod G holds (every lane of a column has the same max).
    __device__ __forceinline__ void update_max(float mloc, int j, int G)
    {
        const float m_new = fmaxf(m_lane, mloc);
        if (__any(m_new > m_lane)) {
            const float al = (m_new == -INFINITY) ? 1.0f : fexp2(m_lane - m_new);
            l_lane *= al;
            z_lane *= al;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float ar = __shfl(al, (4 * j + r) & (G - 1));
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt) acc[nt][r] *= ar;
                accb[r] *= ar;
            }
        }
        m_lane = m_new;
    }
};

template <int D, int BITS>
__global__ void __launch_bounds__(256, 2) decode_main_kernel(DecodeArgs a)
{
    using L = Layout<D, BITS>;
    // pages per wave in LDS (kStages - 1 in flight): three for pages up to
    // 5 KB, two for the 8.5 KB 4-bit pages, keeping two workgroups per CU
    constexpr int kStages = L::kPageBytes <= 5120 ? 3 : 2;
    constexpr int kC = L::kChunks;   // D / 32
    constexpr int kNT = L::kNTiles;  // D / 16
    constexpr int kNw = L::kNw;
    constexpr int kOpw = L::kOpsPerWord;

    // page stages of the four waves; after its loops a wave reuses its own
    // stage area for its slice of the merge buffer
    constexpr int kPB = L::kPageBytes;
    constexpr int kDma = (kPB + 1023) / 1024;  // direct-to-LDS loads per page
    constexpr int kSlot = kDma * 1024;
    constexpr int kWaveLds = kStages * kSlot > 16 * D * 4 ? kStages * kSlot : 16 * D * 4;
    __shared__ __attribute__((aligned(16))) uint8_t lds[4 * kWaveLds];
    __shared__ float sM[4][8], sL[4][8], sZ[4][8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = lane >> 4, n = lane & 15;
    const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int G = a.G;
    const int g = n & (G - 1);
    const int cls = n < G ? 0 : (n < 2 * G ? 1 : 2);  // 0: hi column/row, 1: lo, 2: unused

    const int32_t S = a.seq_len[b];
    int32_t qend = a.quant_end[b];
    qend = qend < S ? qend : S;
    const int32_t q_hi = qend > a.s_sink ? qend : a.s_sink;  // quantised: [s_sink, q_hi)
    const int32_t n_qpages = (q_hi - a.s_sink + kPage - 1) / kPage;
    const int32_t n_wunits = a.win_slots / kPage;
    const int32_t n_units = n_qpages + n_wunits;  // pages first, then the window units
    const int32_t ring = a.win_slots - a.s_sink;
    // the ring holds positions [q_hi, S); the oldest sits at ring index a0
    const int32_t a0 = S > q_hi ? (q_hi - a.s_sink) % ring : 0;
    const int32_t ring_live = S > q_hi ? S - q_hi : 0;

    // this wave's units
    const int upw = a.units_per_wave;
    const int w0 = (split * 4 + wave) * upw;
    const int w1 = min(w0 + upw, n_units);

    const float *qrow = a.qt + ((int64_t)b * a.n_q + h * G + g) * D;
    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;

    WaveState<D> st;
    st.init();

    // B operands of the score products: hi and lo parts of q~ (2^-sh scaled
    // for pages); columns n < 2G carry query head g = n mod G.
    uint32_t bhi[kC][4], blo[kC][4];
    float zsum = 0.0f, qbias = 0.0f;
    auto build_b = [&](bool pages) {
        float part = 0.0f, zs = 0.0f;
#pragma unroll
        for (int c = 0; c < kC; ++c) {
            float x[8];
            if (cls < 2) {
                const f32x4 lo4 = *reinterpret_cast<const f32x4 *>(qrow + 32 * c + 8 * j);
                const f32x4 hi4 = *reinterpret_cast<const f32x4 *>(qrow + 32 * c + 8 * j + 4);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[e] = lo4[e];
                    x[4 + e] = hi4[e];
                }
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = 0.0f;
            }
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                zs += x[2 * p] + x[2 * p + 1];
                const float sc = pages ? slot_scale<BITS>(2 * p) : 1.0f;
                split_hi_lo(x[2 * p] * sc, x[2 * p + 1] * sc, bhi[c][p], blo[c][p]);
                part += (bf16_bits_to_f32(bhi[c][p] & 0xFFFFu) + bf16_hi_to_f32(bhi[c][p])) +
                        (bf16_bits_to_f32(blo[c][p] & 0xFFFFu) + bf16_hi_to_f32(blo[c][p]));
            }
        }
        zsum = wave_sum_xor_16_32(zs);
        qbias = pages ? 128.0f * wave_sum_xor_16_32(part) : 0.0f;
    };
    auto bop = [](const uint32_t (&v)[4]) {
        return __builtin_bit_cast(bf16x8, u32x4{v[0], v[1], v[2], v[3]});
    };

    // ---------------------------------------------------- quantised pages
    // Pages are copied whole, global -> LDS, by the direct-to-LDS loads
    // (64 lanes x 16 B per instruction, lane l's bytes at slot + 16 l), so
    // a stage holds the page block byte for byte.  A wave keeps kStages - 1
    // pages in flight while it computes the oldest one; the compiler does not
    // track these loads, so the waits below are explicit.
    const int pw1 = min(w1, n_qpages);
    if (w0 < pw1) {
        build_b(true);
        // widening masks in scalar registers and the biases in vector
        // registers (one v_mov each, opaque to the optimizer), so that
        // (word & mask) | bias selects v_and_or_b32 with one scalar operand
        WidenMasks wk = a.wk, wv = a.wv;
        asm volatile("v_mov_b32 %0, %1" : "=v"(wk.bias) : "s"(a.wk.bias));
        asm volatile("v_mov_b32 %0, %1" : "=v"(wv.bias) : "s"(a.wv.bias));
        const f16x8 c1024 = __builtin_bit_cast(f16x8, u32x4{kBiasF16x2, kBiasF16x2, kBiasF16x2, kBiasF16x2});
        // the wave's page-table entries, one per lane, read once
        int32_t tbl = -1;
        if (w0 + lane < pw1 && w0 + lane < a.max_pages)
            tbl = a.page_table[(int64_t)b * a.max_pages + w0 + lane];
        uint8_t *stage = lds + wave * kWaveLds;
        // Every page of the run issues exactly kDma loads; a page-table entry
        // outside the pool loads physical page 0 instead (its data is never
        // used), which keeps the count of outstanding loads a closed form.
        auto phys_of = [&](int u) -> int32_t { return __builtin_amdgcn_readlane(tbl, u - w0); };
        auto issue = [&](int u, int s) {
            int32_t phys = phys_of(u);
            if (phys < 0 || phys >= a.n_pages) phys = 0;
            const uint8_t *src = a.pages + ((int64_t)phys * a.n_kv + h) * L::kPageBytes + 16 * lane;
            uint8_t *dst = stage + s * kSlot;
#pragma unroll
            for (int i = 0; i < kDma; ++i) {
                if (i + 1 < kDma || 1024 * i + 16 * lane < L::kPageBytes)
                    __builtin_amdgcn_global_load_lds(src + 1024 * i, lds_ptr(dst + 1024 * i), 16, 0, 0);
            }
        };
        if (a.n_pages > 0) {
#pragma unroll
        for (int s = 0; s < kStages - 1; ++s)
            if (w0 + s < pw1) issue(w0 + s, s);
        for (int u = w0; u < pw1; ++u) {
            const int s = (u - w0) % kStages;
            if (u + kStages - 1 < pw1) issue(u + kStages - 1, (u - w0 + kStages - 1) % kStages);
            // pages issued after page u: min(kStages - 1, pw1 - 1 - u)
            // stage_ready: page u has landed in LDS once at most the later
            // pages' loads are outstanding
            wait_vmcnt_at_most<kStages - 1, kDma>(kDma * min(kStages - 1, pw1 - 1 - u));
            {
                const int32_t phys = phys_of(u);
                if (phys < 0 || phys >= a.n_pages) continue;
            }
            const uint8_t *pg = stage + s * kSlot;
            const int32_t nvalid = min(kPage, q_hi - (a.s_sink + u * kPage));
            // scores S^T[token][column] - 128 sum q~', four tiles of 16 tokens
            uint32_t kw[L::kWordsPerLane];
            uint32_t kp[2][8];
            {
                u32x4 x[L::kWordsPerLane / 4], y[2][2];
#pragma unroll
                for (int q4 = 0; q4 < L::kWordsPerLane / 4; ++q4)
                    x[q4] = lds_read16(pg + 16 * (lane * (L::kWordsPerLane / 4) + q4));
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2)
                        y[kc][h2] = lds_read16(pg + L::kParamOffset + 4 * (32 * kc + 8 * j) + 16 * h2);
                lds_reads_done(x, y);
#pragma unroll
                for (int q4 = 0; q4 < L::kWordsPerLane / 4; ++q4)
#pragma unroll
                    for (int e = 0; e < 4; ++e) kw[4 * q4 + e] = x[q4][e];
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                        for (int e = 0; e < 4; ++e) kp[kc][4 * h2 + e] = y[kc][h2][e];
            }
            f32x4 sc[4];
#pragma unroll
            for (int tau = 0; tau < 4; ++tau) {
                sc[tau] = f32x4{-qbias, -qbias, -qbias, -qbias};
#pragma unroll
                for (int w = 0; w < kNw; ++w) {
                    uint32_t op[L::kCodesPerWord / 2];
                    widen_word<BITS>(kw[tau * kNw + w], op, wk);
#pragma unroll
                    for (int o = 0; o < kOpw; ++o) {
                        const int c = w * kOpw + o;
                        const bf16x8 A = as_op(op + 4 * o);
                        sc[tau] = mfma16(A, bop(bhi[c]), sc[tau]);
                        sc[tau] = mfma16(A, bop(blo[c]), sc[tau]);
                    }
                }
            }
            // logits (base 2): s (S - 128 sum q~') + z sum q~
            float lg[4][4];
#pragma unroll
            for (int tau = 0; tau < 4; ++tau)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const uint32_t kprm = kp[tau >> 1][4 * (tau & 1) + r];
                    lg[tau][r] = fmaf(f16_bits_to_f32(kprm & 0xFFFFu), sc[tau][r],
                                      f16_bits_to_f32(kprm >> 16) * zsum);
                }
            if (nvalid < kPage) {
#pragma unroll
                for (int tau = 0; tau < 4; ++tau)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (score_token(tau, j, r) >= nvalid) lg[tau][r] = -INFINITY;
            }
            float mloc = -INFINITY;
#pragma unroll
            for (int tau = 0; tau < 4; ++tau)
#pragma unroll
                for (int r = 0; r < 4; ++r) mloc = fmaxf(mloc, lg[tau][r]);
            st.update_max(wave_max_xor_16_32(mloc), j, G);
            // weights p s 4^-p as fp16, in the A rows g < G
            uint32_t vp[2][8];
            uint32_t vw[L::kWordsPerLane];
            {
                u32x4 x[L::kWordsPerLane / 4], y[2][2];
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2)
                        y[kc][h2] = lds_read16(pg + L::kParamOffset + 4 * kPage + 4 * (32 * kc + 8 * j) + 16 * h2);
#pragma unroll
                for (int q4 = 0; q4 < L::kWordsPerLane / 4; ++q4)
                    x[q4] = lds_read16(pg + L::kRegionBytes + 16 * (lane * (L::kWordsPerLane / 4) + q4));
                lds_reads_done(x, y);
#pragma unroll
                for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                        for (int e = 0; e < 4; ++e) vp[kc][4 * h2 + e] = y[kc][h2][e];
#pragma unroll
                for (int q4 = 0; q4 < L::kWordsPerLane / 4; ++q4)
#pragma unroll
                    for (int e = 0; e < 4; ++e) vw[4 * q4 + e] = x[q4][e];
            }
            uint32_t aop[2][4];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    float wv2[2];
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int i = 2 * p + e;  // slot: token 32 kc + 8 j + i
                        const float pr = fexp2(lg[2 * kc + (i >> 2)][i & 3] - st.m_lane);
                        const uint32_t vprm = vp[kc][i];
                        st.l_lane += pr;
                        st.z_lane = fmaf(pr, f16_bits_to_f32(vprm >> 16), st.z_lane);
                        wv2[e] = pr * (f16_bits_to_f32(vprm & 0xFFFFu) * slot_scale_f16<BITS>(i));
                    }
                    aop[kc][p] = cls == 0 ? pack_f16_rne(wv2[0], wv2[1]) : 0u;
                }
            // P V, plus the row sums that remove the 1024 offset
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const f16x8 A = __builtin_bit_cast(f16x8, u32x4{aop[kc][0], aop[kc][1], aop[kc][2], aop[kc][3]});
#pragma unroll
                for (int uu = 0; uu < 2 * kNw; ++uu) {
                    uint32_t op[L::kCodesPerWord / 2];
                    widen_word_f16<BITS>(vw[kc * 2 * kNw + uu], op, wv);
#pragma unroll
                    for (int o = 0; o < kOpw; ++o) {
                        const int nt = uu * kOpw + o;
                        st.acc[nt] = mfma16h(A, as_op_h(op + 4 * o), st.acc[nt]);
                    }
                }
                st.accb = mfma16h(A, c1024, st.accb);
            }
        }
        }
    }

    // ---------------------------------------------------- window units
    const int ww0 = max(w0, n_qpages);
    if (ww0 < w1) {
        build_b(false);
        for (int u = ww0; u < w1; ++u) {
            const int32_t slot0 = (u - n_qpages) * kPage;
            // slot validity of the unit, one bit per slot
            bool mine;
            {
                const int32_t sl = slot0 + lane;
                if (sl < a.s_sink) mine = sl < S;
                else mine = ((sl - a.s_sink - a0 + ring) % ring) < ring_live;
            }
            const uint64_t vmask = __ballot(mine);
            if (vmask == 0) continue;
            auto valid = [&](int t) -> bool { return (vmask >> t) & 1u; };
            const uint16_t *wk = a.win_k + (head_win + slot0) * D;
            // All loads stay inside this unit's slots, so they are issued
            // unconditionally (a branch per load would serialise them);
            // dead slots are zeroed afterwards, whatever bits they held.
            u32x4 kx[4][kC];
#pragma unroll
            for (int tau = 0; tau < 4; ++tau)
#pragma unroll
                for (int c = 0; c < kC; ++c)
                    kx[tau][c] = *reinterpret_cast<const u32x4 *>(
                        wk + (int64_t)score_token(tau, n >> 2, n & 3) * D + 32 * c + 8 * j);
            const uint16_t *wvp = a.win_v + head_win * D + slot0;
            u32x4 vx[2][kNT];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt)
                    vx[kc][nt] = *reinterpret_cast<const u32x4 *>(
                        wvp + (int64_t)(16 * nt + n) * a.win_slots + 32 * kc + 8 * j);
            f32x4 sc[4];
#pragma unroll
            for (int tau = 0; tau < 4; ++tau) {
                // A row n of tile tau is token score_token(tau, n / 4, n % 4)
                const uint32_t keep = valid(score_token(tau, n >> 2, n & 3)) ? 0xFFFFFFFFu : 0u;
                sc[tau] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < kC; ++c) {
                    const u32x4 x = {kx[tau][c][0] & keep, kx[tau][c][1] & keep,
                                     kx[tau][c][2] & keep, kx[tau][c][3] & keep};
                    const bf16x8 A = __builtin_bit_cast(bf16x8, x);
                    sc[tau] = mfma16(A, bop(bhi[c]), sc[tau]);
                    sc[tau] = mfma16(A, bop(blo[c]), sc[tau]);
                }
            }
            float lg[4][4];
            float mloc = -INFINITY;
#pragma unroll
            for (int tau = 0; tau < 4; ++tau)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float v = valid(score_token(tau, j, r)) ? sc[tau][r] : -INFINITY;
                    lg[tau][r] = v;
                    mloc = fmaxf(mloc, v);
                }
            st.update_max(wave_max_xor_16_32(mloc), j, G);
            uint32_t aop[2][4];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    float pr[2];
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int i = 2 * p + e;
                        pr[e] = fexp2(lg[2 * kc + (i >> 2)][i & 3] - st.m_lane);
                    }
                    st.l_lane += pr[0] + pr[1];
                    uint32_t hi, lo;
                    split_hi_lo(pr[0], pr[1], hi, lo);
                    aop[kc][p] = cls == 0 ? hi : (cls == 1 ? lo : 0u);
                }
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const bf16x8 A = bop(aop[kc]);
                const uint32_t bits8 = (uint32_t)(vmask >> (32 * kc + 8 * j)) & 0xFFu;
                uint32_t msk[4];
#pragma unroll
                for (int p = 0; p < 4; ++p)
                    msk[p] = (((bits8 >> (2 * p)) & 1u) ? 0x0000FFFFu : 0u) |
                             (((bits8 >> (2 * p + 1)) & 1u) ? 0xFFFF0000u : 0u);
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt) {
                    const u32x4 x = vx[kc][nt];
                    const u32x4 y = {x[0] & msk[0], x[1] & msk[1], x[2] & msk[2], x[3] & msk[3]};
                    st.acc[nt] = mfma16(A, __builtin_bit_cast(bf16x8, y), st.acc[nt]);
                }
            }
        }
    }

    // ---------------------------------------------------- merge the waves
    // head g: rows g (pages and window hi parts) and g + G (window lo parts)
    const float l_col = wave_sum_xor_16_32(st.l_lane);
    const float z_col = wave_sum_xor_16_32(st.z_lane);
    // this wave's stage reads are complete: every value read was consumed
    float(*sC)[16][D] = reinterpret_cast<float(*)[16][D]>(lds);
    auto sCw = [&](int w) -> float(*)[D] { return reinterpret_cast<float(*)[D]>(lds + w * kWaveLds); };
    {
        float(*mine)[D] = sCw(wave);
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) mine[4 * j + r][16 * nt + n] = st.acc[nt][r] - st.accb[r];
    }
    (void)sC;
    if (lane < G) {
        sM[wave][lane] = st.m_lane;
        sL[wave][lane] = l_col;
        sZ[wave][lane] = z_col;
    }
    __syncthreads();

    float *part = a.part + (((int64_t)b * a.n_kv + h) * a.n_splits + split) * G * (D + 2);
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
                o += f * (sCw(w)[gg][ch] + sCw(w)[gg + G][ch] + sZ[w][gg]);
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

// ------------------------------------------------------------------ combine

// One workgroup per (query head, sequence): the split maxima and weights go
// through LDS, then every channel thread sums its column with the loads
// unrolled so they are in flight together.
template <int D>
__global__ void __launch_bounds__(D) decode_combine_kernel(const float *part, float *out,
                                                           int32_t n_kv, int32_t G,
                                                           int32_t n_splits)
{
    __shared__ float fw[kMaxSplits];
    __shared__ float red[D];
    const int qh = blockIdx.x, b = blockIdx.y;
    const int h = qh / G, g = qh % G;
    const int ch = threadIdx.x;
    const int n_q = n_kv * G;
    const int64_t stride = (int64_t)G * (D + 2);
    const float *pp = part + (((int64_t)b * n_kv + h) * n_splits) * stride + g * (D + 2);
    float mx = -INFINITY;
    for (int s = ch; s < n_splits; s += D) {
        const float m = pp[s * stride + D];
        fw[s] = m;
        mx = fmaxf(mx, m);
    }
    red[ch] = mx;
    __syncthreads();
    for (int off = D / 2; off > 0; off >>= 1) {
        if (ch < off) red[ch] = fmaxf(red[ch], red[ch + off]);
        __syncthreads();
    }
    const float M = red[0];
    for (int s = ch; s < n_splits; s += D)
        fw[s] = (fw[s] == -INFINITY) ? 0.0f : fexp2(fw[s] - M);
    __syncthreads();
    float o = 0.0f, l = 0.0f;
    if (M != -INFINITY) {
#pragma unroll 8
        for (int s = 0; s < n_splits; ++s) {
            const float f = fw[s];
            o = fmaf(f, pp[s * stride + ch], o);
            l = fmaf(f, pp[s * stride + D + 1], l);
        }
    }
    out[((int64_t)b * n_q + qh) * D + ch] = (l > 0.0f) ? o / l : 0.0f;
}

// ------------------------------------------------------------------ host

struct DecodePlan {
    int32_t units_per_wave, n_splits;
    size_t qt_bytes, part_bytes;
};

static bool make_plan(const wushkv_cache *c, int32_t n_q, int32_t max_seq_len, DecodePlan &p)
{
    const int32_t G = n_q / c->n_kv_heads;
    const int64_t qpages = max_seq_len > c->s_sink ? (max_seq_len - c->s_sink + kPage - 1) / kPage : 0;
    const int64_t units = c->win_slots / kPage + qpages;
    const int64_t heads = (int64_t)c->batch * c->n_kv_heads;
    // about one full residency round of waves (256 CUs x 8 waves), with at
    // least 2 and at most 32 units per wave so ragged lengths still balance
    int64_t upw = (units * heads + 2047) / 2048;
    if (upw < 2) upw = 2;
    if (upw > 32) upw = 32;
    int64_t splits = (units + 4 * upw - 1) / (4 * upw);
    if (splits > kMaxSplits) {
        upw = (units + 4 * kMaxSplits - 1) / (4 * kMaxSplits);
        splits = (units + 4 * upw - 1) / (4 * upw);
    }
    if (splits < 1 || splits > kMaxSplits || upw > 0x7FFFFFFF / 4 / kMaxSplits) return false;
    p.units_per_wave = (int32_t)upw;
    p.n_splits = (int32_t)splits;
    p.qt_bytes = ((size_t)c->batch * n_q * c->head_dim * 4 + 255) / 256 * 256;
    p.part_bytes = (size_t)heads * splits * G * (c->head_dim + 2) * 4;
    return true;
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

extern "C" size_t wushkv_decode_workspace_bytes(const wushkv_cache *c, int32_t n_q_heads,
                                                int32_t max_seq_len)
{
    if (check_decode_args(c, n_q_heads, max_seq_len) != WUSHKV_OK) return 0;
    DecodePlan p;
    if (!make_plan(c, n_q_heads, max_seq_len, p)) return 0;
    return p.qt_bytes + p.part_bytes;
}

extern "C" int wushkv_decode_attention(const wushkv_cache *c, const uint16_t *q, int32_t n_q_heads,
                                       int32_t max_seq_len, const float *t_k_inv, float sm_scale,
                                       float *out, void *workspace, size_t workspace_bytes,
                                       wushkv_stream_t stream)
{
    int st = check_decode_args(c, n_q_heads, max_seq_len);
    if (st != WUSHKV_OK) return st;
    if (!q || !t_k_inv || !out || !workspace) return WUSHKV_EINVAL;
    if (((uintptr_t)q | (uintptr_t)t_k_inv | (uintptr_t)out | (uintptr_t)workspace) & 15u)
        return WUSHKV_EINVAL;
    if (!(sm_scale > 0.0f) || sm_scale == INFINITY) return WUSHKV_EINVAL;
    DecodePlan p;
    if (!make_plan(c, n_q_heads, max_seq_len, p)) return WUSHKV_EINVAL;
    if (workspace_bytes < p.qt_bytes + p.part_bytes) return WUSHKV_EWORKSPACE;

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int32_t G = n_q_heads / c->n_kv_heads;
    float *qt = reinterpret_cast<float *>(workspace);
    float *part = reinterpret_cast<float *>(reinterpret_cast<uint8_t *>(workspace) + p.qt_bytes);

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
    a.G = G;
    a.n_q = n_q_heads;
    a.units_per_wave = p.units_per_wave;
    a.n_splits = p.n_splits;
    a.wk = widen_masks(c->bits);
    a.wv = widen_masks_f16(c->bits);
    a.qt = qt;
    a.part = part;

    const dim3 gq(c->n_kv_heads, c->batch);
    const dim3 gm(p.n_splits, c->n_kv_heads, c->batch);
    const dim3 gc(n_q_heads, c->batch);
    const float scale = sm_scale * kLog2e;
    const int key = c->head_dim * 10 + c->bits;

    timing_begin("decode_qt_kernel", s);
    if (c->head_dim == 128) hipLaunchKernelGGL(decode_qt_kernel<128>, gq, dim3(256), 0, s, q, t_k_inv, qt, c->n_kv_heads, G, scale);
    else hipLaunchKernelGGL(decode_qt_kernel<64>, gq, dim3(256), 0, s, q, t_k_inv, qt, c->n_kv_heads, G, scale);
    timing_end(s);

    timing_begin("decode_main_kernel", s);
    switch (key) {
        case 1282: hipLaunchKernelGGL((decode_main_kernel<128, 2>), gm, dim3(256), 0, s, a); break;
        case 1284: hipLaunchKernelGGL((decode_main_kernel<128, 4>), gm, dim3(256), 0, s, a); break;
        case 642: hipLaunchKernelGGL((decode_main_kernel<64, 2>), gm, dim3(256), 0, s, a); break;
        case 644: hipLaunchKernelGGL((decode_main_kernel<64, 4>), gm, dim3(256), 0, s, a); break;
    }
    timing_end(s);

    timing_begin("decode_combine_kernel", s);
    if (c->head_dim == 128) hipLaunchKernelGGL(decode_combine_kernel<128>, gc, dim3(128), 0, s, part, out, c->n_kv_heads, G, p.n_splits);
    else hipLaunchKernelGGL(decode_combine_kernel<64>, gc, dim3(64), 0, s, part, out, c->n_kv_heads, G, p.n_splits);
    timing_end(s);
    if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
    return WUSHKV_OK;
}
