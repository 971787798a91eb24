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
//                          followed by the quantised pages; a split owns a
//                          run of units and each wave every fourth of them.
//                          Per unit a wave computes 64 scores with the
//                          16x16x32 bf16 matrix instruction (codes as the A
//                          operand, the G query heads as columns), keeps an
//                          online softmax, and accumulates P V with a second
//                          matrix product.  Partials (m, l, o) go to the
//                          workspace.
//   decode_combine_kernel  log-sum-exp merge of the splits.
//
// Scores against codes.  A stored key is k = s c + z per token, so
//   q~ . k = s (q~ . c) + z sum(q~).
// The codes are widened to bf16 as 128 + c 2^sh (see widen_word), hence
//   q~' . (128 + c 2^sh) = 128 sum(q~') + q~ . c   with q~' = q~ 2^-sh,
// and the correction 128 sum(q~') is subtracted per query head.  Values
// likewise: sum_t p_t (s_t c_t + z_t) = sum_t (p_t s_t) c_t + sum_t p_t z_t.
// q~' and the weights p_t s_t 2^-sh are split into bf16 hi + lo parts (about
// 16 significant bits) and both parts go through the matrix cores, so the
// products carry fp32-level accuracy.
#include "common.h"

namespace wushkv {

constexpr float kLog2e = 1.4426950408889634f;

struct DecodeArgs {
    const uint8_t *pages;
    const int32_t *page_table;
    const uint16_t *win_k;
    const uint16_t *win_v;
    const int32_t *seq_len;
    const int32_t *quant_end;
    int32_t n_kv, s_sink, win_slots, max_pages, n_pages;
    int32_t G, n_q;
    int32_t units_per_split, n_splits;
    const float *qt;  // [batch][n_q][D]
    float *part;      // [batch][n_kv][n_splits][G][D + 2]
};

// ------------------------------------------------------------------ q~

template <int D>
__global__ void __launch_bounds__(256) decode_qt_kernel(const uint16_t *q, const float *tinv,
                                                        float *qt, int32_t n_kv, int32_t G,
                                                        float scale)
{
    __shared__ float qs[8 * D];
    const int h = blockIdx.x, b = blockIdx.y;
    const int n_q = n_kv * G;
    const uint16_t *qb = q + ((int64_t)b * n_q + h * G) * D;
    for (int i = threadIdx.x; i < G * D; i += blockDim.x) qs[i] = bf16_bits_to_f32(qb[i]);
    __syncthreads();
    const float *T = tinv + (int64_t)h * D * D;
    for (int jj = threadIdx.x; jj < D; jj += blockDim.x) {
        float acc[8];
#pragma unroll
        for (int g = 0; g < 8; ++g) acc[g] = 0.0f;
        for (int i = 0; i < D; ++i) {
            const float t = T[(int64_t)i * D + jj];
#pragma unroll
            for (int g = 0; g < 8; ++g)
                if (g < G) acc[g] = fmaf(qs[g * D + i], t, acc[g]);
        }
        for (int g = 0; g < G; ++g) qt[((int64_t)b * n_q + h * G + g) * D + jj] = acc[g] * scale;
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
__device__ __forceinline__ float readlane_f(float x, int l)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// hi = bf16(x) (nearest even), lo = bf16(x - hi), for a pair of values.
__device__ __forceinline__ void split_hi_lo(float x0, float x1, uint32_t &hi, uint32_t &lo,
                                            float &h0, float &h1, float &l0, float &l1)
{
    hi = pack_bf16_rne(x0, x1);
    h0 = bf16_bits_to_f32(hi & 0xFFFFu);
    h1 = bf16_bits_to_f32(hi >> 16);
    lo = pack_bf16_rne(x0 - h0, x1 - h1);
    l0 = bf16_bits_to_f32(lo & 0xFFFFu);
    l1 = bf16_bits_to_f32(lo >> 16);
}

// Token of the page (or window unit) whose score lands in accumulator row
// 4 j + r of score tile tau.
__device__ __forceinline__ int score_token(int tau, int j, int r)
{
    return 32 * (tau >> 1) + 8 * j + 4 * (tau & 1) + r;
}

template <int D, int BITS>
__global__ void __launch_bounds__(256, 2) decode_main_kernel(DecodeArgs a)
{
    using L = Layout<D, BITS>;
    constexpr int kC = L::kChunks;    // D / 32
    constexpr int kNT = L::kNTiles;   // D / 16
    constexpr int kNw = L::kNw;
    constexpr int kWpl = L::kWordsPerLane;

    __shared__ float sC[4][16][D];
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
    const int32_t n_units = n_wunits + n_qpages;
    const int32_t ring = a.win_slots - a.s_sink;
    // ring holds positions [q_hi, S); the oldest sits at ring index a0
    const int32_t a0 = S > q_hi ? (q_hi - a.s_sink) % ring : 0;
    const int32_t ring_live = S > q_hi ? S - q_hi : 0;

    const float *qrow = a.qt + ((int64_t)b * a.n_q + h * G + g) * D;
    float zsum = 0.0f;  // sum of q~ over the channels (zero-point term)
    if (cls < 2) {
#pragma unroll
        for (int c = 0; c < kC; ++c)
#pragma unroll
            for (int i = 0; i < 8; ++i) zsum += qrow[32 * c + 8 * j + i];
    }
    zsum = wave_sum_xor_16_32(zsum);

    // B operands for the score products (hi and lo parts), rebuilt when the
    // wave switches between window units (plain q~) and pages (q~ 2^-sh).
    uint32_t bhi[kC][4], blo[kC][4];
    float qbias = 0.0f;  // 128 * sum of the operand values, pages only
    int mode = -1;       // 0 window, 1 pages
    auto build_b = [&](int m) {
        float part = 0.0f;
#pragma unroll
        for (int c = 0; c < kC; ++c)
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const float sc = m ? slot_scale<BITS>(2 * p) : 1.0f;
                float x0 = 0.0f, x1 = 0.0f;
                if (cls < 2) {
                    x0 = qrow[32 * c + 8 * j + 2 * p] * sc;
                    x1 = qrow[32 * c + 8 * j + 2 * p + 1] * sc;
                }
                float h0, h1, l0, l1;
                split_hi_lo(x0, x1, bhi[c][p], blo[c][p], h0, h1, l0, l1);
                part += (h0 + l0) + (h1 + l1);
            }
        qbias = m ? 128.0f * wave_sum_xor_16_32(part) : 0.0f;
        mode = m;
    };

    // online-softmax state
    float m_run[8];
#pragma unroll
    for (int gg = 0; gg < 8; ++gg) m_run[gg] = -INFINITY;
    float m_lane = -INFINITY;  // m_run[g] of this lane's column
    float l_lane = 0.0f;       // sum of p over this lane's tokens (hi columns only)
    float z_lane = 0.0f;       // value-side corrections (pages)
    f32x4 acc[kNT];
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int u_begin = split * a.units_per_split;
    const int u_end = min(u_begin + a.units_per_split, n_units);
    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;

    for (int u = u_begin + wave; u < u_end; u += 4) {
        const bool is_win = u < n_wunits;
        // ---- locate the unit, its valid tokens and load its operands
        int32_t nvalid = 0;
        const uint8_t *pgb = nullptr;
        int32_t slot0 = 0;
        if (!is_win) {
            const int32_t lp = u - n_wunits;
            const int32_t phys = lp < a.max_pages ? a.page_table[(int64_t)b * a.max_pages + lp] : -1;
            if (phys < 0 || phys >= a.n_pages) continue;
            pgb = a.pages + ((int64_t)phys * a.n_kv + h) * L::kPageBytes;
            nvalid = min(kPage, q_hi - (a.s_sink + lp * kPage));
        } else {
            slot0 = u * kPage;
        }
        auto win_valid = [&](int t) -> bool {
            const int32_t sl = slot0 + t;
            if (sl < a.s_sink) return sl < S;
            const int32_t off = (sl - a.s_sink - a0 + ring) % ring;
            return off < ring_live;
        };
        auto tok_valid = [&](int t) -> bool { return is_win ? win_valid(t) : t < nvalid; };
        if (is_win) {
            bool any = false;
            for (int t = lane; t < kPage; t += 64) any |= win_valid(t);
            if (!__any(any)) continue;
        }
        if (mode != (is_win ? 0 : 1)) build_b(is_win ? 0 : 1);

        // ---- scores: S^T[token][col] for four tiles of 16 tokens
        f32x4 sc[4];
        uint32_t vw[kWpl];
        uint32_t kp[2][8], vp[2][8];
        if (!is_win) {
            const u32x4 *kr = reinterpret_cast<const u32x4 *>(pgb) + lane * (kWpl / 4);
            const u32x4 *vr = reinterpret_cast<const u32x4 *>(pgb + L::kRegionBytes) + lane * (kWpl / 4);
            uint32_t kw[kWpl];
#pragma unroll
            for (int q4 = 0; q4 < kWpl / 4; ++q4) {
                u32x4 x = kr[q4], y = vr[q4];
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
                    u32x4 x = kpr[(32 * kc + 8 * j) / 4 + h2];
                    u32x4 y = vpr[(32 * kc + 8 * j) / 4 + h2];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        kp[kc][4 * h2 + e] = x[e];
                        vp[kc][4 * h2 + e] = y[e];
                    }
                }
#pragma unroll
            for (int tau = 0; tau < 4; ++tau) {
                sc[tau] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int w = 0; w < kNw; ++w) {
                    uint32_t op[L::kCodesPerWord / 2];
                    widen_word<BITS>(kw[tau * kNw + w], op);
#pragma unroll
                    for (int o = 0; o < L::kOpsPerWord; ++o) {
                        const int c = w * L::kOpsPerWord + o;
                        const bf16x8 A = as_op(op + 4 * o);
                        sc[tau] = mfma16(A, __builtin_bit_cast(bf16x8, u32x4{bhi[c][0], bhi[c][1], bhi[c][2], bhi[c][3]}), sc[tau]);
                        sc[tau] = mfma16(A, __builtin_bit_cast(bf16x8, u32x4{blo[c][0], blo[c][1], blo[c][2], blo[c][3]}), sc[tau]);
                    }
                }
            }
        } else {
            const uint16_t *wk = a.win_k + (head_win + slot0) * D;
#pragma unroll
            for (int tau = 0; tau < 4; ++tau) {
                const int t = score_token(tau, n >> 2, n & 3);  // A row n of tile tau
                const bool ok = win_valid(t);
                sc[tau] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < kC; ++c) {
                    u32x4 x = {0u, 0u, 0u, 0u};
                    if (ok) x = *reinterpret_cast<const u32x4 *>(wk + (int64_t)t * D + 32 * c + 8 * j);
                    const bf16x8 A = __builtin_bit_cast(bf16x8, x);
                    sc[tau] = mfma16(A, __builtin_bit_cast(bf16x8, u32x4{bhi[c][0], bhi[c][1], bhi[c][2], bhi[c][3]}), sc[tau]);
                    sc[tau] = mfma16(A, __builtin_bit_cast(bf16x8, u32x4{blo[c][0], blo[c][1], blo[c][2], blo[c][3]}), sc[tau]);
                }
            }
        }

        // ---- logits (base 2), masked
        float lg[4][4];
        float mloc = -INFINITY;
#pragma unroll
        for (int tau = 0; tau < 4; ++tau)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = score_token(tau, j, r);
                float v;
                if (!is_win) {
                    const uint32_t kprm = kp[tau >> 1][4 * (tau & 1) + r];
                    const float ks = f16_bits_to_f32(kprm & 0xFFFFu), kz = f16_bits_to_f32(kprm >> 16);
                    v = fmaf(ks, sc[tau][r] - qbias, kz * zsum);
                } else {
                    v = sc[tau][r];
                }
                v = (cls < 2 && tok_valid(t)) ? v : -INFINITY;
                lg[tau][r] = v;
                mloc = fmaxf(mloc, v);
            }
        mloc = wave_max_xor_16_32(mloc);
        const float m_new_lane = fmaxf(m_lane, mloc);
        // rescale when any column's running max moved
        bool moved = false;
        float alpha[8];
#pragma unroll
        for (int gg = 0; gg < 8; ++gg) {
            float mn = gg < G ? fmaxf(m_run[gg], readlane_f(mloc, gg)) : -INFINITY;
            alpha[gg] = (mn == -INFINITY) ? 1.0f : fexp2(m_run[gg] - mn);
            moved |= (mn != m_run[gg]) && gg < G;
            m_run[gg] = gg < G ? mn : m_run[gg];
        }
        if (moved) {
            const float al = (m_new_lane == -INFINITY) ? 1.0f : fexp2(m_lane - m_new_lane);
            l_lane *= al;
            z_lane *= al;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int gr = (4 * j + r) & (G - 1);
                float ar = alpha[0];
#pragma unroll
                for (int gg = 1; gg < 8; ++gg) ar = (gr == gg) ? alpha[gg] : ar;
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt) acc[nt][r] *= ar;
            }
        }
        m_lane = m_new_lane;

        // ---- probabilities -> A operand of the P V product
        uint32_t aop[2][4];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                float w2[2], pr2[2], vz2[2];
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const int i = 2 * p + e;              // slot: token 32 kc + 8 j + i
                    const int tau = 2 * kc + (i >> 2), r = i & 3;
                    const float pr = (lg[tau][r] == -INFINITY) ? 0.0f : fexp2(lg[tau][r] - m_new_lane);
                    pr2[e] = pr;
                    if (!is_win) {
                        const uint32_t vprm = vp[kc][i];
                        const float vs = f16_bits_to_f32(vprm & 0xFFFFu);
                        vz2[e] = (pr == 0.0f) ? 0.0f : pr * f16_bits_to_f32(vprm >> 16);
                        w2[e] = (pr == 0.0f) ? 0.0f : pr * (vs * slot_scale<BITS>(i));
                    } else {
                        vz2[e] = 0.0f;
                        w2[e] = pr;
                    }
                }
                uint32_t hi, lo;
                float h0, h1, l0, l1;
                split_hi_lo(w2[0], w2[1], hi, lo, h0, h1, l0, l1);
                aop[kc][p] = cls == 0 ? hi : (cls == 1 ? lo : 0u);
                if (cls == 0) {
                    l_lane += pr2[0] + pr2[1];
                    if (!is_win) z_lane += (vz2[0] + vz2[1]) - 128.0f * (h0 + h1);
                } else if (cls == 1 && !is_win) {
                    z_lane -= 128.0f * (l0 + l1);
                }
            }
        }

        // ---- P V
        if (!is_win) {
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const bf16x8 A = as_op(aop[kc]);
#pragma unroll
                for (int uu = 0; uu < 2 * kNw; ++uu) {
                    uint32_t op[L::kCodesPerWord / 2];
                    widen_word<BITS>(vw[kc * 2 * kNw + uu], op);
#pragma unroll
                    for (int o = 0; o < L::kOpsPerWord; ++o) {
                        const int nt = uu * L::kOpsPerWord + o;
                        acc[nt] = mfma16(A, as_op(op + 4 * o), acc[nt]);
                    }
                }
            }
        } else {
            const uint16_t *wv = a.win_v + head_win * D + slot0;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                const bf16x8 A = as_op(aop[kc]);
                uint32_t msk[4];
                bool anyv = false;
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    const bool v0 = win_valid(32 * kc + 8 * j + 2 * p);
                    const bool v1 = win_valid(32 * kc + 8 * j + 2 * p + 1);
                    msk[p] = (v0 ? 0x0000FFFFu : 0u) | (v1 ? 0xFFFF0000u : 0u);
                    anyv |= v0 | v1;
                }
#pragma unroll
                for (int nt = 0; nt < kNT; ++nt) {
                    const int ch = 16 * nt + n;
                    u32x4 x = {0u, 0u, 0u, 0u};
                    if (anyv)
                        x = *reinterpret_cast<const u32x4 *>(wv + (int64_t)ch * a.win_slots + 32 * kc + 8 * j);
                    u32x4 y = {x[0] & msk[0], x[1] & msk[1], x[2] & msk[2], x[3] & msk[3]};
                    acc[nt] = mfma16(A, __builtin_bit_cast(bf16x8, y), acc[nt]);
                }
            }
        }
    }

    // ---- combine the four waves of the workgroup through LDS
    l_lane = wave_sum_xor_16_32(l_lane);
    z_lane = wave_sum_xor_16_32(z_lane);
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) sC[wave][4 * j + r][16 * nt + n] = acc[nt][r];
    if (lane < 8) {
        sM[wave][lane] = lane < G ? m_run[0] : -INFINITY;
#pragma unroll
        for (int gg = 1; gg < 8; ++gg)
            if (lane == gg) sM[wave][lane] = gg < G ? m_run[gg] : -INFINITY;
    }
    // lanes n < G (j = 0) hold l for column g; lanes n < 2G hold z parts
    if (lane < G) sL[wave][lane] = l_lane;
    if (lane < 2 * G && lane >= G) sZ[wave][lane - G] = z_lane;
    __syncthreads();
    if (lane < G) sZ[wave][lane] += z_lane;  // hi part joins the lo part
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
                o += f * (sC[w][gg][ch] + sC[w][gg + G][ch] + sZ[w][gg]);
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

template <int D>
__global__ void __launch_bounds__(D) decode_combine_kernel(const float *part, float *out,
                                                           int32_t n_kv, int32_t G,
                                                           int32_t n_splits)
{
    const int qh = blockIdx.x, b = blockIdx.y;
    const int h = qh / G, g = qh % G;
    const int ch = threadIdx.x;
    const int n_q = n_kv * G;
    const float *pp = part + (((int64_t)b * n_kv + h) * n_splits) * G * (D + 2) + g * (D + 2);
    const int64_t stride = (int64_t)G * (D + 2);
    float mx = -INFINITY;
    for (int s = 0; s < n_splits; ++s) mx = fmaxf(mx, pp[s * stride + D]);
    float o = 0.0f, l = 0.0f;
    if (mx != -INFINITY) {
        for (int s = 0; s < n_splits; ++s) {
            const float ms = pp[s * stride + D];
            if (ms == -INFINITY) continue;
            const float f = fexp2(ms - mx);
            o += f * pp[s * stride + ch];
            l += f * pp[s * stride + D + 1];
        }
    }
    out[((int64_t)b * n_q + qh) * D + ch] = (l > 0.0f) ? o / l : 0.0f;
}

// ------------------------------------------------------------------ host

struct DecodePlan {
    int32_t units_per_split, n_splits;
    size_t qt_bytes, part_bytes;
};

static bool make_plan(const wushkv_cache *c, int32_t n_q, int32_t max_seq_len, DecodePlan &p)
{
    const int32_t G = n_q / c->n_kv_heads;
    const int64_t qpages = max_seq_len > c->s_sink ? (max_seq_len - c->s_sink + kPage - 1) / kPage : 0;
    const int64_t units = c->win_slots / kPage + qpages;
    const int64_t heads = (int64_t)c->batch * c->n_kv_heads;
    // aim at about 4096 workgroups, at least 4 units (one per wave) each,
    // in multiples of 4 so the waves of a split share its units evenly
    int64_t ups = (units * heads + 4095) / 4096;
    if (ups < 4) ups = 4;
    ups = (ups + 3) / 4 * 4;
    const int64_t splits = (units + ups - 1) / ups;
    if (splits < 1 || splits > 65535) return false;
    p.units_per_split = (int32_t)ups;
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
    a.units_per_split = p.units_per_split;
    a.n_splits = p.n_splits;
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
