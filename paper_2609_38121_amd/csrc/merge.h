// Log-sum-exp merge of split-K attention partials (Eq. (2) evaluated over
// disjoint position ranges and recombined), shared by the decode combine
// kernel and the fused step's finishing kernel.
#pragma once
#include "common.h"

namespace wushkv {

constexpr int kMaxSplits = 1024;

// One query head: the n_splits partials (o[D] relative to m, m, l) at pp,
// pp + stride, ..  (m in base 2) merge into
//   dst = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s,  M = max_s m_s,
// zero when no split saw a position.  Threads 0 .. D - 1 of the workgroup own
// one channel each; every thread of the workgroup calls it (barriers).  fw:
// kMaxSplits floats of LDS, red: D floats.
template <int D>
__device__ __forceinline__ void merge_splits(const float *pp, int64_t stride, int32_t n_splits,
                                             float *dst, int tid, float *fw, float *red)
{
    const bool act = tid < D;
    float mx = -INFINITY;
    if (act) {
        for (int s = tid; s < n_splits; s += D) {
            const float m = pp[s * stride + D];
            fw[s] = m;
            mx = fmaxf(mx, m);
        }
        red[tid] = mx;
    }
    __syncthreads();
    for (int off = D / 2; off > 0; off >>= 1) {
        if (tid < off) red[tid] = fmaxf(red[tid], red[tid + off]);
        __syncthreads();
    }
    const float M = red[0];
    if (act)
        for (int s = tid; s < n_splits; s += D)
            fw[s] = (fw[s] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(fw[s] - M);
    __syncthreads();
    if (!act) return;
    float o = 0.0f, l = 0.0f;
    if (M != -INFINITY) {
#pragma unroll 8
        for (int s = 0; s < n_splits; ++s) {
            const float f = fw[s];
            o = fmaf(f, pp[s * stride + tid], o);
            l = fmaf(f, pp[s * stride + D + 1], l);
        }
    }
    dst[tid] = (l > 0.0f) ? o / l : 0.0f;
}

}  // namespace wushkv
