// wushkv_wush_transform: the WUSH transform of Eq. (1) for a batch of
// (Gram matrix M, Hessian H) pairs, one d x d transform per pair (Sec. 3;
// per key or value head in Eq. (4) and Alg. 1).
//
//   L L^T = H_d = H + gamma tr(H)/d I            Cholesky
//   U Lam U^T = L^T M_d L,  M_d = M + gamma tr(M)/d I
//   c = ((1 + gamma) tr(M))^(1/2) tr(Lam^(1/2))^(-1/2)
//   T = c Had Lam^(-1/4) U^T L^T,   T^{-1} = c^{-1} M_d (L U) Lam^(-3/4) Had
//
// (the second form of T^{-1} follows from L^{-T} U = M_d L U Lam^{-1}).
//
// One workgroup per pair, everything in one LDS frame of d columns, each
// column 2d entries long (a B half and an L half), fp32:
//   1. Cholesky of H_d into the L halves, of M_d (= R R^T) into the B halves;
//   2. B = R^T L, so that B^T B = L^T M_d L;
//   3. one-sided (Hestenes) Jacobi on the columns of [B; L]: plane rotations
//      that make the B columns mutually orthogonal, applied to the L columns
//      as well.  At convergence the B columns have squared norms Lam and the
//      L columns are L U: the eigendecomposition without forming L^T M_d L,
//      and with the eigenvalues' relative accuracy of a one-sided method.
//      The d/2 disjoint pairs of a round (a round-robin tournament) rotate in
//      parallel, each by 1024/d threads (512 per workgroup);
//   4. the eigenpairs in ascending order, each eigenvector's sign fixed so
//      that the largest-magnitude entry of L u_k is positive (the paper
//      fixes neither; Had mixes them, so T depends on both);
//   5. T by a fast Walsh-Hadamard transform of the rows Lam^(-1/4) (L U)^T,
//      and T^{-1} from the product M_d (L U) and a second transform.
#include <cmath>

#include "common.h"

namespace wushkv {

constexpr int kWushMaxSweeps = 40;
// Threads of a workgroup: eight waves, two per SIMD, so that one wave's LDS
// and barrier waits overlap the other's arithmetic (the frame's LDS admits
// one workgroup per compute unit).
constexpr int kWushThreads = 512;
constexpr int kWushWaves = kWushThreads / 64;

// Sum of one value per wave (in red[wave]) in a fixed order.
__device__ __forceinline__ float wave_total(const float *red)
{
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < kWushWaves; ++w) t += red[w];
    return t;
}

// Column stride of the LDS frame: 16-byte aligned, and 32 banks apart for
// neighbouring columns.  In a Jacobi round the eight lanes of a pair read
// 32 consecutive floats of its column (32 banks) and the next eight lanes
// the neighbouring column, so a 16-lane group's reads fall on distinct
// banks.
template <int D>
struct WushLds {
    static constexpr int kP = 2 * D + 32;
};

// Lane exchange within aligned groups of N lanes (N a power of two <= 64):
// the sum over the group, the same value in every lane of the group (each
// step adds the same two partial sums in every lane, so all lanes agree bit
// for bit).  Groups of up to 16 lanes sum by DPP inside the lanes' row:
// quad permutations, then the half-row and the row mirrors, which pair each
// quad (each half row) with the other one of its group.
template <int CTRL>
__device__ __forceinline__ float wush_dpp(float x)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF,
                                                                  0xF, false));
}
template <int N>
__device__ __forceinline__ float group_sum(float x)
{
    if constexpr (N <= 16) {
        if constexpr (N >= 2) x += wush_dpp<0xB1>(x);   // quad_perm [1, 0, 3, 2]
        if constexpr (N >= 4) x += wush_dpp<0x4E>(x);   // quad_perm [2, 3, 0, 1]
        if constexpr (N >= 8) x += wush_dpp<0x141>(x);  // row_half_mirror
        if constexpr (N >= 16) x += wush_dpp<0x140>(x); // row_mirror
        return x;
    } else {
#pragma unroll
        for (int off = 1; off < N; off <<= 1) x += __shfl_xor(x, off);
        return x;
    }
}

// In-place Cholesky of the symmetric matrix held in rows off .. off + D - 1
// of columns 0 .. D - 1 (entry (i, k) at X[k * P + off + i], lower triangle
// read): afterwards the lower triangle holds the factor and the upper is
// zero.  Returns false (in every thread) on a pivot that is not positive.
template <int D>
__device__ bool cholesky(float *X, int off, int tid)
{
    constexpr int P = WushLds<D>::kP;
    __shared__ int bad;
    if (tid == 0) bad = 0;
    __syncthreads();
    for (int j = 0; j < D; ++j) {
        float *cj = X + j * P + off;
        const float piv = cj[j];
        const float ljj = piv > 0.0f ? sqrtf(piv) : 0.0f;
        if (tid == 0 && !(piv > 0.0f)) bad = 1;
        const float inv = piv > 0.0f ? 1.0f / ljj : 0.0f;
        __syncthreads();  // every thread has read the pivot
        for (int i = j + 1 + tid; i < D; i += kWushThreads) cj[i] *= inv;
        if (tid == 0) cj[j] = ljj;
        __syncthreads();
        // trailing update of the lower triangle: A[i][k] -= l_i l_k, i >= k > j
        const int n = D - 1 - j;
        for (int e = tid; e < n * n; e += kWushThreads) {
            const int kk = e / n, ii = e % n;
            if (ii < kk) continue;
            const int k = j + 1 + kk, i = j + 1 + ii;
            X[k * P + off + i] -= cj[i] * cj[k];
        }
        __syncthreads();
    }
    for (int e = tid; e < D * D; e += kWushThreads) {
        const int k = e / D, i = e % D;
        if (i < k) X[k * P + off + i] = 0.0f;
    }
    __syncthreads();
    return bad == 0;
}

// Symmetric input (lower triangle read) into rows off .. of the frame, with
// damping gamma tr/d on the diagonal.  Returns tr (undamped).
template <int D>
__device__ float load_damped(const float *A, float *X, int off, float gamma, int tid, float *red)
{
    constexpr int P = WushLds<D>::kP;
    float t = 0.0f;
    for (int i = tid; i < D; i += kWushThreads) t += A[i * D + i];
    t = group_sum<64>(t);
    if ((tid & 63) == 0) red[tid >> 6] = t;
    __syncthreads();
    const float tr = wave_total(red);
    const float damp = gamma * tr / (float)D;
    for (int e = tid; e < D * D; e += kWushThreads) {
        const int i = e / D, k = e % D;  // row-major read, coalesced
        if (i >= k) X[k * P + off + i] = A[e] + (i == k ? damp : 0.0f);
    }
    __syncthreads();
    return tr;
}

// Unnormalised Walsh-Hadamard transform (Sylvester order) of every column's
// first D entries: x_r <- sum_r' (-1)^popcount(r & r') x_r'.
template <int D>
__device__ void fwht_columns(float *X, int tid)
{
    constexpr int P = WushLds<D>::kP;
    for (int h = 1; h < D; h <<= 1) {
        for (int e = tid; e < D * (D / 2); e += kWushThreads) {
            const int col = e / (D / 2), m = e % (D / 2);
            const int r0 = (m / h) * 2 * h + m % h, r1 = r0 + h;
            float *c = X + col * P;
            const float a = c[r0], b = c[r1];
            c[r0] = a + b;
            c[r1] = a - b;
        }
        __syncthreads();
    }
}

template <int D>
__global__ void __launch_bounds__(kWushThreads) wush_kernel(const float *m_all, const float *h_all, float gamma,
                                                   float *t_all, float *tinv_all, int32_t *sweeps_out)
{
    constexpr int P = WushLds<D>::kP;
    constexpr int kPairs = D / 2;
    constexpr int kTpp = kWushThreads / kPairs;  // threads per pair: 8 (d 128) or 16 (d 64)
    constexpr int kRows = D / kTpp;     // rows of each half per thread
    constexpr float kTol = 4.0f * (D == 128 ? 11.3137085f : 8.0f) * 5.9604645e-8f;
    __shared__ __attribute__((aligned(16))) float X[D * P];
    __shared__ float lam[D], scl[D];
    __shared__ int perm[D];
    __shared__ float red[kWushWaves];
    const int tid = threadIdx.x;
    const int64_t pair = blockIdx.x;
    const float *M = m_all + pair * D * D;
    const float *H = h_all + pair * D * D;
    float *T = t_all + pair * D * D;
    float *Ti = tinv_all != nullptr ? tinv_all + pair * D * D : nullptr;

    // ---- 1. Cholesky factors: L of H_d (rows D ..), R of M_d (rows 0 ..)
    (void)load_damped<D>(H, X, D, gamma, tid, red);
    bool ok = cholesky<D>(X, D, tid);
    const float trM = load_damped<D>(M, X, 0, gamma, tid, red);
    ok = cholesky<D>(X, 0, tid) && ok;
    if (!ok) {
        for (int e = tid; e < D * D; e += kWushThreads) {
            T[e] = NAN;
            if (Ti != nullptr) Ti[e] = NAN;
        }
        if (sweeps_out != nullptr && tid == 0) sweeps_out[pair] = -1;
        return;
    }

    // ---- 2. B = R^T L in 8 x 8 register tiles, then over R
    {
        constexpr int kT = D / 8;  // tiles per side
        float acc[8][8];
#pragma unroll
        for (int a = 0; a < 8; ++a)
#pragma unroll
            for (int b = 0; b < 8; ++b) acc[a][b] = 0.0f;
        const int tile = tid;  // D = 128: 256 tiles, D = 64: 64 tiles, one per thread
        const bool have = tile < kT * kT;
        const int ti = have ? tile / kT : 0, tj = have ? tile % kT : 0;
        if (have) {
            const int k0 = 8 * (ti > tj ? ti : tj);
            for (int k = k0; k < D; ++k) {
                float r[8], l[8];
#pragma unroll
                for (int a = 0; a < 8; ++a) {
                    const int i = 8 * ti + a, j = 8 * tj + a;
                    r[a] = k >= i ? X[i * P + k] : 0.0f;      // R[k][i]
                    l[a] = k >= j ? X[j * P + D + k] : 0.0f;  // L[k][j]
                }
#pragma unroll
                for (int a = 0; a < 8; ++a)
#pragma unroll
                    for (int b = 0; b < 8; ++b) acc[a][b] = fmaf(r[a], l[b], acc[a][b]);
            }
        }
        __syncthreads();
        if (have) {
#pragma unroll
            for (int a = 0; a < 8; ++a)
#pragma unroll
                for (int b = 0; b < 8; ++b) X[(8 * tj + b) * P + 8 * ti + a] = acc[a][b];  // B[i][j]
        }
        __syncthreads();
    }

    // ---- 3. one-sided Jacobi on the columns of [B; L]
    const int pm = tid / kTpp, part = tid % kTpp;
    int sweeps = 0;
    for (; sweeps < kWushMaxSweeps; ++sweeps) {
        int rotated = 0;
        for (int round = 0; round < D - 1; ++round) {
            // round-robin: position 0 stays, positions 1 .. D-1 turn by one
            // per round; pair m meets positions m and D - 1 - m
            auto at = [&](int pos) { return pos == 0 ? 0 : 1 + (pos - 1 + round) % (D - 1); };
            const int p = at(pm), q = at(D - 1 - pm);
            // this thread's rows of the two B halves stay in registers from
            // the dot products to the rotation: the 4-row pieces
            // 4 (kTpp k + part) .. + 3, one 16-byte access each
            float *cp = X + p * P, *cq = X + q * P;
            f32x4 xb[kRows / 4], yb[kRows / 4];
            float al = 0.0f, be = 0.0f, ga = 0.0f;
#pragma unroll
            for (int k = 0; k < kRows / 4; ++k) {
                const int r = 4 * (kTpp * k + part);
                xb[k] = *reinterpret_cast<const f32x4 *>(cp + r);
                yb[k] = *reinterpret_cast<const f32x4 *>(cq + r);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    al = fmaf(xb[k][i], xb[k][i], al);
                    be = fmaf(yb[k][i], yb[k][i], be);
                    ga = fmaf(xb[k][i], yb[k][i], ga);
                }
            }
            al = group_sum<kTpp>(al);
            be = group_sum<kTpp>(be);
            ga = group_sum<kTpp>(ga);
            // rotate while the columns' cosine exceeds what rounding leaves
            // behind (a few units of 2^-24 sqrt(d))
            if (fabsf(ga) > kTol * sqrtf(al * be) && ga != 0.0f) {
                const float zeta = (be - al) / (2.0f * ga);
                const float t = copysignf(1.0f, zeta) / (fabsf(zeta) + sqrtf(1.0f + zeta * zeta));
                const float cs = 1.0f / sqrtf(1.0f + t * t);
                const float sn = cs * t;
#pragma unroll
                for (int k = 0; k < kRows / 4; ++k) {
                    const int r = 4 * (kTpp * k + part);
                    f32x4 u, v;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        u[i] = fmaf(cs, xb[k][i], -sn * yb[k][i]);
                        v[i] = fmaf(sn, xb[k][i], cs * yb[k][i]);
                    }
                    *reinterpret_cast<f32x4 *>(cp + r) = u;
                    *reinterpret_cast<f32x4 *>(cq + r) = v;
                }
#pragma unroll
                for (int k = 0; k < kRows / 4; ++k) {
                    const int r = D + 4 * (kTpp * k + part);
                    const f32x4 x = *reinterpret_cast<const f32x4 *>(cp + r);
                    const f32x4 y = *reinterpret_cast<const f32x4 *>(cq + r);
                    f32x4 u, v;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        u[i] = fmaf(cs, x[i], -sn * y[i]);
                        v[i] = fmaf(sn, x[i], cs * y[i]);
                    }
                    *reinterpret_cast<f32x4 *>(cp + r) = u;
                    *reinterpret_cast<f32x4 *>(cq + r) = v;
                }
                rotated = 1;
            }
            __syncthreads();
        }
        if (!__syncthreads_or(rotated)) break;
    }

    // ---- 4. eigenvalues, their order, the eigenvector signs, c
    for (int k = tid; k < D; k += kWushThreads) {
        const float *ck = X + k * P;
        float s = 0.0f;
        for (int i = 0; i < D; ++i) s = fmaf(ck[i], ck[i], s);
        lam[k] = s;
        // sign of u_k: the largest-magnitude entry of L u_k made positive
        float best = -1.0f, v = 0.0f;
        for (int i = 0; i < D; ++i) {
            const float a = fabsf(ck[D + i]);
            if (a > best) {
                best = a;
                v = ck[D + i];
            }
        }
        scl[k] = v < 0.0f ? -1.0f : 1.0f;
    }
    // (every slot of perm holds a valid column even if non-finite norms
    // left ranks tied)
    for (int r = tid; r < D; r += kWushThreads) perm[r] = r;
    __syncthreads();
    for (int k = tid; k < D; k += kWushThreads) {
        int rank = 0;
        const float lk = lam[k];
        for (int j = 0; j < D; ++j) rank += (lam[j] < lk) || (lam[j] == lk && j < k);
        perm[rank] = k;
    }
    float rs = 0.0f;
    for (int k = tid; k < D; k += kWushThreads) rs += sqrtf(lam[k]);
    rs = group_sum<64>(rs);
    __syncthreads();
    if ((tid & 63) == 0) red[tid >> 6] = rs;
    __syncthreads();
    const float sum_sqrt = wave_total(red);
    const float c = sqrtf((1.0f + gamma) * trM) / sqrtf(sum_sqrt);
    const float had = 1.0f / sqrtf((float)D);

    // ---- 5a. T: column j of the B halves gets y_r[j] = s_k lam_k^(-1/4)
    // (L u_k)[j], k = perm[r]; the transform along r gives row r of Had Y
    for (int e = tid; e < D * D; e += kWushThreads) {
        const int j = e / D, r = e % D;
        const int k = perm[r];
        X[j * P + r] = scl[k] * powf(lam[k], -0.25f) * X[k * P + D + j];
    }
    __syncthreads();
    fwht_columns<D>(X, tid);
    for (int e = tid; e < D * D; e += kWushThreads) {
        const int i = e / D, j = e % D;  // row-major write, coalesced
        T[e] = (c * had) * X[j * P + i];
    }
    if (sweeps_out != nullptr && tid == 0) sweeps_out[pair] = sweeps;
    if (Ti == nullptr) return;
    __syncthreads();

    // ---- 5b. T^{-1} = c^-1 M_d (L U) Lam^(-3/4) Had: M_d into the B halves
    // (column j holds M_d[.][j]), Z = M_d W in 8 x 8 tiles, row i of Z into
    // column i, then the transform along each row
    const float damp = gamma * trM / (float)D;
    for (int e = tid; e < D * D; e += kWushThreads) {
        const int i = e / D, j = e % D;
        const float v = i >= j ? M[e] : M[j * D + i];  // the lower triangle, mirrored
        X[j * P + i] = v + (i == j ? damp : 0.0f);
    }
    __syncthreads();
    {
        constexpr int kT = D / 8;
        float acc[8][8];
#pragma unroll
        for (int a = 0; a < 8; ++a)
#pragma unroll
            for (int b = 0; b < 8; ++b) acc[a][b] = 0.0f;
        const int tile = tid;
        const bool have = tile < kT * kT;
        const int ti = have ? tile / kT : 0, tr = have ? tile % kT : 0;
        if (have) {
            int kr[8];
            float sc[8];
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                kr[b] = perm[8 * tr + b];
                sc[b] = scl[kr[b]] * powf(lam[kr[b]], -0.75f) / c;
            }
            for (int j = 0; j < D; ++j) {
                float mv[8], w[8];
#pragma unroll
                for (int a = 0; a < 8; ++a) mv[a] = X[j * P + 8 * ti + a];   // M_d[i][j]
#pragma unroll
                for (int b = 0; b < 8; ++b) w[b] = X[kr[b] * P + D + j];     // (L u_k)[j]
#pragma unroll
                for (int a = 0; a < 8; ++a)
#pragma unroll
                    for (int b = 0; b < 8; ++b) acc[a][b] = fmaf(mv[a], w[b], acc[a][b]);
            }
#pragma unroll
            for (int b = 0; b < 8; ++b)
#pragma unroll
                for (int a = 0; a < 8; ++a) acc[a][b] *= sc[b];
        }
        __syncthreads();
        if (have) {
#pragma unroll
            for (int a = 0; a < 8; ++a)
#pragma unroll
                for (int b = 0; b < 8; ++b) X[(8 * ti + a) * P + 8 * tr + b] = acc[a][b];  // Z[i][r]
        }
        __syncthreads();
    }
    fwht_columns<D>(X, tid);
    for (int e = tid; e < D * D; e += kWushThreads) {
        const int i = e / D, r = e % D;
        Ti[e] = had * X[i * P + r];
    }
}

}  // namespace wushkv

using namespace wushkv;

extern "C" int wushkv_wush_transform(const float *m, const float *h, int32_t count, int32_t d,
                                     float gamma, float *t_out, float *t_inv_out,
                                     int32_t *sweeps_out, wushkv_stream_t stream)
{
    if (count < 0 || !(gamma >= 0.0f) || gamma == INFINITY) return WUSHKV_EINVAL;
    if (d != 64 && d != 128) return WUSHKV_EUNSUPPORTED;
    if (count == 0) return WUSHKV_OK;
    if (!m || !h || !t_out) return WUSHKV_EINVAL;
    if (((uintptr_t)m | (uintptr_t)h | (uintptr_t)t_out | (uintptr_t)t_inv_out |
         (uintptr_t)sweeps_out) & 15u)
        return WUSHKV_EINVAL;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const dim3 grid((unsigned)count);
    if (d == 128)
        launch("wush_kernel", wush_kernel<128>, grid, dim3(kWushThreads), s, m, h, gamma, t_out, t_inv_out, sweeps_out);
    else
        launch("wush_kernel", wush_kernel<64>, grid, dim3(kWushThreads), s, m, h, gamma, t_out, t_inv_out, sweeps_out);
    if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
    return WUSHKV_OK;
}
