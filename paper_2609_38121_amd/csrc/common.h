// Device-side helpers shared by the WUSH-KV kernels (gfx950 only).
//
// Number formats, the packed-page index arithmetic documented in
// include/wushkv.h, and the launch/timing plumbing of the host library.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

#include "wushkv.h"

namespace wushkv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;

constexpr int kPage = WUSHKV_PAGE_TOKENS;  // tokens per page

// Bits of the page field that holds one code: 3-bit codes are stored in the
// 4-bit page format, each in a 4-bit field whose top bit is zero, so that
// every kernel reads them as 4-bit codes.
__host__ __device__ constexpr int storage_bits(int bits) { return bits == 3 ? 4 : bits; }

// ---------------------------------------------------------------- formats

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// Two fp32 -> packed bf16 pair (low half = a), round to nearest even
// (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16_rne(float a, float b)
{
    f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Two fp32 -> packed fp16 pair (low half = a), round to nearest even
// (v_cvt_pk_f16_f32).
__device__ __forceinline__ uint32_t pack_f16_rne(float a, float b)
{
    f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2));
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h)
{
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}

// fp32 -> fp16 bits, round to nearest even (v_cvt_f16_f32 under the default
// rounding mode); overflow gives infinity.
__device__ __forceinline__ uint32_t f32_to_f16_bits(float x)
{
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));
}

// ---------------------------------------------------------------- layout
// See the "Code words" section of include/wushkv.h.

template <int D, int BITS>
struct Layout {
    static constexpr int kCodesPerWord = 32 / BITS;            // B
    static constexpr int kOpsPerWord = kCodesPerWord / 8;      // B / 8
    static constexpr int kNw = D * BITS / 128;                 // V words per (lane, slice)
    static constexpr int kWordsPerLane = 4 * kNw;              // V words per lane
    static constexpr int kKLanes = D / 2;                      // lanes holding key codes
    static constexpr int kKWordsPerLane = 4 * BITS;            // key words per lane (4 tiles)
    static constexpr int kRegionBytes = 8 * D * BITS;          // one code region
    static constexpr int kParamOffset = 2 * kRegionBytes;
    static constexpr int kPageBytes = 2 * kRegionBytes + 8 * kPage;
    static constexpr int kChunks = D / 32;                     // 32-channel chunks
    static constexpr int kNTiles = D / 16;                     // PV N-tiles

    // Bit of value code (operand o, slot i) inside its word: slot i sits in
    // half word i % 2 at field v_field(o, i / 2) (see widen_word_f16).
    __host__ __device__ static constexpr int v_field(int o, int r)
    {
        return BITS == 2 ? (o == 0 ? (r == 0 ? 6 : r == 1 ? 10 : r == 2 ? 8 : 12)
                                   : (r == 0 ? 2 : r == 1 ? 0 : r == 2 ? 4 : 14))
                         : (r == 0 ? 4 : r == 1 ? 0 : r == 2 ? 8 : 12);
    }
    __host__ __device__ static constexpr int v_bit(int o, int i) { return 16 * (i & 1) + v_field(o, i >> 1); }

    // K region: (token t of the page, channel ch) -> (word index, bit).
    // Lane 16 j + n holds tokens 4 n .. 4 n + 3 (tile t % 4) and channels
    // 32 j .. 32 j + 31, BITS words per tile, 4 BITS words in all; its k-th
    // word is word 4 of 16-byte chunk k / 4, and chunk q holds every lane's
    // 16 bytes in lane order (one 128-bit LDS read per chunk touches
    // consecutive addresses).  Inside a word the channels split into two
    // halves of 16 / BITS codes; code i of half h sits at bit
    // 2 BITS i + BITS h, so that one mask (and one shift for h = 1) spreads
    // a word into nibbles (2-bit) or bytes (4-bit), one code each.
    __host__ __device__ static constexpr int k_word(int lane, int k) { return (k >> 2) * (4 * kKLanes) + 4 * lane + (k & 3); }
    __host__ __device__ static inline void k_pos(int t, int ch, int &word, int &bit)
    {
        constexpr int kSpan = 32 / BITS;  // channels per word
        const int n = t >> 2, tt = t & 3, j = ch >> 5, q = ch & 31;
        const int w = q / kSpan, r = q % kSpan, h = r / (kSpan / 2), i = r % (kSpan / 2);
        word = k_word(16 * j + n, BITS * tt + w);
        bit = 2 * BITS * i + BITS * h;
    }
    // V region: (token t of the page, channel ch) -> (word index, bit).
    // Lane 16 j + m's k-th word (k = kc 2nw + u) is word k % 4 of chunk
    // k / 4, chunks again holding every lane's 16 bytes in lane order.
    __host__ __device__ static constexpr int v_word(int lane, int k) { return (k >> 2) * 256 + 4 * lane + (k & 3); }
    __host__ __device__ static inline void v_pos(int t, int ch, int &word, int &bit)
    {
        int kc = t >> 5, j = (t >> 3) & 3, i = t & 7;
        int nt = ch >> 4, m = ch & 15;
        int u = nt / kOpsPerWord, o = nt % kOpsPerWord;
        word = v_word(16 * j + m, kc * 2 * kNw + u);
        bit = v_bit(o, i);
    }
};

// Widen the value codes of one word into fp16 operand registers: out[4 o +
// r] is register r (slots 2r, 2r+1, one per half word) of operand o, each
// code c in the fraction bits of an fp16 subnormal with exponent field zero:
// the value c 2^T 2^-24, where T is the code's target field.  No offset is
// added, so nothing has to be removed afterwards.  The matrix instruction
// multiplies subnormal inputs exactly, but aligns each product by its
// operands' exponent fields: a code far below the top of the fraction would
// lose that many bits when summed with other products, so every code is
// moved within two bits of the top, T = 6 or 8 (2-bit: registers 0-1 and
// 2-3; the other operand carries 2^-(T - 6)) or T = 4 (4-bit).  The page
// layout (Layout::v_field) puts the codes where four shifts and one mask per
// register (2-bit; three shifts for 4-bit) reach those targets.
template <int BITS>
__device__ __forceinline__ void widen_word_f16(uint32_t w, uint32_t *out)
{
    if constexpr (BITS == 2) {
        constexpr uint32_t m6 = 0x00C000C0u, m8 = 0x03000300u;
        const uint32_t l4 = w << 4, r4 = w >> 4, l6 = w << 6, r6 = w >> 6;
        out[0] = w & m6;   // field 6
        out[1] = r4 & m6;  // field 10
        out[2] = w & m8;   // field 8
        out[3] = r4 & m8;  // field 12
        out[4] = l4 & m6;  // field 2
        out[5] = l6 & m6;  // field 0
        out[6] = l4 & m8;  // field 4
        out[7] = r6 & m8;  // field 14
    } else {
        constexpr uint32_t m4 = 0x00F000F0u;
        out[0] = w & m4;          // field 4
        out[1] = (w << 4) & m4;   // field 0
        out[2] = (w >> 4) & m4;   // field 8
        out[3] = (w >> 8) & m4;   // field 12
    }
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f16x8 as_op_h(const uint32_t *u)
{
    u32x4 v = {u[0], u[1], u[2], u[3]};
    return __builtin_bit_cast(f16x8, v);
}

__device__ __forceinline__ f32x4 mfma16h(f16x8 a, f16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// k~ = T_K k (Alg. 2 step 3) for a tile of up to 16 key rows on the
// 16x16x32 bf16 matrix instruction.  Lane (j, n) of a wave supplies row n's
// channels 32 c + 8 j .. 32 c + 8 j + 7 (aop[c], c < D / 32) and, from
// load(), the T_K rows of output channels 16 (nt0 + nt) + n over the same
// channels (bop[nt][c]).  apply() accumulates the D / 32 chunks in chunk
// order from zero in fp32; row 4 j + r, output channel 16 (nt0 + nt) + n
// ends in acc[nt][r], and the caller rounds it once to bf16.  Each output
// element depends only on its own row and column, and every path that forms
// k~ (the prefill tiles, short appends and the fused decode step) goes
// through this with the key in the same operand positions, so a token's k~
// does not depend on the path that formed it.
template <int D, int NT>
struct KeyTile {
    static constexpr int kC = D / 32;
    bf16x8 bop[NT][kC];
    __device__ __forceinline__ void load(const uint16_t *tk, int h, int nt0, int lane)
    {
        const int j = lane >> 4, n = lane & 15;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const uint16_t *row = tk + ((int64_t)h * D + 16 * (nt0 + nt) + n) * D + 8 * j;
#pragma unroll
            for (int c = 0; c < kC; ++c) bop[nt][c] = *reinterpret_cast<const bf16x8 *>(row + 32 * c);
        }
    }
    __device__ __forceinline__ void apply(const bf16x8 (&aop)[kC], f32x4 (&acc)[NT]) const
    {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < kC; ++c)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) acc[nt] = mfma16(aop[c], bop[nt][c], acc[nt]);
    }
};

// floor(a / b) for b > 0.
__host__ __device__ __forceinline__ int64_t floor_div(int64_t a, int64_t b)
{
    int64_t q = a / b;
    if ((a % b != 0) && (a < 0)) q -= 1;
    return q;
}

// S_quant after the cache grew to s_new entries (Alg. 2, S_quant update).
__host__ __device__ __forceinline__ int32_t next_quant_end(int32_t s_new, int32_t s_quant,
                                                           int32_t s_sink, int32_t s_keep,
                                                           int32_t s_flush)
{
    int64_t start = s_quant > s_sink ? s_quant : s_sink;
    int64_t cand = start + floor_div((int64_t)s_new - s_keep - start, s_flush) * s_flush;
    return (int32_t)(cand > s_quant ? cand : s_quant);
}

// Ring slot of a recent-window position p >= s_sink.
__host__ __device__ __forceinline__ int32_t ring_slot(int32_t p, int32_t s_sink, int32_t ring)
{
    return s_sink + (p - s_sink) % ring;
}

// ------------------------------------------------------- host-side plumbing

// Launch bookkeeping for wushkv_timing_*; defined in api.hip.  While timing
// is on, each launch takes the next pair of events, which the runtime
// records at the start and the end of that kernel's execution.
struct TimedLaunch {
    hipEvent_t start = nullptr, stop = nullptr;
};
TimedLaunch timing_slot(const char *name);

template <typename Kernel, typename... Args>
inline void launch(const char *name, Kernel kernel, dim3 grid, dim3 block, hipStream_t s,
                   Args... args)
{
    const TimedLaunch t = timing_slot(name);
    if (t.start != nullptr)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, s, t.start, t.stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

}  // namespace wushkv
