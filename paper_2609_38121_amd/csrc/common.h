// Device-side helpers shared by the WUSH-KV kernels (gfx950 only).
//
// Number formats, the packed-page index arithmetic documented in
// include/wushkv.h, and the launch/timing plumbing of the host library.
#pragma once

#include <hip/hip_runtime.h>
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
constexpr uint32_t kBias2 = 0x43004300u;      // two bf16 128.0: 0x4300 | c == 128 + c
constexpr uint32_t kBiasF16x2 = 0x64006400u;  // two fp16 1024.0: 0x6400 | c == 1024 + c

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
    static constexpr int kNw = D * BITS / 128;                 // words per (lane, tile)
    static constexpr int kWordsPerLane = 4 * kNw;
    static constexpr int kRegionBytes = 8 * D * BITS;          // one code region
    static constexpr int kParamOffset = 2 * kRegionBytes;
    static constexpr int kPageBytes = 2 * kRegionBytes + 8 * kPage;
    static constexpr int kChunks = D / 32;                     // score K-chunks
    static constexpr int kNTiles = D / 16;                     // PV N-tiles

    // Bit offset of element e inside its word.
    __host__ __device__ static constexpr int elem_bit(int e) { return 16 * (e & 1) + BITS * (e >> 1); }

    // K region: (token t of the page, channel ch) -> (word index, bit).
    __host__ __device__ static inline void k_pos(int t, int ch, int &word, int &bit)
    {
        int tau = 2 * (t >> 5) + ((t >> 2) & 1);
        int m = 4 * ((t >> 3) & 3) + (t & 3);
        int c = ch >> 5, j = (ch >> 3) & 3, i = ch & 7;
        int w = c / kOpsPerWord, o = c % kOpsPerWord;
        word = (16 * j + m) * kWordsPerLane + tau * kNw + w;
        bit = elem_bit(8 * o + i);
    }
    // V region: (token t of the page, channel ch) -> (word index, bit).
    __host__ __device__ static inline void v_pos(int t, int ch, int &word, int &bit)
    {
        int kc = t >> 5, j = (t >> 3) & 3, i = t & 7;
        int nt = ch >> 4, m = ch & 15;
        int u = nt / kOpsPerWord, o = nt % kOpsPerWord;
        word = (16 * j + m) * kWordsPerLane + kc * 2 * kNw + u;
        bit = elem_bit(8 * o + i);
    }
};

// Widen the codes of one word into bf16 operand registers: out[e] holds
// elements 2e (low half) and 2e+1 (high half) as bf16 values 128 + c * 2^s.
// For 2-bit codes the shift s depends on the slot pair p = e % 4 as
// s = {0, 2, 4, 0}[p]; the other matrix operand carries 2^-s for those slots.
// 4-bit codes use s = 0.
//
// Each output is (word & mask) | bias, one v_and_or_b32.  That encoding
// takes no literal constants, so the masks and the bias arrive as kernel
// arguments (scalar registers) instead of compile-time constants, which
// keeps the compiler from splitting the operation in two.
struct WidenMasks {
    uint32_t m0, m1, m2;  // field masks (see the widen functions)
    uint32_t bias;        // two copies of the offset value's bit pattern
    uint32_t m3;
};

inline WidenMasks widen_masks(int bits)
{
    return bits == 2 ? WidenMasks{0x00030003u, 0x000C000Cu, 0x00300030u, kBias2, 0u}
                     : WidenMasks{0x000F000Fu, 0x000F000Fu, 0x000F000Fu, kBias2, 0u};
}

template <int BITS>
__device__ __forceinline__ void widen_word(uint32_t w, uint32_t *out, const WidenMasks &k);

template <>
__device__ __forceinline__ void widen_word<2>(uint32_t w, uint32_t *out, const WidenMasks &k)
{
    out[0] = (w & k.m0) | k.bias;
    out[1] = (w & k.m1) | k.bias;
    out[2] = (w & k.m2) | k.bias;
    const uint32_t t6 = w >> 6, t8 = w >> 8, t14 = w >> 14;
    out[3] = (t6 & k.m0) | k.bias;
    out[4] = (t8 & k.m0) | k.bias;
    out[5] = (t8 & k.m1) | k.bias;
    out[6] = (t8 & k.m2) | k.bias;
    out[7] = (t14 & k.m0) | k.bias;
}

template <>
__device__ __forceinline__ void widen_word<4>(uint32_t w, uint32_t *out, const WidenMasks &k)
{
    out[0] = (w & k.m0) | k.bias;
    out[1] = ((w >> 4) & k.m0) | k.bias;
    out[2] = ((w >> 8) & k.m0) | k.bias;
    out[3] = ((w >> 12) & k.m0) | k.bias;
}

// The same widening into fp16 operands, 1024 + c 2^s: fp16 keeps 10
// fraction bits, so 2-bit fields fit at s = 0, 2, 4, 6 and one shift by 8
// reaches the upper byte of each half word (s = 2p for slot pair p); 4-bit
// fields fit at s = 0 and 4 (s = 4 (p % 2)).
inline WidenMasks widen_masks_f16(int bits)
{
    return bits == 2 ? WidenMasks{0x00030003u, 0x000C000Cu, 0x00300030u, kBiasF16x2, 0x00C000C0u}
                     : WidenMasks{0x000F000Fu, 0x00F000F0u, 0x000F000Fu, kBiasF16x2, 0x00F000F0u};
}

template <int BITS>
__device__ __forceinline__ void widen_word_f16(uint32_t w, uint32_t *out, const WidenMasks &k);

template <>
__device__ __forceinline__ void widen_word_f16<2>(uint32_t w, uint32_t *out, const WidenMasks &k)
{
    out[0] = (w & k.m0) | k.bias;
    out[1] = (w & k.m1) | k.bias;
    out[2] = (w & k.m2) | k.bias;
    out[3] = (w & k.m3) | k.bias;
    const uint32_t t8 = w >> 8;
    out[4] = (t8 & k.m0) | k.bias;
    out[5] = (t8 & k.m1) | k.bias;
    out[6] = (t8 & k.m2) | k.bias;
    out[7] = (t8 & k.m3) | k.bias;
}

template <>
__device__ __forceinline__ void widen_word_f16<4>(uint32_t w, uint32_t *out, const WidenMasks &k)
{
    out[0] = (w & k.m0) | k.bias;
    out[1] = (w & k.m1) | k.bias;
    const uint32_t t8 = w >> 8;
    out[2] = (t8 & k.m0) | k.bias;
    out[3] = (t8 & k.m1) | k.bias;
}

// 2^-s of operand slot i for the fp16 widening above.
template <int BITS>
__host__ __device__ constexpr float slot_scale_f16(int i)
{
    return BITS == 2 ? (i >> 1) == 0 ? 1.0f : (i >> 1) == 1 ? 0.25f : (i >> 1) == 2 ? 0.0625f : 0.015625f
                     : ((i >> 1) & 1) ? 0.0625f : 1.0f;
}

// 2^-s of operand slot i (0..7) for the widened codes above.
template <int BITS>
__host__ __device__ constexpr float slot_scale(int i)
{
    return BITS == 2 ? ((i >> 1) == 1 ? 0.25f : ((i >> 1) == 2 ? 0.0625f : 1.0f)) : 1.0f;
}

__device__ __forceinline__ bf16x8 as_op(const uint32_t *u)
{
    u32x4 v = {u[0], u[1], u[2], u[3]};
    return __builtin_bit_cast(bf16x8, v);
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

// Launch bookkeeping for wushkv_timing_*; defined in api.hip.
void timing_begin(const char *name, hipStream_t s);
void timing_end(hipStream_t s);

}  // namespace wushkv
