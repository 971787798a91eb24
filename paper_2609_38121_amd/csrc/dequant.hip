// wushkv_dequant: reconstruct stored entries x = scale * code + zero
// (Eq. (7), last term) straight from the packed pages.  One thread per
// (position, four consecutive channels), written as one 16-byte store per
// output; reads the page layout of include/wushkv.h.
#include "common.h"

namespace wushkv {

template <int D, int BITS>
__global__ void __launch_bounds__(256) dequant_kernel(const uint8_t *pages, const int32_t *page_table,
                                                      int32_t n_kv, int32_t s_sink, int32_t max_pages,
                                                      int32_t n_pages, int32_t b, int32_t start,
                                                      int32_t count, float *k_out, float *v_out)
{
    using L = Layout<D, BITS>;
    constexpr int kQuads = D / 4;  // threads per position
    // four consecutive channels from a multiple of 4 share one key word:
    // a word spans 32 / BITS >= 8 channels, aligned to its span
    static_assert(32 / BITS >= 8, "four key channels per word");
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int h = blockIdx.y;
    if (idx >= (int64_t)count * kQuads) return;
    const int32_t pos = start + (int32_t)(idx / kQuads);
    const int ch0 = 4 * (int)(idx % kQuads);
    const int32_t rel = pos - s_sink;
    const int32_t lp = rel / kPage, t = rel % kPage;
    const int32_t phys = lp < max_pages ? page_table[(int64_t)b * max_pages + lp] : -1;
    const int64_t o = ((int64_t)h * count + (pos - start)) * D + ch0;
    if (phys < 0 || phys >= n_pages) {
        const float4 nan4 = make_float4(NAN, NAN, NAN, NAN);
        if (k_out) *reinterpret_cast<float4 *>(k_out + o) = nan4;
        if (v_out) *reinterpret_cast<float4 *>(v_out + o) = nan4;
        return;
    }
    const uint8_t *pg = pages + ((int64_t)phys * n_kv + h) * L::kPageBytes;
    const uint32_t *w = reinterpret_cast<const uint32_t *>(pg);
    const uint32_t *pk = reinterpret_cast<const uint32_t *>(pg + L::kParamOffset);
    const uint32_t mask = (1u << BITS) - 1u;
    if (k_out) {
        int word, bit;
        L::k_pos(t, ch0, word, bit);
        const uint32_t kw = w[word];
        const uint32_t prm = pk[t];
        const float sc = f16_bits_to_f32(prm & 0xFFFFu), zr = f16_bits_to_f32(prm >> 16);
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            int we, be;
            L::k_pos(t, ch0 + e, we, be);
            r[e] = fmaf(sc, (float)((kw >> be) & mask), zr);
        }
        *reinterpret_cast<float4 *>(k_out + o) = make_float4(r[0], r[1], r[2], r[3]);
    }
    if (v_out) {
        const uint32_t prm = pk[kPage + t];
        const float sc = f16_bits_to_f32(prm & 0xFFFFu), zr = f16_bits_to_f32(prm >> 16);
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            int we, be;
            L::v_pos(t, ch0 + e, we, be);
            r[e] = fmaf(sc, (float)((w[L::kRegionBytes / 4 + we] >> be) & mask), zr);
        }
        *reinterpret_cast<float4 *>(v_out + o) = make_float4(r[0], r[1], r[2], r[3]);
    }
}

}  // namespace wushkv

using namespace wushkv;

int wushkv_validate_cache(const wushkv_cache *c);  // api.hip

extern "C" int wushkv_dequant(const wushkv_cache *c, int32_t b, int32_t start, int32_t count,
                              float *k_out, float *v_out, wushkv_stream_t stream)
{
    int st = wushkv_validate_cache(c);
    if (st != WUSHKV_OK) return st;
    if (b < 0 || b >= c->batch || count < 0 || start < c->s_sink) return WUSHKV_EINVAL;
    if ((int64_t)start + count > (int64_t)c->s_sink + (int64_t)kPage * c->max_pages_per_seq)
        return WUSHKV_EINVAL;
    if (count == 0 || (!k_out && !v_out)) return WUSHKV_OK;
    if (((uintptr_t)k_out | (uintptr_t)v_out) & 15u) return WUSHKV_EINVAL;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t n = (int64_t)count * (c->head_dim / 4);
    if ((n + 255) / 256 > 0x7FFFFFFF) return WUSHKV_EINVAL;
    dim3 grid((unsigned)((n + 255) / 256), (unsigned)c->n_kv_heads);
    const int key = c->head_dim * 10 + storage_bits(c->bits);
#define WUSHKV_DQ(D_, B_)                                                                     \
    launch("dequant_kernel", dequant_kernel<D_, B_>, grid, dim3(256), s, c->pages, c->page_table, \
           c->n_kv_heads, c->s_sink, c->max_pages_per_seq, c->n_pages, b, start, count, k_out,   \
           v_out)
    switch (key) {
        case 1282: WUSHKV_DQ(128, 2); break;
        case 1284: WUSHKV_DQ(128, 4); break;
        case 642: WUSHKV_DQ(64, 2); break;
        case 644: WUSHKV_DQ(64, 4); break;
    }
#undef WUSHKV_DQ
    if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
    return WUSHKV_OK;
}
