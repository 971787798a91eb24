// wushkv_read_probe: a plain streaming read of a device buffer, the
// reference against which the hot path's bandwidth is read (how much of the
// nominal HBM peak a kernel that only reads can reach on this device).
//
// Each workgroup (256 threads) reads one 64 KB block, in one of two ways:
//   mode 0  16-byte vector loads into registers, 16 per thread, consecutive
//           threads on consecutive 16-byte chunks;
//   mode 1  16-byte direct-to-LDS loads (global_load_lds_dwordx4), 1 KB per
//           wave instruction, into a four-slot ring per wave: the path the
//           decode kernel's pages take.
// Every loaded word feeds an XOR written once per workgroup, so no load can
// be dropped.
#include "common.h"

namespace wushkv {

constexpr int kProbeBlock = 65536;  // bytes per workgroup

__device__ __forceinline__ void probe_dma16(const void *src, uint32_t lds_base)
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

__global__ void __launch_bounds__(256) read_probe_vgpr_kernel(const uint8_t *buf, uint32_t *sink)
{
    const uint8_t *blk = buf + (int64_t)blockIdx.x * kProbeBlock;
    u32x4 v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
        v[i] = *reinterpret_cast<const u32x4 *>(blk + 4096 * i + 16 * threadIdx.x);
    uint32_t x = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) x ^= v[i][0] ^ v[i][1] ^ v[i][2] ^ v[i][3];
    __shared__ uint32_t red[256];
    red[threadIdx.x] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = 0;
        for (int i = 0; i < 256; ++i) r ^= red[i];
        sink[blockIdx.x] = r;
    }
}

__global__ void __launch_bounds__(256) read_probe_lds_kernel(const uint8_t *buf, uint32_t *sink)
{
    __shared__ __attribute__((aligned(16))) uint8_t ring[4][4][1024];  // [wave][slot][1 KB]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // wave w reads chunks w, w + 4, .. of the block's 64 chunks of 1 KB
    const uint8_t *src = buf + (int64_t)blockIdx.x * kProbeBlock + 1024 * wave + 16 * lane;
    const uint32_t base = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(void __attribute__((address_space(3))) *)&ring[wave][0][0]);
    uint32_t x = 0;
    // four in flight: issue chunks 0..3, then per chunk: wait for the oldest,
    // read it, refill its slot
    for (int c = 0; c < 4; ++c) probe_dma16(src + 4096 * c, base + 1024 * c);
    for (int c = 0; c < 16; ++c) {
        if (c <= 12) asm volatile("s_waitcnt vmcnt(3)" ::: "memory");
        else if (c == 13) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
        else if (c == 14) asm volatile("s_waitcnt vmcnt(1)" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        const u32x4 v = *reinterpret_cast<const u32x4 *>(&ring[wave][c & 3][16 * lane]);
        x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (c + 4 < 16) probe_dma16(src + 4096 * (c + 4), base + 1024 * (c & 3));
    }
    __shared__ uint32_t red[256];
    red[threadIdx.x] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = 0;
        for (int i = 0; i < 256; ++i) r ^= red[i];
        sink[blockIdx.x] = r;
    }
}

}  // namespace wushkv

using namespace wushkv;

extern "C" int wushkv_read_probe(const void *buf, size_t bytes, int32_t mode, uint32_t *sink,
                                 wushkv_stream_t stream)
{
    if (!buf || !sink || (bytes % kProbeBlock) != 0 || bytes == 0) return WUSHKV_EINVAL;
    if (((uintptr_t)buf | (uintptr_t)sink) & 15u) return WUSHKV_EINVAL;
    if (mode != 0 && mode != 1) return WUSHKV_EINVAL;
    const size_t blocks = bytes / kProbeBlock;
    if (blocks > 0x7FFFFFFF) return WUSHKV_EINVAL;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (mode == 0)
        launch("read_probe_vgpr_kernel", read_probe_vgpr_kernel, dim3((unsigned)blocks), dim3(256), s,
               (const uint8_t *)buf, sink);
    else
        launch("read_probe_lds_kernel", read_probe_lds_kernel, dim3((unsigned)blocks), dim3(256), s,
               (const uint8_t *)buf, sink);
    if (hipGetLastError() != hipSuccess) return WUSHKV_ELAUNCH;
    return WUSHKV_OK;
}
