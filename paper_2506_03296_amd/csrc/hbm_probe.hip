// hbm_probe.hip -- HBM read-bandwidth probes (include/apex_hbm_probe.h).
#include <hip/hip_runtime.h>

#include "apex_hbm_probe.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void stream_kernel(const u32x4* __restrict__ p, size_t n16,
                                                     uint32_t* sink)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 a = p[i], b = p[i + stride], c = p[i + 2 * stride], d = p[i + 3 * stride];
        acc ^= a ^ b ^ c ^ d;
    }
    for (; i < n16; i += stride) acc ^= p[i];
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) *sink = 1u;
}

__global__ __launch_bounds__(256) void gather_kernel(const u32x4* __restrict__ p,
                                                     const int32_t* __restrict__ ids,
                                                     int64_t n_chunks, uint32_t* sink)
{
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
    int64_t w = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (; w + waves < n_chunks; w += 2 * waves) {
        const u32x4* c0 = p + (size_t)ids[w] * 256 + lane;
        const u32x4* c1 = p + (size_t)ids[w + waves] * 256 + lane;
        const u32x4 a0 = c0[0], a1 = c0[64], a2 = c0[128], a3 = c0[192];
        const u32x4 b0 = c1[0], b1 = c1[64], b2 = c1[128], b3 = c1[192];
        acc ^= a0 ^ a1 ^ a2 ^ a3 ^ b0 ^ b1 ^ b2 ^ b3;
    }
    for (; w < n_chunks; w += waves) {
        const u32x4* c0 = p + (size_t)ids[w] * 256 + lane;
        acc ^= c0[0] ^ c0[64] ^ c0[128] ^ c0[192];
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) *sink = 1u;
}

int default_blocks(int blocks)
{
    if (blocks > 0) return blocks;
    int dev = 0, cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return -1;
    return cu * 8;
}

}  // namespace

extern "C" {

int apex_hbm_probe_stream(const void* buf, size_t bytes, int blocks, uint32_t* sink, void* stream)
{
    if (!buf || !sink || bytes % 16 || blocks < 0) return -1;
    blocks = default_blocks(blocks);
    if (blocks <= 0) return -4;
    stream_kernel<<<blocks, 256, 0, (hipStream_t)stream>>>((const u32x4*)buf, bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

int apex_hbm_probe_gather(const void* buf, const int32_t* chunk_ids, int64_t n_chunks, int blocks,
                          uint32_t* sink, void* stream)
{
    if (!buf || !chunk_ids || !sink || n_chunks < 0 || blocks < 0) return -1;
    if (n_chunks == 0) return 0;
    blocks = default_blocks(blocks);
    if (blocks <= 0) return -4;
    gather_kernel<<<blocks, 256, 0, (hipStream_t)stream>>>((const u32x4*)buf, chunk_ids, n_chunks,
                                                          sink);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
