// kv_append.hip -- paged KV-cache append (include/apex_kv_append.h).
//
// Each new token owns Hkv rows of d fp16 values in K and in V; each row is
// moved by d / 8 lanes with one 16-byte load and one 16-byte store per lane
// per cache.  A pass of a 256-lane work group covers 256 / (d / 8)
// consecutive (token, kv-head) rows, so the reads of a wave are contiguous in
// the new-row buffer and every write is a whole 16-byte-aligned piece of one
// cache row; a work group makes four passes with all loads in flight before
// the stores.
// The slot check runs per row, so padding and out-of-pool slots cost a load
// of the slot and nothing else.
#include <hip/hip_runtime.h>

#include <limits.h>
#include <stdint.h>

#include "apex_kv_append.h"
#include "status.h"

namespace {

using apex::fail;

constexpr int kAppendThreads = 256;
constexpr int kMaxRowVecs = kAppendThreads;   // d <= 2048
constexpr int kRowsPerThread = 4;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kAppendThreads) void kv_append_kernel(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new, int64_t token_vecs,
    u32x4* __restrict__ k_cache, u32x4* __restrict__ v_cache, const int64_t* __restrict__ slots,
    int rows, int Hkv, int row_vecs, int rows_per_pass, int block_size, int64_t capacity)
{
    // a work group covers kRowsPerThread passes of rows_per_pass consecutive
    // rows; all loads of a thread are issued before its stores
    const int local_row = (int)threadIdx.x / row_vecs;
    const int c = (int)threadIdx.x - local_row * row_vecs;
    if (local_row >= rows_per_pass) return;
    const int64_t base = (int64_t)blockIdx.x * rows_per_pass * kRowsPerThread + local_row;
    u32x4 kv[kRowsPerThread], vv[kRowsPerThread];
    int64_t dst[kRowsPerThread];
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
        dst[i] = -1;
        const int64_t r64 = base + (int64_t)i * rows_per_pass;
        if (r64 >= rows) continue;
        const int r = (int)r64;
        const int t = r / Hkv;
        const int g = r - t * Hkv;
        const int64_t slot = slots[t];
        if (slot < 0 || slot >= capacity) continue;
        const int64_t block = slot / block_size;
        const int64_t pos = slot - block * block_size;
        dst[i] = ((block * Hkv + g) * block_size + pos) * row_vecs + c;
        const int64_t src = (int64_t)t * token_vecs + (int64_t)g * row_vecs + c;
        kv[i] = k_new[src];
        vv[i] = v_new[src];
    }
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
        if (dst[i] < 0) continue;
        k_cache[dst[i]] = kv[i];
        v_cache[dst[i]] = vv[i];
    }
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

}  // namespace

extern "C" int apex_kv_append(const void* k_new, const void* v_new, int64_t new_token_stride,
                              void* k_cache, void* v_cache, const int64_t* slot_mapping, int T,
                              int Hkv, int d, int block_size, int64_t num_blocks, void* stream)
{
    apex::clear_error();
    if (T < 0) return fail(APEX_ERR_INVALID_ARG, "T = %d is negative", T);
    if (Hkv <= 0 || block_size <= 0)
        return fail(APEX_ERR_INVALID_ARG, "Hkv = %d and block_size = %d must be positive", Hkv, block_size);
    if (num_blocks < 0) return fail(APEX_ERR_INVALID_ARG, "num_blocks is negative");
    if (d <= 0 || d % 8 != 0 || d / 8 > kMaxRowVecs)
        return fail(APEX_ERR_UNSUPPORTED, "head dim %d unsupported (a multiple of 8 up to %d)", d,
                    8 * kMaxRowVecs);
    const int64_t row_elems = (int64_t)Hkv * d;
    const int64_t stride = new_token_stride == 0 ? row_elems : new_token_stride;
    if (stride < row_elems || stride % 8 != 0)
        return fail(APEX_ERR_INVALID_ARG, "new_token_stride %lld must be 0 or a multiple of 8 >= Hkv * d",
                    (long long)new_token_stride);
    if ((int64_t)T * Hkv > INT_MAX) return fail(APEX_ERR_UNSUPPORTED, "T * Hkv exceeds 2^31 - 1");
    if (num_blocks > INT64_MAX / ((int64_t)Hkv * block_size * d * 2))
        return fail(APEX_ERR_INVALID_ARG, "cache size overflows");
    if (T == 0) return APEX_OK;
    if (!k_new || !v_new || !k_cache || !v_cache || !slot_mapping)
        return fail(APEX_ERR_INVALID_ARG, "a tensor pointer is NULL");
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16))
        return fail(APEX_ERR_INVALID_ARG, "k_new, v_new, k_cache and v_cache must be 16-byte aligned");
    if (!aligned(slot_mapping, 8)) return fail(APEX_ERR_INVALID_ARG, "slot_mapping must be 8-byte aligned");
    const size_t cache_bytes = (size_t)num_blocks * Hkv * block_size * d * 2;
    const size_t new_bytes = ((size_t)(T - 1) * stride + row_elems) * 2;
    if (overlaps(k_cache, cache_bytes, v_cache, cache_bytes))
        return fail(APEX_ERR_INVALID_ARG, "k_cache overlaps v_cache");
    const void* inputs[3] = {k_new, v_new, slot_mapping};
    const size_t input_bytes[3] = {new_bytes, new_bytes, (size_t)T * 8};
    for (int i = 0; i < 3; ++i)
        if (overlaps(inputs[i], input_bytes[i], k_cache, cache_bytes) ||
            overlaps(inputs[i], input_bytes[i], v_cache, cache_bytes))
            return fail(APEX_ERR_INVALID_ARG, "an input overlaps a cache");
    if (num_blocks == 0) return APEX_OK;   // every slot is out of the pool

    const int row_vecs = d / 8;
    const int rows_per_pass = kAppendThreads / row_vecs;
    const int rows = T * Hkv;
    const int64_t rows_per_group = (int64_t)rows_per_pass * kRowsPerThread;
    const unsigned groups = (unsigned)(((int64_t)rows + rows_per_group - 1) / rows_per_group);
    kv_append_kernel<<<groups, kAppendThreads, 0, (hipStream_t)stream>>>(
        (const u32x4*)k_new, (const u32x4*)v_new, stride / 8, (u32x4*)k_cache, (u32x4*)v_cache,
        slot_mapping, rows, Hkv, row_vecs, rows_per_pass, block_size, num_blocks * block_size);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(APEX_ERR_HIP, "kv_append launch failed: %s", hipGetErrorString(e));
    return APEX_OK;
}
