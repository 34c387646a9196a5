// plan_policy.h -- split-K partition policy for batched paged decode attention.
//
// Decode attention streams every cached K/V row of every request once
// (APEX Sec. 2.2 and Sec. 2.3: it is the memory-bandwidth-bound part of a
// decode step).  A batch is ragged: a few long requests and many short ones
// cannot fill 256 compute units one (request, kv-head) pair at a time, so the
// token range of a long request is cut into block-aligned ranges that run in
// parallel and are merged afterwards with a log-sum-exp combine.  The policy
// below is compiled for both the host (inspection, tests) and the device
// (the planner kernel), so that both see the same decisions.
//
//   units  = sum_b ceil(L_b / block_size) * Hkv       (one unit = one block of
//                                                       one kv-head: 8 KiB of K+V
//                                                       at d = 128, bs = 16)
//   chunk  = max(kMinChunkBlocks, ceil(units / target_items))   [blocks]
//   n_b    = 1 if blocks_b <= chunk, else ceil(blocks_b / chunk)
//   per_b  = ceil(blocks_b / n_b)  (balanced ranges, each <= chunk)
//
// so the number of work items sum_b n_b * Hkv never exceeds
// target_items + B * Hkv.  A forced split count n gives every request with
// L_b > 0 exactly n ranges of ceil(blocks_b / n) blocks (trailing ranges may
// be empty), which tests use to exercise the combine.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace apex {

constexpr int kHeadDim = 128;
constexpr int kBlockSize = 16;
constexpr int kMinChunkBlocks = 8;     // 2 blocks per wave of a 4-wave work group
constexpr int kDefaultItemsPerCu = 16;
constexpr int kMaxItemsPerCu = 256;

struct SplitPlan {
    int n;    // number of token ranges
    int per;  // blocks per range
};

__host__ __device__ inline int64_t blocks_of(int32_t len, int bs)
{
    return len > 0 ? ((int64_t)len + bs - 1) / bs : 0;
}

__host__ __device__ inline int64_t target_items(int num_cu, int items_per_cu)
{
    int ipc = items_per_cu > 0 ? items_per_cu : kDefaultItemsPerCu;
    if (ipc > kMaxItemsPerCu) ipc = kMaxItemsPerCu;
    return (int64_t)(num_cu > 0 ? num_cu : 1) * ipc;
}

__host__ __device__ inline int64_t chunk_blocks(int64_t units, int64_t target)
{
    int64_t c = (units + target - 1) / target;
    return c < kMinChunkBlocks ? kMinChunkBlocks : c;
}

__host__ __device__ inline SplitPlan split_request(int64_t blocks, int64_t chunk, int forced)
{
    SplitPlan s;
    if (blocks <= 0) {
        s.n = 1;
        s.per = 0;
        return s;
    }
    if (forced > 0) {
        s.n = forced;
    } else {
        s.n = blocks <= chunk ? 1 : (int)((blocks + chunk - 1) / chunk);
    }
    s.per = (int)((blocks + s.n - 1) / s.n);
    return s;
}

// Upper bound on work items (and on partial-result slots) for a call.
__host__ __device__ inline int64_t max_items(int B, int Hkv, int num_cu, int items_per_cu,
                                             int forced)
{
    if (forced > 0) return (int64_t)B * Hkv * forced;
    return target_items(num_cu, items_per_cu) + (int64_t)B * Hkv;
}

}  // namespace apex
