// plan_policy.h -- work partition of batched paged decode attention.
//
// Decode attention streams every cached K/V row of every request once (APEX
// Sec. 2.2 and Sec. 2.3: it is the memory-bandwidth-bound part of a decode
// step).  A batch is ragged -- a few long requests next to many short ones --
// so the work is cut by amount, not by request.  One unit is one block of one
// kv-head (16 tokens: 4 KiB of K plus 4 KiB of V at d = 128); the units are
// laid out in (request b, kv-head g, block) order.  Besides its units, a
// worker pays a fixed cost for every (request, kv-head) pair it attends --
// the block-id and first-tile latency, the merge and the emit -- so each
// non-empty pair is charged K = kSegmentCostUnits extra positions: on a line
// of V = U + K P positions (P pairs) every pair has its K cost positions
// followed by its blocks, and worker w of W takes the positions
// [floor(w V / W), floor((w + 1) V / W)).  The blocks among them form a
// contiguous range of units, so every worker walks consecutive units as
// before, and a run of short pairs no longer lands on one worker.  A
// (request, kv-head) pair whose units straddle workers is finished by a
// log-sum-exp combine of the workers' partial results.  Each worker has at
// most two partial segments (its first and its last), which fixes where
// they are stored.  Forced grids (tests) take K = 0: equal units.
//
// These functions are compiled for both the host (inspection, tests) and the
// device (every worker runs them on its own), so both see the same partition.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace apex {

constexpr int kHeadDim = 128;
constexpr int kBlockSize = 16;
constexpr int kMinUnitsPerWorker = 16;  // four blocks per wave of a 4-wave work group
constexpr int64_t kUnitsPerCuForOne = 1024;   // 8 MiB of K/V per CU
// Cost of a pair's segment in units: a short segment takes about 2-3 us of
// latency (block ids, first tiles, merge, emit), the time a work group
// streams about eight blocks in.
constexpr int kSegmentCostUnits = 8;

// floor(a / b) for a >= 0, b > 0.  A 64-bit division is a long software
// sequence on the GPU; the partition's operands nearly always fit in 32 bits,
// where the hardware-assisted 32-bit sequence gives the same quotient.  The
// 64-bit one is kept out of line, so that the code a work group runs before
// its first load stays short.
__host__ __device__ __attribute__((noinline)) inline int64_t div_floor_wide(int64_t a, int64_t b)
{
    return a / b;
}

__host__ __device__ inline int64_t div_floor(int64_t a, int64_t b)
{
    if (__builtin_expect(((uint64_t)a | (uint64_t)b) <= 0xffffffffull, 1))
        return (int64_t)((uint32_t)a / (uint32_t)b);
    return div_floor_wide(a, b);
}

__host__ __device__ inline uint32_t div_floor(uint32_t a, uint32_t b) { return a / b; }

__host__ __device__ inline int64_t blocks_of(int32_t len, int bs)
{
    return len > 0 ? ((int64_t)len + bs - 1) / bs : 0;
}

// Workers that get units: at most the launched ones; enough that each has
// about min_units units, but never fewer than the non-empty (request,
// kv-head) pairs -- a small batch would otherwise queue several short pairs
// on one work group, one after another, while most of the device idles.
// With cus > 0 (the device's compute units), a batch of at most one pair per
// CU and at most kUnitsPerCuForOne units per CU uses only the first `cus`
// work groups: one per CU (work groups are handed out round-robin over the
// XCDs and then over their CUs), no pair split between two groups, and no
// second group sharing the CU.
// The integer type I is int64_t, or uint32_t where the caller has shown that
// every operand and cus * kUnitsPerCuForOne fit (the kernel's 32-bit path).
template <typename I>
__host__ __device__ inline I active_workers_t(I units, I launched, I min_units, I pairs, I cus)
{
    if (cus > 0 && pairs <= cus && units <= cus * (I)kUnitsPerCuForOne && launched > cus) launched = cus;
    I w = div_floor(units, min_units > 0 ? min_units : (I)1);
    if (w < pairs) w = pairs;
    if (w < 1) w = 1;
    return w < launched ? w : launched;
}

__host__ __device__ inline int64_t active_workers(int64_t units, int64_t launched, int min_units,
                                                  int64_t pairs, int64_t cus)
{
    return active_workers_t<int64_t>(units, launched, min_units, pairs, cus);
}

// First position of worker w on the cost line of `positions` positions (the
// range of w is [worker_start(w), worker_start(w+1))).
__host__ __device__ inline int64_t worker_start(int64_t w, int64_t positions, int64_t workers)
{
    return div_floor(w * positions, workers);
}

// The worker whose range holds position v (0 <= v < positions).
__host__ __device__ inline int64_t worker_of(int64_t v, int64_t positions, int64_t workers)
{
    return div_floor((v + 1) * workers - 1, positions);
}

// Position of the first block of the pair with index `pair` (in (request,
// kv-head) order over the non-empty pairs) whose units start at unit p0:
// every pair up to and including it adds its K cost positions.
__host__ __device__ inline int64_t first_block_position(int64_t p0, int64_t pair, int64_t K)
{
    return p0 + K * (pair + 1);
}

// Partial slot that worker w uses for a split pair whose first contributor
// is wf: the first contributor holds the pair's start and runs past its
// range, so the pair is its last segment (slot 2w + 1); every later one
// starts inside the pair, so the pair is its first segment (slot 2w).
__host__ __device__ inline int64_t partial_slot(int64_t w, int64_t wf)
{
    return w == wf ? 2 * w + 1 : 2 * w;
}

}  // namespace apex
