// kernels.h -- gfx950 kernel of batched paged decode attention.
//
// One call = one launch of attn_kernel<G, kCheck, kAppend> on a persistent
// grid of W work groups (4 waves each); kCheck adds the optional input check
// (block ids against the pool, contexts against an explicit table row),
// kAppend the fused append of the current token's K/V.  Every work
// group
//   1. reads context_lens once and derives the partition of plan_policy.h on
//      its own (block sums, a prefix scan, the longest request for the tight
//      block-table stride; 32-bit arithmetic unless the batch is too large
//      for it), so no planner kernel runs before it;
//   2. walks its contiguous range of (request b, kv-head g, block) units
//      (ranges of equal cost, a pair's cost being its blocks plus a fixed
//      start-up charge) segment by segment.  In a segment the four waves
//      take the blocks of one (b, g) pair round-robin; per 16-token block a
//      wave gathers the paged K/V rows with 128-bit loads (two blocks in
//      flight per wave), computes the G q-heads' scores as S^T = K Q^T with
//      four 16x16x32 fp16 MFMAs (q-heads padded to 16 columns), runs an
//      online softmax (running max and sum in base 2, log2(e) folded into
//      the scale), and accumulates O^T += V^T P^T in fp32 with sixteen
//      16x16x16 fp16 MFMAs -- the weights P as two fp16 parts, 22 bits --
//      V^T being assembled in registers with byte permutes.
//      Each wave's K/V pipeline runs on across segments: between two long
//      segments the last steps of one already load the next one's first
//      blocks, and the next segment's Q operand is loaded one segment ahead;
//   3. merges the waves' states in LDS and either writes the fp16 output rows
//      (the segment is the whole pair) or stores an fp32 partial
//      (accumulator, max, sum) and bumps the pair's arrival counter; the last
//      work group to arrive combines the pair's partials and writes the rows;
//   4. writes the zero rows of requests with no context (their share of them).
//
// The attention is the standard softmax attention that APEX runs for its
// GPU-resident decode requests over their paged KV (Sec. 3.1, Sec. 3.3,
// Sec. 4.1); splitting a pair's tokens is exact up to rounding: with per-range
// maxima m_s, sums l_s and unnormalised accumulators a_s,
//   out = sum_s 2^(m_s - M) a_s / sum_s 2^(m_s - M) l_s,   M = max_s m_s.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan_policy.h"

namespace apex {

typedef _Float16 f16;
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kAttnThreads = 256;
constexpr int kWaves = kAttnThreads / 64;
constexpr int kCachedLens = 2048;   // context_lens kept in LDS up to this batch size
constexpr int kCombineChunk = 8;    // partials loaded at once by the combining work group

struct AttnParams {
    const f16* q;          // [B][Hq][D]
    const f16* k;          // [NB][Hkv][BS][D]
    const f16* v;
    f16* out;              // [B][Hq][D]
    float* lse;            // optional [B][Hq], natural log
    int32_t* counters;     // [B][Hkv] arrival counters, zero between calls
    float* pacc;           // [2W][G][D] partial accumulators
    float* pml;            // [2W][G][2] partial (max in log2 units, sum)
    int64_t bt_stride;     // 0 = tight: ceil(max L / BS)
    float scale_log2;      // scale * log2(e)
    int B;
    int Hq;
    int Hkv;
    int min_units;         // minimum units per active worker
    int seg_cost;          // cost positions charged per pair (plan_policy.h), 0 = equal units
    int cus;               // compute units for the one-group-per-CU rule (0 = off)
    int launched;          // work groups launched (the grid size)
    int64_t num_blocks;    // physical blocks in the caches (input check only)
    unsigned* error_word;  // input-check error bits (input check only)
    // Fused append (optional): the current token's K/V rows, [B][Hkv][D] with
    // new_stride elements between tokens.  The caches then hold the first
    // L - 1 tokens of a request; the current one is attended from these rows
    // and written to its slot (position L - 1) by the work group that emits
    // the pair.
    const f16* k_new;
    const f16* v_new;
    int64_t new_stride;
    f16* k_store;          // the caches, written by the fused append
    f16* v_store;
#ifdef APEX_TRACE_WORK_GROUPS
    uint64_t* trace;       // [trace_groups][kTraceWords] work-group timeline, or null
    int64_t trace_groups;
#endif
};

#ifdef APEX_TRACE_WORK_GROUPS
// Work-group timeline of the diagnostic build: per work group, in ticks of
// the 100 MHz real-time clock, its first instruction, the end of its
// partition prologue, the completion of wave 0's first tiles and its end;
// then its segments, the split ones among them, and its units.
constexpr int kTraceWords = 8;
__device__ inline uint64_t trace_clock() { return __builtin_amdgcn_s_memrealtime(); }
// the work group's row, kept in LDS while it runs (no register stays live
// across the block loop for it)
__shared__ uint64_t s_trace[kTraceWords];
#endif

// Input-check error bits (apex_decode.h: APEX_DEVICE_ERR_*).
constexpr unsigned kErrBlockId = 1u;      // a block id outside [0, num_blocks)
constexpr unsigned kErrTableRow = 2u;     // a context past its block-table row

__device__ inline void report_error(const AttnParams& p, unsigned bits)
{
    __hip_atomic_fetch_or(p.error_word, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Reinterpret one 32-bit word as two fp16 values.  Taken by value on purpose:
// clang's __builtin_bit_cast applied directly to a vector element expression
// (e.g. v.y) reads element 0 instead (seen in the gfx950 assembly).
__device__ inline f16x2 as_h2(unsigned int u)
{
    return __builtin_bit_cast(f16x2, u);
}

__device__ inline float wave_shfl_xor(float x, int mask)
{
    return __shfl_xor(x, mask, 64);
}

__device__ inline float exp2_fast(float x)
{
    return __builtin_amdgcn_exp2f(x);
}

// Inclusive prefix sum / max over the 64 lanes of a wave with DPP (row
// shifts within each 16-lane row, then the row broadcasts of lanes 15 and 31
// into the rows above): a few VALU cycles per step, where a cross-lane
// shuffle goes through the LDS crossbar.  Lane 63 ends with the wave's total.
__device__ inline int wave_incl_sum(int x)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15, rows 1, 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31, rows 2, 3
    return x;
}

// As wave_incl_sum for fp32 values (lane 63 ends with the wave's sum).
__device__ inline float wave_incl_sum_f32(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x111, 0xf, 0xf, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x112, 0xf, 0xf, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x114, 0xf, 0xf, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x118, 0xf, 0xf, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xa, 0xf, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xc, 0xf, false));
    return x;
}

// As wave_incl_sum with max, for x >= 0.
__device__ inline int wave_incl_max(int x)
{
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false));
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false));
    return x;
}

// Max / sum of the values a lane's column holds in the four 16-lane rows of
// its wave (the rows' lanes l, l + 16, l + 32, l + 48), with the gfx950 row
// swaps: each swap returns the lane's own value and its partner's (rows
// paired as 0-1, 2-3, then halves as 0-32), so the pair's max / sum is the
// step of a xor-16 / xor-32 butterfly without the LDS crossbar of a shuffle.
__device__ inline float rows_max4(float x)
{
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ inline float rows_sum4(float x)
{
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ inline int uniform(int x)
{
    return __builtin_amdgcn_readfirstlane(x);
}

__device__ inline int64_t uniform64(int64_t x)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <typename T>
__device__ inline T* uniform_ptr(T* p)
{
    return (T*)uniform64((int64_t)p);
}

// Device-scope coherent accesses (relaxed atomics at agent scope).  On gfx950
// they carry the sc1 cache-coherence bit, so work groups on different XCDs
// (each with its own L2) see each other's values without any cache flush.
__device__ inline void store_coherent(float* p, float v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline float load_coherent(const float* p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Two fp16 halves from two words: the low (sel = kLoHalves) or high
// (sel = kHiHalves) half of a in the low half of the result, the same half of
// b in the high half.
constexpr unsigned kLoHalves = 0x05040100u;
constexpr unsigned kHiHalves = 0x07060302u;
__device__ inline unsigned pack_halves(unsigned a, unsigned b, unsigned sel)
{
    return __builtin_amdgcn_perm(b, a, sel);
}

// One (block, kv-head) slab of K or V: 16 rows of 128 fp16 values.
constexpr int kSlabBytes = kBlockSize * kHeadDim * 2;
// Buffer-resource word 3 for raw (untyped) buffer access on gfx9-family GPUs.
constexpr int kRawBufferWord3 = 0x00020000;
// Cache policy of the K/V loads: non-temporal (bit 1) -- each row is read
// exactly once per call, so it should not displace reusable lines.
constexpr int kStreamingLoad = 2;

// Operand layouts of one slab (lane = 16 q + c, q = lane / 16, c = lane % 16):
//   K: word i of lane (c, q) = token c, dims [32i + 8q, +8)   (A of S^T = K Q^T)
//   V: word e of lane (c, q) = token 4q + e, dims [8c, 8c + 8)
__device__ inline int k_lane_offset(int lane) { return (lane & 15) * 256 + (lane >> 4) * 16; }
__device__ inline int v_lane_offset(int lane) { return (lane >> 4) * 1024 + (lane & 15) * 16; }

// Loads a slab with buffer instructions: the slab base lives in scalar
// registers (a fresh resource per block), the lane offset in a VGPR that
// never changes.  The resource's extent bounds every access; an extent of 0
// turns the four loads into no-ops that return zeros, which lets a pipeline
// issue the same loads every step.
__device__ inline void load_slab(u32x4 (&w)[4], const f16* slab, int bytes, int lane_off,
                                 int stride)
{
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc((void*)uniform_ptr(slab), (short)0, bytes, kRawBufferWord3);
#pragma unroll
    for (int i = 0; i < 4; ++i)
        w[i] = __builtin_amdgcn_raw_buffer_load_b128(r, lane_off + stride * i, 0, kStreamingLoad);
}

// This wave's share of one segment (blocks lo..hi-1 of pair (b, g)): its
// blocks are first, first + 4, ... < hi, n of them.  A wave with no block in
// the segment, and the "next segment" after a work group's last one, have
// n = 0.
struct WaveSeg {
    const int32_t* bt;   // block-table entry of the wave's first block
    const f16* kpair;    // K / V of kv-head g in block 0 (a block id adds id * step)
    const f16* vpair;
    const f16* qrow;     // this lane's Q^T operand row (q-head g*G + lane % 16, if < G)
    int first;           // the wave's first block (index into the pair's blocks)
    int n;
    int b, g;            // the pair
};

template <int G>
__device__ inline WaveSeg wave_seg(const AttnParams& p, const int32_t* bt_row, int b, int g, int lo,
                                   int hi, int wave, int lane)
{
    WaveSeg s;
    s.first = uniform(lo + wave);
    s.n = s.first < hi ? (hi - s.first + kWaves - 1) / kWaves : 0;
    s.bt = bt_row + s.first;
    const size_t head_off = (size_t)uniform(g) * (kBlockSize * kHeadDim);
    s.kpair = uniform_ptr(p.k + head_off);
    s.vpair = uniform_ptr(p.v + head_off);
    const int col = lane & 15;
    s.qrow = p.q + ((size_t)b * p.Hq + (size_t)g * G + (col < G ? col : 0)) * kHeadDim + 8 * (lane >> 4);
    s.b = b;
    s.g = g;
    return s;
}

// Q^T operand: lane (h, q) holds head h's dims [32i + 8q, +8) for MFMA i;
// columns past the group are zero.
template <int G>
__device__ inline void load_q(f16x8 (&qop)[4], const WaveSeg& s, int lane)
{
    if ((lane & 15) < G) {
#pragma unroll
        for (int i = 0; i < 4; ++i) qop[i] = *(const f16x8*)(s.qrow + 32 * i);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) qop[i] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }
}

// The K/V pipeline of one wave, carried from segment to segment.  Tile t
// (t = 0, 1) holds the wave's blocks of parity t.  When a segment and the next
// both span at least kPrefetchBlocks blocks (every wave has at least four of
// each), a segment's last two steps refill the tiles with the next segment's
// blocks 0 and 1: they are in flight while the work group merges and emits
// the segment, and the next segment starts with its first loads issued long
// before.  Otherwise the next segment loads its first blocks itself.
constexpr int kPrefetchBlocks = 16;

struct WaveTiles {
    u32x4 kt0[4], vt0[4], kt1[4], vt1[4];
    int cur0, cur1;      // ids of the blocks in the tiles
    int nid0, nid1;      // ids of the blocks that refill the tiles next
    bool prefetched;     // the tiles hold the segment's blocks 0 and 1
    f16x8 qop[4];        // Q^T of the current segment
    f16x8 qnext[4];      // Q^T of the next segment (loaded one segment ahead)
};

// Fused append.  Scaled logits (log2 units) of the current token for the G
// q-heads of pair (b, g), computed by one wave (lane l takes dims 2l, 2l + 1):
// the loads, then (once they are complete) the sums.
template <int G>
struct NewTokenRows {
    f16x2 k2;
    f16x2 q2[G];
};

template <int G>
__device__ inline void load_new_token_rows(const AttnParams& p, int b, int g, int lane, NewTokenRows<G>& r)
{
    r.k2 = *(const f16x2*)(p.k_new + (size_t)b * p.new_stride + (size_t)g * kHeadDim + 2 * lane);
#pragma unroll
    for (int h = 0; h < G; ++h)
        r.q2[h] = *(const f16x2*)(p.q + ((size_t)b * p.Hq + (size_t)g * G + h) * kHeadDim + 2 * lane);
}

template <int G>
__device__ inline void new_token_logits(const AttnParams& p, const NewTokenRows<G>& r, int lane, float* s_new)
{
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const float x = wave_incl_sum_f32(fmaf((float)r.q2[h][0], (float)r.k2[0], (float)r.q2[h][1] * (float)r.k2[1]));
        if (lane == 63) s_new[h] = x * p.scale_log2;
    }
}

// The current token's K and V elements `dim` of kv-head g of request b and
// the id of the block that holds its slot (position Lc - 1, Lc = the full
// length), loaded ahead of the emit that needs them.  With the input check a
// position past an explicit table row (a context cut to its row, already
// reported) has no slot: the row's last slot holds a cached token.  The
// slot's table entry is the same for the whole work group, so it is read
// through the constant address space (the scalar path); `safe` is any
// readable entry, read instead when there is no slot.
// (The emit's loops give a thread elements idx = tid + k kAttnThreads, all
// of one dim when kAttnThreads is a multiple of the head dimension.)
static_assert(kAttnThreads % kHeadDim == 0, "a thread's emit elements share one dim");
struct NewTokenElems {
    f16 kn, vn;
    int id;
    bool in_row;
};

template <bool kCheck>
__device__ inline NewTokenElems load_new_token_elems(const AttnParams& p, const int32_t* bt_row,
                                                     const int32_t* safe, int b, int g, int Lc, int dim)
{
    NewTokenElems e;
    const size_t src = (size_t)b * p.new_stride + (size_t)g * kHeadDim + dim;
    e.kn = p.k_new[src];
    e.vn = p.v_new[src];
    e.in_row = !(kCheck && p.bt_stride > 0 && (int64_t)((Lc - 1) / kBlockSize) >= p.bt_stride);
    const int32_t* a = e.in_row ? bt_row + (Lc - 1) / kBlockSize : safe;
    e.id = *(const __attribute__((address_space(4))) int32_t*)a;
    return e;
}

// Per-wave attention over its blocks of segment cs; ns is the work group's
// next segment (n = 0 if none), `safe` any readable block-table entry, pf_next
// whether the tiles continue into ns, cur_row the block-table row of cs's
// request (with the fused append, ne receives this thread's elements of the
// current token for the emit: dim = thread index mod 128).  Lane
// (h = lane % 16, q = lane / 16) keeps m (running max of head h, log2 units,
// equal on the four lanes of h), l (sum of the weights of its tokens) and
// acc[t][i] (running P.V of head h at dim 32q + 8i + t).  On return the
// wave's state is in s_acc/s_m/s_l and the tiles hold (in flight) the next
// segment's first blocks.
template <int G, bool kCheck, bool kAppend>
__device__ inline void wave_attend(const AttnParams& p, const WaveSeg& cs, const WaveSeg& ns,
                                   const int32_t* safe, bool pf_next, int L, WaveTiles& st, int wave,
                                   int lane,
                                   float (*s_acc)[G][kHeadDim], float (*s_m)[G], float (*s_l)[G],
                                   float* s_new, const int32_t* cur_row, NewTokenElems& ne)
{
    constexpr int D = kHeadDim;
    constexpr int BS = kBlockSize;
    const int col = lane & 15;
    const int q = lane >> 4;
    const int n = cs.n;

    const uint32_t step = (uint32_t)((size_t)p.Hkv * BS * D);
    const int koff = k_lane_offset(lane);
    const int voff = v_lane_offset(lane);
    // with the input check, a block id outside the pool is never read: its
    // loads get a zero extent like those past the end
    auto id_ok = [&](int id) -> bool { return !kCheck || (id >= 0 && (int64_t)id < p.num_blocks); };
    // block id at position pos of this (here) or the next segment's wave
    // list; `ok` false reads the safe entry (the id is then unused).  The
    // table is read-only during the call: reading it through the constant
    // address space keeps the load on the scalar path.
    auto id_at = [&](bool here, int pos, bool ok) -> int {
        const int32_t* a = ok ? (here ? cs.bt : ns.bt) + kWaves * pos : safe;
        return *(const __attribute__((address_space(4))) int32_t*)a;
    };
    // the tiles continue into the next segment (the work group's choice:
    // both segments are long)
    const bool pf = pf_next;

    if (!st.prefetched) {
        // load the segment's blocks 0 and 1 (tile 0 first)
        st.cur0 = id_at(true, 0, n > 0);
        st.cur1 = id_at(true, 1, n > 1);
        const int nb0 = n > 0 && id_ok(st.cur0) ? kSlabBytes : 0;
        const int nb1 = n > 1 && id_ok(st.cur1) ? kSlabBytes : 0;
        load_slab(st.kt0, cs.kpair + (uint64_t)(uint32_t)st.cur0 * step, nb0, koff, 64);
        load_slab(st.vt0, cs.vpair + (uint64_t)(uint32_t)st.cur0 * step, nb0, voff, 256);
        load_slab(st.kt1, cs.kpair + (uint64_t)(uint32_t)st.cur1 * step, nb1, koff, 64);
        load_slab(st.vt1, cs.vpair + (uint64_t)(uint32_t)st.cur1 * step, nb1, voff, 256);
        st.nid0 = id_at(true, 2, n > 2);
        st.nid1 = id_at(true, 3, n > 3);
    }
    // Everything loaded before the loop (the tiles, mostly issued during the
    // previous segment's last steps, and this segment's Q^T, issued one
    // segment ahead) is complete from here on, so the loop's own waits are
    // those of its two-deep pipeline alone.
    __builtin_amdgcn_s_waitcnt(0);
#ifdef APEX_TRACE_WORK_GROUPS
    if (wave == 0 && lane == 0 && s_trace[2] == 0) s_trace[2] = trace_clock();
#endif
#pragma unroll
    for (int i = 0; i < 4; ++i) st.qop[i] = st.qnext[i];
    load_q<G>(st.qnext, ns, lane);   // used by the next segment only
    // With the fused append: the rows of the current token's logits for this
    // pair (wave 0 sums them after the loop; the merge reads them) and this
    // thread's elements for the emit.  Issued after the wait above, they
    // complete during the block loop instead of adding a round trip to the
    // segment's entry and to its emit.  Every wave issues the row loads, a
    // few hundred bytes: with a branch on the wave around them the compiler's
    // wait placement could not tell that every path passes the loop's waits.
    NewTokenRows<G> nt;
    if (kAppend) {
        load_new_token_rows<G>(p, cs.b, cs.g, lane, nt);
        ne = load_new_token_elems<kCheck>(p, cur_row, safe, cs.b, cs.g, L + 1, (wave * 64 + lane) % D);
    }

    float m = -INFINITY, l = 0.f;
    f32x4 acc[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

    // One block: consume (kt, vt) holding block k (id cur) of tile t = k % 2,
    // refill them with the tile's next element (id nid: this segment's block
    // k + 2, else the next segment's block t), look up the id of the element
    // after that.  Slab addresses are formed in scalar registers only, block
    // ids arrive through the scalar path ahead of use, and every step issues
    // eight loads (zero-extent when there is no element) so the compiler can
    // wait for exactly the oldest slab.
    auto block_step = [&](u32x4 (&kt)[4], u32x4 (&vt)[4], int k, int& cur, int& nid) {
        const int t = k & 1;
        // refill: this segment's block k + 2, else the next segment's block
        // t (with pf), else nothing
        const bool r_here = k + 2 < n;
        const bool r_ok = r_here || pf;
        // the id of the tile's element after that: block k + 4 here, else the
        // next segment's block t or t + 2
        const bool l_here = k + 4 < n;
        const int l_pos = l_here ? k + 4 : (r_here ? t : t + 2);
        const int id_next = id_at(l_here, l_pos, l_here || pf);
        const int id2 = nid;
        const f16* kbase = r_here ? cs.kpair : ns.kpair;
        const f16* vbase = r_here ? cs.vpair : ns.vpair;
        const int nbytes = r_ok && id_ok(id2) ? kSlabBytes : 0;
        const int tok0 = (cs.first + kWaves * k) * BS;
        const int cur_id = cur;
        cur = id2;
        nid = id_next;
        if (kCheck && !id_ok(cur_id)) {
            // skip the block (its tokens take no part), keep the pipeline going
            if (lane == 0) report_error(p, kErrBlockId);
            load_slab(kt, kbase + (uint64_t)(uint32_t)id2 * step, nbytes, koff, 64);
            load_slab(vt, vbase + (uint64_t)(uint32_t)id2 * step, nbytes, voff, 256);
            return;
        }
        // S^T = K Q^T: lane (h, q) gets the scores of tokens 4q..4q+3 of head h
        f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 4; ++i)
            s = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, kt[i]), st.qop[i], s, 0, 0, 0);
        // K is consumed: refill it (in place: the barrier keeps the scheduler
        // from issuing the loads above the products that read the tile)
        __builtin_amdgcn_sched_barrier(0);
        load_slab(kt, kbase + (uint64_t)(uint32_t)id2 * step, nbytes, koff, 64);

        float sv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) sv[i] = s[i] * p.scale_log2;
        const bool tail = tok0 > L - BS;   // the pair's last, partial block (no overflow at L near 2^31)
        if (tail) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (tok0 + 4 * q + i >= L) sv[i] = -INFINITY;
        }
        const float bm = rows_max4(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])));
        const float mnew = fmaxf(m, bm);   // finite: the block holds a valid token
        const float alpha = exp2_fast(m - mnew);
        f32x4 pw;
#pragma unroll
        for (int i = 0; i < 4; ++i) pw[i] = exp2_fast(sv[i] - mnew);
        // the weights as two fp16 MFMA operands: ph = pw rounded to fp16 and
        // pl = the rest rounded to fp16, together 22 significant bits (the
        // rest pw - ph is exact in fp32); the normaliser sums the same parts
        const f16x4 ph = __builtin_convertvector(pw, f16x4);
        const f32x4 ph32 = __builtin_convertvector(ph, f32x4);
        const f16x4 pl = __builtin_convertvector(pw - ph32, f16x4);
        const f32x4 pq = ph32 + __builtin_convertvector(pl, f32x4);
        l = l * alpha + ((pq[0] + pq[1]) + (pq[2] + pq[3]));
        m = mnew;

        // V^T operands in registers: tile t row c is dim 8c + t, its k index
        // is token 4q + e; rows of masked tokens are zeroed (they may hold NaN)
        unsigned a[8][2];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const unsigned sel = (t & 1) ? kHiHalves : kLoHalves;
            const int w = t >> 1;
            a[t][0] = pack_halves(vt[0][w], vt[1][w], sel);
            a[t][1] = pack_halves(vt[2][w], vt[3][w], sel);
        }
        // V is consumed: refill it (in place)
        __builtin_amdgcn_sched_barrier(0);
        load_slab(vt, vbase + (uint64_t)(uint32_t)id2 * step, nbytes, voff, 256);
        if (tail) {
            const bool ok0 = tok0 + 4 * q + 0 < L, ok1 = tok0 + 4 * q + 1 < L;
            const bool ok2 = tok0 + 4 * q + 2 < L, ok3 = tok0 + 4 * q + 3 < L;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                a[t][0] = (ok0 ? a[t][0] & 0x0000ffffu : 0u) | (ok1 ? a[t][0] & 0xffff0000u : 0u);
                a[t][1] = (ok2 ? a[t][1] & 0x0000ffffu : 0u) | (ok3 ? a[t][1] & 0xffff0000u : 0u);
            }
        }
        if (alpha != 1.f) {
#pragma unroll
            for (int t = 0; t < 8; ++t) acc[t] *= alpha;
        }
        // O^T += V^T P^T, eight 16-dim tiles, the high parts of P, then the
        // low parts (independent accumulators between the two passes)
        typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const u32x2 av = {a[t][0], a[t][1]};
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, av), ph, acc[t], 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const u32x2 av = {a[t][0], a[t][1]};
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, av), pl, acc[t], 0, 0, 0);
        }
    };

    // pairs of blocks, then an odd last block on tile 0 (a loop with a single
    // exit keeps both tiles in the same registers from one segment to the next)
    int k = 0;
    for (; k + 1 < n; k += 2) {
        block_step(st.kt0, st.vt0, k, st.cur0, st.nid0);
        block_step(st.kt1, st.vt1, k + 1, st.cur1, st.nid1);
    }
    if (k < n) block_step(st.kt0, st.vt0, k, st.cur0, st.nid0);
    st.prefetched = pf;
    if (kAppend && uniform(wave) == 0) new_token_logits<G>(p, nt, lane, s_new);

    // the wave's state for head h: l summed over the four token groups
    const float lw = rows_sum4(l);
    if (col < G) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float* dst = &s_acc[wave][col][32 * q + 8 * i];
            *(f32x4*)dst = f32x4{acc[0][i], acc[1][i], acc[2][i], acc[3][i]};
            *(f32x4*)(dst + 4) = f32x4{acc[4][i], acc[5][i], acc[6][i], acc[7][i]};
        }
        if (q == 0) {
            s_m[wave][col] = m;
            s_l[wave][col] = lw;
        }
    }
}

__device__ inline void write_row(const AttnParams& p, int b, int head, int dim, float M, float num,
                                 float den)
{
    const float o = den > 0.f ? num / den : 0.f;
    p.out[((size_t)b * p.Hq + head) * kHeadDim + dim] = (f16)o;
    if (p.lse && dim == 0)
        p.lse[(size_t)b * p.Hq + head] =
            den > 0.f ? (M + __log2f(den)) * 0.69314718055994531f : -INFINITY;
}

// Folds the current token (logit sn in log2 units, value vn) into a merged
// state: running max M (log2 units; -inf when empty) and num, den relative
// to it, with its fp32 weight.
__device__ inline void fold_new_token(float sn, float vn, float& M, float& num, float& den)
{
    const float M2 = fmaxf(M, sn);
    const float r = M == -INFINITY ? 0.f : exp2_fast(M - M2);
    const float wgt = exp2_fast(sn - M2);
    num = fmaf(wgt, vn, num * r);
    den = fmaf(den, r, wgt);
    M = M2;
}

// Writes those elements to the slot (with the input check, a block id outside
// the pool is reported and not written).
template <bool kCheck>
__device__ inline void store_new_token(const AttnParams& p, const NewTokenElems& e, int g, int Lc, int dim)
{
    if (!e.in_row) return;
    if (kCheck && !(e.id >= 0 && (int64_t)e.id < p.num_blocks)) {
        if (dim == 0) report_error(p, kErrBlockId);
        return;
    }
    const size_t dst = (((size_t)(uint32_t)e.id * p.Hkv + g) * kBlockSize + (Lc - 1) % kBlockSize) * kHeadDim + dim;
    p.k_store[dst] = e.kn;
    p.v_store[dst] = e.vn;
}

template <int G, bool kCheck, bool kAppend>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2))) void attn_kernel(AttnParams p,
                                                        const int32_t* __restrict__ bt,
                                                        const int32_t* __restrict__ lens)
{
    constexpr int D = kHeadDim;
    __shared__ float s_acc[kWaves][G][D];
    __shared__ float s_m[kWaves][G];
    __shared__ float s_l[kWaves][G];
    __shared__ int s_lens[kCachedLens];
    __shared__ int s_wsum[kWaves];
    __shared__ int s_wmax[kWaves];
    __shared__ int s_wcnt[kWaves];
    __shared__ int s_loc_b;
    __shared__ int64_t s_loc_pre;
    __shared__ int s_loc_g;
    __shared__ int s_loc_blk;
    __shared__ int64_t s_loc_vf;
    __shared__ int s_last;
    __shared__ float s_new[G];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t w = blockIdx.x;
    const int B = p.B;
    const bool cached = B <= kCachedLens;
#ifdef APEX_TRACE_WORK_GROUPS
    if (tid < kTraceWords) s_trace[tid] = tid == 0 ? trace_clock() : 0;
#endif

    // 1. partition.  context_lens is read from memory once: each thread sums
    // the blocks of a contiguous run of requests (and keeps the lengths in
    // LDS when they fit); wave-level scans plus one barrier give the prefix
    // sums, the total, the longest request and the non-empty requests.
    const int seg = (B + kAttnThreads - 1) / kAttnThreads;
    const int r0 = min(B, tid * seg);
    const int r1 = min(B, r0 + seg);
    // with the input check, a context longer than an explicit table row is
    // cut to the row (and reported)
    const int64_t row_tokens = p.bt_stride * kBlockSize;
    auto is_cut = [&](int L) -> bool { return kCheck && p.bt_stride > 0 && L > row_tokens; };
    // Tokens the partition covers: the cached ones.  With the fused append
    // the current token (position L - 1) comes from the new rows, so the
    // caches hold the first L - 1; a context cut to its row keeps every token
    // of the row, and its current token, whose position lies past the row,
    // is attended but has no slot to be stored in.  The tight table stride
    // follows the (cut) full lengths.
    constexpr bool append = kAppend;
    auto cached_len = [&](int L) -> int {
        if (is_cut(L)) return (int)row_tokens;
        return append && L > 0 ? L - 1 : L;
    };
    int tsum = 0, tmax = 0, tcnt = 0;
    for (int b = r0; b < r1; ++b) {
        const int raw = lens[b];
        if (is_cut(raw)) report_error(p, kErrTableRow);
        const int L = cached_len(raw);
        if (cached) s_lens[b] = L;
        const int nb = (int)blocks_of(L, kBlockSize);
        tsum += nb;
        tmax = max(tmax, (int)blocks_of(is_cut(raw) ? (int)row_tokens : raw, kBlockSize));
        tcnt += nb > 0;
    }
    const int own_cnt = tcnt;
    int incl = wave_incl_sum(tsum);
    tmax = wave_incl_max(tmax);
    int incl_cnt = wave_incl_sum(tcnt);
    if (lane == 63) {
        s_wsum[wave] = incl;
        s_wmax[wave] = tmax;
        s_wcnt[wave] = incl_cnt;
    }
    __syncthreads();
    int total = 0, maxb = 0, nonempty = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
        if (v < wave) {
            incl += s_wsum[v];
            incl_cnt += s_wcnt[v];
        }
        total += s_wsum[v];
        maxb = max(maxb, s_wmax[v]);
        nonempty += s_wcnt[v];
    }
    auto len_of = [&](int b) -> int { return cached ? s_lens[b] : cached_len(lens[b]); };

    const int64_t units = (int64_t)uniform(total) * p.Hkv;
    const int64_t pairs = (int64_t)uniform(nonempty) * p.Hkv;
    const int64_t stride = p.bt_stride > 0 ? p.bt_stride : (int64_t)uniform(maxb);
    // the cost line: every non-empty pair's K cost positions, then its blocks
    const int64_t K = p.seg_cost;
    const int64_t V = units + K * pairs;
    // The prologue is serial code of one wave per work group, so its time is
    // its instruction count: when V (launched + 1) < 2^32 (any batch below
    // about 8 M units at the default grid) every product below fits 32 bits
    // and the partition runs in 32-bit arithmetic, else in 64-bit; both give
    // the same ranges.  Lanes 0 and 1 find the range's two ends in one
    // division.
    const bool narrow = ((uint64_t)V >> 32) == 0 && (uint64_t)V * ((uint64_t)p.launched + 1) <= 0xffffffffull;
    int64_t W, v0, v1;
    if (narrow) {
        const uint32_t W32 = active_workers_t<uint32_t>((uint32_t)units, (uint32_t)p.launched, (uint32_t)p.min_units,
                                                        (uint32_t)pairs, (uint32_t)p.cus);
        const uint32_t ends = units > 0 && w < W32 ? (uint32_t)(w + (lane & 1)) * (uint32_t)V / W32 : 0u;
        W = W32;
        v0 = (uint32_t)__builtin_amdgcn_readlane((int)ends, 0);
        v1 = (uint32_t)__builtin_amdgcn_readlane((int)ends, 1);
    } else {
        W = active_workers(units, (int64_t)p.launched, p.min_units, pairs, p.cus);
        const int64_t ends = units > 0 && w < W ? worker_start(w + (lane & 1), V, W) : 0;
        v0 = ((int64_t)__builtin_amdgcn_readlane((int)(ends >> 32), 0) << 32) |
             (uint32_t)__builtin_amdgcn_readlane((int)ends, 0);
        v1 = ((int64_t)__builtin_amdgcn_readlane((int)(ends >> 32), 1) << 32) |
             (uint32_t)__builtin_amdgcn_readlane((int)ends, 1);
    }

    // The worker's blocks are those whose positions lie in [v0, v1).  Request
    // b's positions start at Hkv (pre_b + K pp_b) (pre_b blocks and pp_b
    // non-empty requests before it) and number Hkv (nb_b + K); the thread
    // whose requests hold v0 finds the pair there and its first block at or
    // after v0 (block 0 when v0 is one of the pair's cost positions), and
    // publishes the pair, that block and the position of the pair's block 0.
    // (In I = uint32_t every position is below V < 2^32.)
    auto locate = [&](auto at) {
        using I = decltype(at);
        const I hk = (I)p.Hkv, Kc = (I)K;
        const I lo = (I)(incl - tsum) + Kc * (I)(incl_cnt - own_cnt);
        const I hi = (I)incl + Kc * (I)incl_cnt;
        if (lo * hk <= at && at < hi * hk) {
            I pre = (I)(incl - tsum), vpre = lo * hk;
            for (int b = r0; b < r1; ++b) {
                // with one request per thread, its block count is the scan's
                const I nb = seg == 1 ? (I)tsum : (I)blocks_of(len_of(b), kBlockSize);
                if (nb == 0) continue;
                const I span = (nb + Kc) * hk;
                if (at < vpre + span) {
                    const I g = div_floor(at - vpre, nb + Kc);
                    const I vf = vpre + g * (nb + Kc) + Kc;   // position of the pair's block 0
                    s_loc_b = b;
                    s_loc_pre = (int64_t)pre;
                    s_loc_g = (int)g;
                    s_loc_blk = (int)(at > vf ? at - vf : 0);
                    s_loc_vf = (int64_t)vf;
                    break;
                }
                pre += nb;
                vpre += span;
            }
        }
    };
    if (v0 < v1) {
        if (narrow)
            locate((uint32_t)v0);
        else
            locate(v0);
    }
    __syncthreads();

    // A segment is the worker's blocks of one pair: from block blk of the pair
    // whose block 0 lies at position vf, up to the pair's end or the worker's
    // range end v1, whichever comes first (none when v1 falls on or before
    // the block: the range ends among cost positions).
    auto seg_take = [&](int nb_, int blk_, int64_t vf_) -> int {
        const int64_t left = v1 - (vf_ + blk_);
        return left <= 0 ? 0 : (int)min((int64_t)(nb_ - blk_), left);
    };
    int b = 0, g = 0, blk = 0, L = 0, nb = 0, take = 0;
    int64_t pre = 0, vf = 0;
    if (v0 < v1) {
        b = uniform(s_loc_b);
        pre = uniform64(s_loc_pre);
        g = uniform(s_loc_g);
        blk = uniform(s_loc_blk);
        vf = uniform64(s_loc_vf);
        L = uniform(len_of(b));
        nb = (int)blocks_of(L, kBlockSize);
        take = seg_take(nb, blk, vf);
    }

    if (take > 0) {
    // Moves a segment cursor past its segment to the worker's next one;
    // false when the worker's range is done.
    auto advance = [&](int& b_, int64_t& pre_, int& L_, int& nb_, int& g_, int& blk_, int64_t& vf_,
                       int take_) -> bool {
        blk_ += take_;
        if (blk_ < nb_) return false;   // the range ended inside the pair
        const int64_t vnext = vf_ + nb_ + K;   // the next pair's block 0
        if (v1 <= vnext) return false;
        blk_ = 0;
        vf_ = vnext;
        if (++g_ == p.Hkv) {
            g_ = 0;
            pre_ += nb_;
            do {
                ++b_;
            } while (b_ < B && len_of(b_) <= 0);
            if (b_ >= B) return false;   // unreachable: positions remain after the current pair
            L_ = uniform(len_of(b_));
            nb_ = (int)blocks_of(L_, kBlockSize);
        }
        return true;
    };

    // 2. segments.  Each one is announced to the waves together with the
    // next, so their K/V pipelines run on from one to the other.
#ifdef APEX_TRACE_WORK_GROUPS
    if (tid == 0) s_trace[1] = trace_clock();
#endif
    WaveSeg cs = wave_seg<G>(p, bt + (size_t)uniform(b) * (size_t)stride, b, g, blk, blk + take, wave, lane);
    WaveTiles st;
    st.prefetched = false;
    st.cur0 = st.cur1 = st.nid0 = st.nid1 = 0;
    load_q<G>(st.qnext, cs, lane);
    while (true) {
        int b2 = b, L2 = L, nb2 = nb, g2 = g, blk2 = blk;
        int64_t pre2 = pre, vf2 = vf;
        const bool more = advance(b2, pre2, L2, nb2, g2, blk2, vf2, take);
        const int take2 = more ? seg_take(nb2, blk2, vf2) : 0;
        WaveSeg ns = cs;
        ns.n = 0;
        if (more)
            ns = wave_seg<G>(p, bt + (size_t)uniform(b2) * (size_t)stride, b2, g2, blk2, blk2 + take2, wave,
                             lane);
        NewTokenElems ne;
        wave_attend<G, kCheck, kAppend>(p, cs, ns, bt,
                                        more && take >= kPrefetchBlocks && take2 >= kPrefetchBlocks, L,
                                        st, wave, lane, s_acc, s_m, s_l, s_new,
                                        bt + (size_t)uniform(b) * (size_t)stride, ne);
        __syncthreads();
#ifdef APEX_TRACE_WORK_GROUPS
        if (tid == 0) {
            ++s_trace[4];
            s_trace[6] += take;
        }
#endif

        // 3. merge the waves, emit rows or a partial
        const int64_t wf = worker_of(vf, V, W);
        const int64_t wl = worker_of(vf + nb - 1, V, W);
        const int64_t slot = partial_slot(w, wf);
        for (int idx = tid; idx < G * D; idx += kAttnThreads) {
            const int h = idx / D, dim = idx % D;
            float M = s_m[0][h];
#pragma unroll
            for (int q = 1; q < kWaves; ++q) M = fmaxf(M, s_m[q][h]);
            const float Ms = M == -INFINITY ? 0.f : M;
            float num = 0.f, den = 0.f;
#pragma unroll
            for (int q = 0; q < kWaves; ++q) {
                const float f = exp2_fast(s_m[q][h] - Ms);
                num = fmaf(f, s_acc[q][h][dim], num);
                den = fmaf(f, s_l[q][h], den);
            }
            if (wf == wl) {
                if (append) {
                    fold_new_token(s_new[h], (float)ne.vn, M, num, den);
                    if (h == 0) store_new_token<kCheck>(p, ne, g, L + 1, dim);
                }
                write_row(p, b, g * G + h, dim, M, num, den);
            } else {
                store_coherent(&p.pacc[((size_t)slot * G + h) * D + dim], num);
                if (dim == 0) {
                    store_coherent(&p.pml[((size_t)slot * G + h) * 2 + 0], M);
                    store_coherent(&p.pml[((size_t)slot * G + h) * 2 + 1], den);
                }
            }
        }
        if (wf != wl) {
#ifdef APEX_TRACE_WORK_GROUPS
            if (tid == 0) ++s_trace[5];
#endif
            // The partials are written with device-coherent stores; waiting for
            // them to complete before the arrival is counted makes them visible
            // to the last arriver's device-coherent loads, on whichever XCD it
            // runs, without writing back or invalidating the L2.
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (tid == 0) {
                int32_t* cnt = &p.counters[(size_t)b * p.Hkv + g];
                const int old = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const int last = old == (int)(wl - wf);
                if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                s_last = last;
            }
            __syncthreads();
            if (s_last) {
                // combine the pair's partials: each thread issues the loads of
                // kCombineChunk contributors at once, then folds them in with
                // an online rescale (running max M, numerator, denominator)
                const int nc = (int)(wl - wf + 1);
                // the first contributor's slot is 2wf + 1; every later one
                // starts inside the pair, so its slot is 2v (partial_slot)
                const int64_t first_slot = partial_slot(wf, wf);
                for (int idx = tid; idx < G * D; idx += kAttnThreads) {
                    const int h = idx / D, dim = idx % D;
                    float M = -INFINITY, num = 0.f, den = 0.f;
                    for (int c0 = 0; c0 < nc; c0 += kCombineChunk) {
                        float cm[kCombineChunk], cl[kCombineChunk], ca[kCombineChunk];
#pragma unroll
                        for (int j = 0; j < kCombineChunk; ++j) {
                            cm[j] = -INFINITY;
                            cl[j] = 0.f;
                            ca[j] = 0.f;
                            if (c0 + j < nc) {
                                const int64_t sq = c0 + j == 0 ? first_slot : 2 * (wf + c0 + j);
                                cm[j] = load_coherent(&p.pml[((size_t)sq * G + h) * 2]);
                                cl[j] = load_coherent(&p.pml[((size_t)sq * G + h) * 2 + 1]);
                                ca[j] = load_coherent(&p.pacc[((size_t)sq * G + h) * D + dim]);
                            }
                        }
                        float Mn = M;
#pragma unroll
                        for (int j = 0; j < kCombineChunk; ++j) Mn = fmaxf(Mn, cm[j]);
                        const float Ms = Mn == -INFINITY ? 0.f : Mn;
                        const float r = exp2_fast(M - Ms);
                        num *= r;
                        den *= r;
#pragma unroll
                        for (int j = 0; j < kCombineChunk; ++j) {
                            const float f = exp2_fast(cm[j] - Ms);
                            num = fmaf(f, ca[j], num);
                            den = fmaf(f, cl[j], den);
                        }
                        M = Mn;
                    }
                    if (append) {
                        fold_new_token(s_new[h], (float)ne.vn, M, num, den);
                        if (h == 0) store_new_token<kCheck>(p, ne, g, L + 1, dim);
                    }
                    write_row(p, b, g * G + h, dim, M, num, den);
                }
            }
        }
        __syncthreads();

        if (!more) break;
        b = b2;
        pre = pre2;
        vf = vf2;
        L = L2;
        nb = nb2;
        g = g2;
        blk = blk2;
        take = take2;
        cs = ns;
    }
    }

    // rows of empty requests are zeros (and lse = -inf); with the fused
    // append a request whose only token is the current one returns its V row
    // (lse = its scaled logit) and stores its K/V
    for (int b = (int)w; b < B; b += (int)gridDim.x) {
        if (len_of(b) > 0) continue;
        if (append && lens[b] == 1) {
            const size_t nrow = (size_t)b * p.new_stride;
            for (int i = tid; i < p.Hq * D; i += kAttnThreads) {
                const int h = i / D, dim = i % D;
                p.out[((size_t)b * p.Hq + h) * D + dim] = p.v_new[nrow + (size_t)(h / (p.Hq / p.Hkv)) * D + dim];
            }
            if (p.lse) {
                for (int h = wave; h < p.Hq; h += kWaves) {
                    const f16x2 k2 = *(const f16x2*)(p.k_new + nrow + (size_t)(h / (p.Hq / p.Hkv)) * D + 2 * lane);
                    const f16x2 q2 = *(const f16x2*)(p.q + ((size_t)b * p.Hq + h) * D + 2 * lane);
                    float x = fmaf((float)q2[0], (float)k2[0], (float)q2[1] * (float)k2[1]);
#pragma unroll
                    for (int m = 32; m >= 1; m >>= 1) x += wave_shfl_xor(x, m);
                    if (lane == 0) p.lse[(size_t)b * p.Hq + h] = x * p.scale_log2 * 0.69314718055994531f;
                }
            }
            for (int i = tid; i < p.Hkv * D; i += kAttnThreads)
                store_new_token<kCheck>(
                    p, load_new_token_elems<kCheck>(p, bt + (size_t)b * stride, bt, b, i / D, 1, i % D), i / D, 1,
                    i % D);
        } else {
            for (int i = tid; i < p.Hq * D; i += kAttnThreads) write_row(p, b, i / D, i % D, 0.f, 0.f, 0.f);
        }
    }
#ifdef APEX_TRACE_WORK_GROUPS
    if (p.trace && tid == 0 && w < p.trace_groups) {
        uint64_t* t = p.trace + w * kTraceWords;
        t[0] = s_trace[0];
        t[1] = s_trace[1];
        t[2] = s_trace[2];
        t[3] = trace_clock();
        t[4] = s_trace[4];
        t[5] = s_trace[5];
        t[6] = s_trace[6];
        t[7] = 0;
    }
#endif
}

}  // namespace apex
