// kernels.h -- gfx950 kernels of batched paged decode attention.
//
// One call = three stream-ordered launches:
//   plan_kernel      one work group: reads context_lens, sizes the split-K
//                    ranges (plan_policy.h) and writes a work list ordered
//                    longest range first, plus the tight block-table stride.
//   attn_kernel<G>   one 4-wave work group per work item (request b, kv-head
//                    g, block range).  Gathers the paged K/V rows with 128-bit
//                    loads, computes the G q-heads' scores, runs an online
//                    softmax (running max and sum, base-2 exponentials with
//                    log2(e) folded into the scale) with fp32 P.V
//                    accumulation, merges the waves' states in LDS and either
//                    writes the fp16 output row or an fp32 partial
//                    (acc, max, sum) for the combine.
//   combine_kernel<G> log-sum-exp combine of the partials of split requests.
//
// The attention itself is the standard softmax attention that APEX runs for
// its GPU-resident decode requests over their paged KV (Sec. 3.1, Sec. 3.3,
// Sec. 4.1); the split-K decomposition is exact up to rounding: with per-range
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

struct WsHeader {
    int32_t n_items;
    int32_t maxb;      // ceil(max_b L_b / block_size): the tight table stride
    int32_t n_slots;   // partial-result slots used
    int32_t pad0;
    int64_t chunk;     // planner chunk, in blocks
    int64_t units;     // sum of blocks x Hkv
    int64_t pad[4];
};

struct Item {
    int32_t b, g, blk0, blk1;
    int32_t slot;      // first partial slot of this item, or -1 = write out directly
    int32_t L;
    int32_t pad0, pad1;
};

struct ReqInfo {
    int32_t n;          // ranges
    int32_t per;        // blocks per range
    int32_t slot_base;  // first partial slot of the request, -1 if unsplit
    int32_t L;
};

struct WsPtrs {
    WsHeader* hdr;
    ReqInfo* req;
    Item* items;
    float* pacc;   // [slots][G][d]   unnormalised accumulators
    float* pml;    // [slots][G][2]   (max in log2 units, sum)
};

constexpr int kPlanThreads = 1024;
constexpr int kBins = 1024;   // == kPlanThreads: one bin per thread in the scan
constexpr int kAttnThreads = 256;
constexpr int kWaves = kAttnThreads / 64;

// ---------------------------------------------------------------------------
// planner
// ---------------------------------------------------------------------------

__device__ inline void block_inclusive_scan(int64_t* s, int tid)
{
    for (int off = 1; off < kPlanThreads; off <<= 1) {
        int64_t v = tid >= off ? s[tid - off] : 0;
        __syncthreads();
        s[tid] += v;
        __syncthreads();
    }
}

__device__ inline int bin_of(int64_t len)
{
    return len >= kBins ? kBins - 1 : (int)len;
}

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(const int32_t* __restrict__ lens, int B,
                                                             int Hkv, int64_t target, int forced,
                                                             WsPtrs ws)
{
    __shared__ int64_t s_scan[kPlanThreads];
    __shared__ int64_t s_bins[kPlanThreads];
    __shared__ int s_bin_cursor[kBins];
    __shared__ int64_t s_units;
    __shared__ int s_maxb;

    const int tid = threadIdx.x;
    const int seg = (B + kPlanThreads - 1) / kPlanThreads;
    const int b0 = min(B, tid * seg);
    const int b1 = min(B, b0 + seg);

    if (tid == 0) {
        s_units = 0;
        s_maxb = 0;
    }
    s_bin_cursor[tid] = 0;
    __syncthreads();

    int64_t units = 0;
    int mx = 0;
    for (int b = b0; b < b1; ++b) {
        const int64_t nb = blocks_of(lens[b], kBlockSize);
        units += nb;
        mx = max(mx, (int)nb);
    }
    atomicAdd((unsigned long long*)&s_units, (unsigned long long)units);
    atomicMax(&s_maxb, mx);
    __syncthreads();

    const int64_t chunk = chunk_blocks(s_units * Hkv, target);

    // partial slots (request order) and range-length histogram
    int64_t my_slots = 0;
    for (int b = b0; b < b1; ++b) {
        const int64_t nb = blocks_of(lens[b], kBlockSize);
        const SplitPlan sp = split_request(nb, chunk, forced);
        if (sp.n > 1) my_slots += (int64_t)sp.n * Hkv;
        const int64_t full = sp.per > 0 ? nb / sp.per : 0;
        const int64_t rem = nb - full * sp.per;
        const int64_t empties = sp.n - full - (rem > 0 ? 1 : 0);
        if (full) atomicAdd(&s_bin_cursor[bin_of(sp.per)], (int)(full * Hkv));
        if (rem) atomicAdd(&s_bin_cursor[bin_of(rem)], Hkv);
        if (empties) atomicAdd(&s_bin_cursor[0], (int)(empties * Hkv));
    }
    __syncthreads();
    s_scan[tid] = my_slots;
    // longest ranges first: scan the histogram from the top bin down
    s_bins[tid] = s_bin_cursor[kBins - 1 - tid];
    __syncthreads();
    block_inclusive_scan(s_scan, tid);
    block_inclusive_scan(s_bins, tid);
    const int64_t slot_base = s_scan[tid] - my_slots;
    s_bin_cursor[kBins - 1 - tid] = (int)(s_bins[tid] - s_bin_cursor[kBins - 1 - tid]);
    __syncthreads();

    int64_t slot = slot_base;
    for (int b = b0; b < b1; ++b) {
        const int32_t L = lens[b];
        const int64_t nb = blocks_of(L, kBlockSize);
        const SplitPlan sp = split_request(nb, chunk, forced);
        ReqInfo ri;
        ri.n = sp.n;
        ri.per = sp.per;
        ri.slot_base = sp.n > 1 ? (int32_t)slot : -1;
        ri.L = L;
        ws.req[b] = ri;
        for (int s = 0; s < sp.n; ++s) {
            int64_t lo = (int64_t)s * sp.per;
            int64_t hi = lo + sp.per;
            if (lo > nb) lo = nb;
            if (hi > nb) hi = nb;
            const int bin = bin_of(hi - lo);
            for (int g = 0; g < Hkv; ++g) {
                const int pos = atomicAdd(&s_bin_cursor[bin], 1);
                Item it;
                it.b = b;
                it.g = g;
                it.blk0 = (int32_t)lo;
                it.blk1 = (int32_t)hi;
                it.slot = sp.n > 1 ? (int32_t)(slot + (int64_t)g * sp.n + s) : -1;
                it.L = L;
                it.pad0 = 0;
                it.pad1 = 0;
                ws.items[pos] = it;
            }
        }
        if (sp.n > 1) slot += (int64_t)sp.n * Hkv;
    }
    if (tid == kPlanThreads - 1) {
        WsHeader h = {};
        h.n_items = (int32_t)s_bins[kPlanThreads - 1];
        h.maxb = s_maxb;
        h.n_slots = (int32_t)s_scan[kPlanThreads - 1];
        h.chunk = chunk;
        h.units = s_units * Hkv;
        *ws.hdr = h;
    }
}

// ---------------------------------------------------------------------------
// attention over one work item
// ---------------------------------------------------------------------------

struct AttnParams {
    const f16* q;
    const f16* k;
    const f16* v;
    const int32_t* bt;
    f16* out;
    float* lse;        // optional [B][Hq] natural log
    int64_t bt_stride; // 0 = tight (header maxb)
    WsPtrs ws;
    float scale_log2;  // scale * log2(e)
    int Hq;
    int Hkv;
};

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

template <int G>
__global__ __launch_bounds__(kAttnThreads) void attn_kernel(AttnParams p)
{
    constexpr int D = kHeadDim;
    constexpr int BS = kBlockSize;
    __shared__ float s_acc[kWaves][G][D];
    __shared__ float s_m[kWaves][G];
    __shared__ float s_l[kWaves][G];

    const WsHeader* hdr = p.ws.hdr;
    if ((int)blockIdx.x >= hdr->n_items) return;
    const Item it = p.ws.items[blockIdx.x];
    const int64_t stride = p.bt_stride > 0 ? p.bt_stride : (int64_t)hdr->maxb;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r = lane >> 4;   // row: tokens r, r+4, r+8, r+12 of a block
    const int c = lane & 15;   // column: dims [8c, 8c+8)
    const int b = it.b, g = it.g, L = it.L;

    f16x2 qv[G][4];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const u32x4 raw = *(const u32x4*)(p.q + ((size_t)b * p.Hq + (size_t)g * G + h) * D + 8 * c);
        qv[h][0] = as_h2(raw.x);
        qv[h][1] = as_h2(raw.y);
        qv[h][2] = as_h2(raw.z);
        qv[h][3] = as_h2(raw.w);
    }

    float m[G], l[G], acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    }

    const int32_t* bt_row = p.bt + (size_t)b * (size_t)stride;
    const size_t head_off = (size_t)g * (BS * D) + (size_t)r * D + 8 * c;
    const size_t blk_elems = (size_t)p.Hkv * BS * D;

    u32x4 kc[4], vc[4], kn[4], vn[4];
    int j = it.blk0 + wave;
    if (j < it.blk1) {
        const int pid = __builtin_amdgcn_readfirstlane(bt_row[j]);
        const f16* kb = p.k + (size_t)pid * blk_elems + head_off;
        const f16* vb = p.v + (size_t)pid * blk_elems + head_off;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            kc[i] = *(const u32x4*)(kb + i * 4 * D);
            vc[i] = *(const u32x4*)(vb + i * 4 * D);
        }
    }
    for (; j < it.blk1; j += kWaves) {
        const int jn = j + kWaves;
        if (jn < it.blk1) {
            const int pid = __builtin_amdgcn_readfirstlane(bt_row[jn]);
            const f16* kb = p.k + (size_t)pid * blk_elems + head_off;
            const f16* vb = p.v + (size_t)pid * blk_elems + head_off;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                kn[i] = *(const u32x4*)(kb + i * 4 * D);
                vn[i] = *(const u32x4*)(vb + i * 4 * D);
            }
        }

        // scores of tokens j*16 + r + 4i for the G heads, reduced over the row
        float s[4][G];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const f16x2 k0 = as_h2(kc[i].x);
            const f16x2 k1 = as_h2(kc[i].y);
            const f16x2 k2 = as_h2(kc[i].z);
            const f16x2 k3 = as_h2(kc[i].w);
#pragma unroll
            for (int h = 0; h < G; ++h) {
                float d = __builtin_amdgcn_fdot2(k0, qv[h][0], 0.f, false);
                d = __builtin_amdgcn_fdot2(k1, qv[h][1], d, false);
                d = __builtin_amdgcn_fdot2(k2, qv[h][2], d, false);
                d = __builtin_amdgcn_fdot2(k3, qv[h][3], d, false);
                s[i][h] = d;
            }
        }
#pragma unroll
        for (int msk = 1; msk < 16; msk <<= 1) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int h = 0; h < G; ++h) s[i][h] += wave_shfl_xor(s[i][h], msk);
        }

        const int tok0 = j * BS + r;
        float vf[4][8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const bool valid = tok0 + 4 * i < L;
            const f16x2 v0 = as_h2(vc[i].x);
            const f16x2 v1 = as_h2(vc[i].y);
            const f16x2 v2 = as_h2(vc[i].z);
            const f16x2 v3 = as_h2(vc[i].w);
            vf[i][0] = valid ? (float)v0.x : 0.f;
            vf[i][1] = valid ? (float)v0.y : 0.f;
            vf[i][2] = valid ? (float)v1.x : 0.f;
            vf[i][3] = valid ? (float)v1.y : 0.f;
            vf[i][4] = valid ? (float)v2.x : 0.f;
            vf[i][5] = valid ? (float)v2.y : 0.f;
            vf[i][6] = valid ? (float)v3.x : 0.f;
            vf[i][7] = valid ? (float)v3.y : 0.f;
#pragma unroll
            for (int h = 0; h < G; ++h) s[i][h] = valid ? s[i][h] * p.scale_log2 : -INFINITY;
        }

#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float mx = fmaxf(fmaxf(s[0][h], s[1][h]), fmaxf(s[2][h], s[3][h]));
            const float mnew = fmaxf(m[h], mx);
            const float ms = mnew == -INFINITY ? 0.f : mnew;
            const float alpha = exp2_fast(m[h] - ms);
            float pi[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) pi[i] = exp2_fast(s[i][h] - ms);
            l[h] = l[h] * alpha + ((pi[0] + pi[1]) + (pi[2] + pi[3]));
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float a = acc[h][e] * alpha;
#pragma unroll
                for (int i = 0; i < 4; ++i) a = fmaf(pi[i], vf[i][e], a);
                acc[h][e] = a;
            }
            m[h] = mnew;
        }

#pragma unroll
        for (int i = 0; i < 4; ++i) {
            kc[i] = kn[i];
            vc[i] = vn[i];
        }
    }

    // merge the four rows of the wave
#pragma unroll
    for (int h = 0; h < G; ++h) {
        float mw = fmaxf(m[h], wave_shfl_xor(m[h], 16));
        mw = fmaxf(mw, wave_shfl_xor(mw, 32));
        const float ms = mw == -INFINITY ? 0.f : mw;
        const float f = exp2_fast(m[h] - ms);
        float lw = l[h] * f;
        lw += wave_shfl_xor(lw, 16);
        lw += wave_shfl_xor(lw, 32);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float a = acc[h][e] * f;
            a += wave_shfl_xor(a, 16);
            a += wave_shfl_xor(a, 32);
            acc[h][e] = a;
        }
        if (lane < 16) {
#pragma unroll
            for (int e = 0; e < 8; ++e) s_acc[wave][h][8 * c + e] = acc[h][e];
            if (lane == 0) {
                s_m[wave][h] = mw;
                s_l[wave][h] = lw;
            }
        }
    }
    __syncthreads();

    // merge the waves and emit
    for (int idx = threadIdx.x; idx < G * D; idx += kAttnThreads) {
        const int h = idx / D, dim = idx % D;
        float M = s_m[0][h];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) M = fmaxf(M, s_m[w][h]);
        const float Ms = M == -INFINITY ? 0.f : M;
        float num = 0.f, den = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float f = exp2_fast(s_m[w][h] - Ms);
            num = fmaf(f, s_acc[w][h][dim], num);
            den = fmaf(f, s_l[w][h], den);
        }
        if (it.slot < 0) {
            const float o = den > 0.f ? num / den : 0.f;
            p.out[((size_t)b * p.Hq + (size_t)g * G + h) * D + dim] = (f16)o;
            if (p.lse && dim == 0)
                p.lse[(size_t)b * p.Hq + (size_t)g * G + h] =
                    den > 0.f ? (M + __log2f(den)) * 0.69314718055994531f : -INFINITY;
        } else {
            p.ws.pacc[((size_t)it.slot * G + h) * D + dim] = num;
            if (dim == 0) {
                p.ws.pml[((size_t)it.slot * G + h) * 2 + 0] = M;
                p.ws.pml[((size_t)it.slot * G + h) * 2 + 1] = den;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// log-sum-exp combine of split requests
// ---------------------------------------------------------------------------

struct CombineParams {
    f16* out;
    float* lse;
    WsPtrs ws;
    int Hq;
    int Hkv;
};

template <int G>
__global__ __launch_bounds__(kAttnThreads) void combine_kernel(CombineParams p)
{
    constexpr int D = kHeadDim;
    const int b = blockIdx.x / p.Hkv;
    const int g = blockIdx.x % p.Hkv;
    const ReqInfo ri = p.ws.req[b];
    if (ri.n <= 1) return;
    const int64_t base = (int64_t)ri.slot_base + (int64_t)g * ri.n;
    for (int idx = threadIdx.x; idx < G * D; idx += kAttnThreads) {
        const int h = idx / D, dim = idx % D;
        float M = -INFINITY;
        for (int s = 0; s < ri.n; ++s) M = fmaxf(M, p.ws.pml[((base + s) * G + h) * 2]);
        const float Ms = M == -INFINITY ? 0.f : M;
        float num = 0.f, den = 0.f;
        for (int s = 0; s < ri.n; ++s) {
            const float f = exp2_fast(p.ws.pml[((base + s) * G + h) * 2] - Ms);
            num = fmaf(f, p.ws.pacc[((base + s) * G + h) * D + dim], num);
            den = fmaf(f, p.ws.pml[((base + s) * G + h) * 2 + 1], den);
        }
        const float o = den > 0.f ? num / den : 0.f;
        p.out[((size_t)b * p.Hq + (size_t)g * G + h) * D + dim] = (f16)o;
        if (p.lse && dim == 0)
            p.lse[(size_t)b * p.Hq + (size_t)g * G + h] =
                den > 0.f ? (M + __log2f(den)) * 0.69314718055994531f : -INFINITY;
    }
}

}  // namespace apex
