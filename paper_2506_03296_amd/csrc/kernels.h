// kernels.h -- gfx950 kernel of batched paged decode attention.
//
// One call = one launch of attn_kernel<G> on a persistent grid of W work
// groups (4 waves each).  Every work group
//   1. reads context_lens and derives the partition of plan_policy.h on its
//      own (block sums, a prefix scan, the longest request for the tight
//      block-table stride), so no planner kernel runs before it;
//   2. walks its contiguous range of (request b, kv-head g, block) units
//      segment by segment.  In a segment the four waves take the blocks of
//      one (b, g) pair round-robin; per 16-token block a wave gathers the
//      paged K/V rows with 128-bit loads (prefetching its next block),
//      computes the G q-heads' scores as S^T = K Q^T with four
//      16x16x32 fp16 MFMAs (q-heads padded to 16 columns), runs an online
//      softmax (running max and sum in base 2, log2(e) folded into the
//      scale), and accumulates O^T += V^T P^T in fp32 with eight 16x16x16
//      fp16 MFMAs, V^T being assembled in registers with byte permutes;
//   3. merges the waves' states in LDS and either writes the fp16 output rows
//      (the segment is the whole pair) or stores an fp32 partial
//      (accumulator, max, sum) and bumps the pair's arrival counter; the last
//      work group to arrive combines the pair's partials and writes the rows.
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

struct AttnParams {
    const f16* q;          // [B][Hq][D]
    const f16* k;          // [NB][Hkv][BS][D]
    const f16* v;
    const int32_t* bt;     // [B][stride]
    const int32_t* lens;   // [B]
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

__device__ inline int uniform(int x)
{
    return __builtin_amdgcn_readfirstlane(x);
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

// One 16-token block of one kv-head, as the MFMA operands want it.
//   K: lane (t = lane % 16, q = lane / 16), word j = token t, dims [32j + 8q, +8)
//   V: lane (c = lane % 16, q = lane / 16), word e = token 4q + e, dims [8c, 8c + 8)
struct KVTile {
    u32x4 k[4];
    u32x4 v[4];
};

__device__ inline void load_tile(KVTile& t, const f16* kb, const f16* vb, int lane)
{
    const int col = lane & 15, q = lane >> 4;
    const f16* kp = kb + col * kHeadDim + 8 * q;
    const f16* vp = vb + (4 * q) * kHeadDim + 8 * col;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        t.k[i] = *(const u32x4*)(kp + 32 * i);
        t.v[i] = *(const u32x4*)(vp + i * kHeadDim);
    }
}

// Online-softmax state of one wave.  Lane (h = lane % 16, q = lane / 16):
// m = running max of head h (log2 units, equal on the four lanes of h),
// l = running sum of the weights of the lane's tokens, acc[t][i] = running
// P.V of head h at dim 32q + 8i + t.
struct WaveState {
    float m, l;
    f32x4 acc[8];
};

// Scores, online softmax and P.V of one block.  tok0 = first token of the
// block; tokens at or past L are masked (their V rows may hold anything).
template <int G>
__device__ inline void attend_tile(WaveState& st, KVTile& t, const f16x8 (&qop)[4], int tok0, int L,
                                   float scale_log2, int lane)
{
    const int q = lane >> 4;
    // S^T = K Q^T: lane (h, q) gets the scores of tokens 4q..4q+3 for head h
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i)
        s = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, t.k[i]), qop[i], s, 0, 0, 0);

    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) sv[i] = s[i] * scale_log2;
    if (tok0 + kBlockSize > L) {   // last, partial block of the pair
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (tok0 + 4 * q + i >= L) {
                sv[i] = -INFINITY;
                t.v[i] = u32x4{0u, 0u, 0u, 0u};
            }
        }
    }

    float bm = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    bm = fmaxf(bm, wave_shfl_xor(bm, 16));
    bm = fmaxf(bm, wave_shfl_xor(bm, 32));
    const float mnew = fmaxf(st.m, bm);   // finite: the block holds a valid token
    const float alpha = exp2_fast(st.m - mnew);
    f32x4 pw;
#pragma unroll
    for (int i = 0; i < 4; ++i) pw[i] = exp2_fast(sv[i] - mnew);
    const f16x4 ph = __builtin_convertvector(pw, f16x4);
    // the normaliser uses the same fp16-rounded weights as the numerator
    const float psum = ((float)ph[0] + (float)ph[1]) + ((float)ph[2] + (float)ph[3]);
    st.l = st.l * alpha + psum;
    if (alpha != 1.f) {
#pragma unroll
        for (int tt = 0; tt < 8; ++tt) st.acc[tt] *= alpha;
    }
    st.m = mnew;

    // O^T += V^T P^T, eight 16-dim tiles; tile tt row c is dim 8c + tt
#pragma unroll
    for (int tt = 0; tt < 8; ++tt) {
        const int w = tt >> 1;
        const unsigned sel = (tt & 1) ? kHiHalves : kLoHalves;
        unsigned a0, a1;
        switch (w) {
            case 0: a0 = pack_halves(t.v[0].x, t.v[1].x, sel); a1 = pack_halves(t.v[2].x, t.v[3].x, sel); break;
            case 1: a0 = pack_halves(t.v[0].y, t.v[1].y, sel); a1 = pack_halves(t.v[2].y, t.v[3].y, sel); break;
            case 2: a0 = pack_halves(t.v[0].z, t.v[1].z, sel); a1 = pack_halves(t.v[2].z, t.v[3].z, sel); break;
            default: a0 = pack_halves(t.v[0].w, t.v[1].w, sel); a1 = pack_halves(t.v[2].w, t.v[3].w, sel); break;
        }
        typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 a = {a0, a1};
        st.acc[tt] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a), ph, st.acc[tt], 0, 0, 0);
    }
}

// Per-wave attention over blocks lo + wave, lo + wave + 4, ... < hi of pair
// (b, g).  On return the wave's state is in s_acc/s_m/s_l.
template <int G>
__device__ inline void wave_attend(const AttnParams& p, const int32_t* bt_row, int b, int g, int L,
                                   int lo, int hi, int wave, int lane, float (*s_acc)[G][kHeadDim],
                                   float (*s_m)[G], float (*s_l)[G])
{
    constexpr int D = kHeadDim;
    constexpr int BS = kBlockSize;
    const int col = lane & 15;
    const int q = lane >> 4;

    // Q^T operand: lane (h, q) holds head h's dims [32i + 8q, +8) for MFMA i;
    // columns past the group are zero
    f16x8 qop[4];
    if (col < G) {
        const f16* qrow = p.q + ((size_t)b * p.Hq + (size_t)g * G + col) * D + 8 * q;
#pragma unroll
        for (int i = 0; i < 4; ++i) qop[i] = *(const f16x8*)(qrow + 32 * i);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) qop[i] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }

    WaveState st;
    st.m = -INFINITY;
    st.l = 0.f;
#pragma unroll
    for (int tt = 0; tt < 8; ++tt) st.acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const size_t head_off = (size_t)g * (BS * D);
    const size_t blk_elems = (size_t)p.Hkv * BS * D;
    KVTile ta, tb;
    int j = lo + wave;
    if (j < hi) {
        const size_t base = (size_t)uniform(bt_row[j]) * blk_elems + head_off;
        load_tile(ta, p.k + base, p.v + base, lane);
    }
    while (j < hi) {
        int jn = j + kWaves;
        if (jn < hi) {
            const size_t base = (size_t)uniform(bt_row[jn]) * blk_elems + head_off;
            load_tile(tb, p.k + base, p.v + base, lane);
        }
        attend_tile<G>(st, ta, qop, j * BS, L, p.scale_log2, lane);
        j = jn;
        if (j >= hi) break;
        jn = j + kWaves;
        if (jn < hi) {
            const size_t base = (size_t)uniform(bt_row[jn]) * blk_elems + head_off;
            load_tile(ta, p.k + base, p.v + base, lane);
        }
        attend_tile<G>(st, tb, qop, j * BS, L, p.scale_log2, lane);
        j = jn;
    }

    // the wave's state for head h: l summed over the four token groups
    float lw = st.l + wave_shfl_xor(st.l, 16);
    lw += wave_shfl_xor(lw, 32);
    if (col < G) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float* dst = &s_acc[wave][col][32 * q + 8 * i];
            *(f32x4*)dst = f32x4{st.acc[0][i], st.acc[1][i], st.acc[2][i], st.acc[3][i]};
            *(f32x4*)(dst + 4) = f32x4{st.acc[4][i], st.acc[5][i], st.acc[6][i], st.acc[7][i]};
        }
        if (q == 0) {
            s_m[wave][col] = st.m;
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

template <int G>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2))) void attn_kernel(AttnParams p)
{
    constexpr int D = kHeadDim;
    __shared__ float s_acc[kWaves][G][D];
    __shared__ float s_m[kWaves][G];
    __shared__ float s_l[kWaves][G];
    __shared__ int s_scan[kAttnThreads];
    __shared__ int s_maxb;
    __shared__ int s_loc_b;
    __shared__ int64_t s_loc_pre;
    __shared__ int s_last;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t w = blockIdx.x;
    const int B = p.B;

    // rows of empty requests are zeros (and lse = -inf)
    for (int b = (int)w; b < B; b += (int)gridDim.x) {
        if (p.lens[b] <= 0) {
            for (int i = tid; i < p.Hq * D; i += kAttnThreads) write_row(p, b, i / D, i % D, 0.f, 0.f, 0.f);
        }
    }

    // 1. partition: block sums per thread segment, scan, longest request
    const int seg = (B + kAttnThreads - 1) / kAttnThreads;
    const int r0 = min(B, tid * seg);
    const int r1 = min(B, r0 + seg);
    int tsum = 0, tmax = 0;
    for (int b = r0; b < r1; ++b) {
        const int nb = (int)blocks_of(p.lens[b], kBlockSize);
        tsum += nb;
        tmax = max(tmax, nb);
    }
    if (tid == 0) s_maxb = 0;
    s_scan[tid] = tsum;
    __syncthreads();
    atomicMax(&s_maxb, tmax);
    for (int off = 1; off < kAttnThreads; off <<= 1) {
        const int v = tid >= off ? s_scan[tid - off] : 0;
        __syncthreads();
        s_scan[tid] += v;
        __syncthreads();
    }
    const int64_t units = (int64_t)s_scan[kAttnThreads - 1] * p.Hkv;
    const int64_t stride = p.bt_stride > 0 ? p.bt_stride : (int64_t)s_maxb;
    const int64_t W = active_workers(units, (int64_t)gridDim.x, p.min_units);
    if (w >= W || units == 0) return;
    const int64_t u0 = worker_start(w, units, W);
    const int64_t u1 = worker_start(w + 1, units, W);
    if (u0 >= u1) return;

    // locate the pair holding unit u0
    {
        const int64_t excl = s_scan[tid] - tsum;
        if (excl * p.Hkv <= u0 && u0 < (int64_t)s_scan[tid] * p.Hkv) {
            int64_t pre = excl;
            for (int b = r0; b < r1; ++b) {
                const int64_t nb = blocks_of(p.lens[b], kBlockSize);
                if (u0 < (pre + nb) * p.Hkv) {
                    s_loc_b = b;
                    s_loc_pre = pre;
                    break;
                }
                pre += nb;
            }
        }
    }
    __syncthreads();

    int b = uniform(s_loc_b);
    int64_t pre = s_loc_pre;
    int L = uniform(p.lens[b]);
    int nb = (int)blocks_of(L, kBlockSize);
    int64_t off = u0 - pre * p.Hkv;
    int g = (int)(off / nb);
    int blk = (int)(off % nb);
    int64_t u = u0;

    // 2. segments
    while (true) {
        const int take = (int)min((int64_t)(nb - blk), u1 - u);
        const int lo = blk, hi = blk + take;
        const int32_t* bt_row = p.bt + (size_t)b * (size_t)stride;
        wave_attend<G>(p, bt_row, b, g, L, lo, hi, wave, lane, s_acc, s_m, s_l);
        __syncthreads();

        // 3. merge the waves, emit rows or a partial
        const int64_t p0 = pre * p.Hkv + (int64_t)g * nb;
        const int64_t wf = worker_of(p0, units, W);
        const int64_t wl = worker_of(p0 + nb - 1, units, W);
        const int64_t slot = partial_slot(w, p0, units, W);
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
                for (int idx = tid; idx < G * D; idx += kAttnThreads) {
                    const int h = idx / D, dim = idx % D;
                    float M = -INFINITY;
                    for (int64_t q = wf; q <= wl; ++q) {
                        const int64_t sq = partial_slot(q, p0, units, W);
                        M = fmaxf(M, load_coherent(&p.pml[((size_t)sq * G + h) * 2]));
                    }
                    const float Ms = M == -INFINITY ? 0.f : M;
                    float num = 0.f, den = 0.f;
                    for (int64_t q = wf; q <= wl; ++q) {
                        const int64_t sq = partial_slot(q, p0, units, W);
                        const float f = exp2_fast(load_coherent(&p.pml[((size_t)sq * G + h) * 2]) - Ms);
                        num = fmaf(f, load_coherent(&p.pacc[((size_t)sq * G + h) * D + dim]), num);
                        den = fmaf(f, load_coherent(&p.pml[((size_t)sq * G + h) * 2 + 1]), den);
                    }
                    write_row(p, b, g * G + h, dim, M, num, den);
                }
            }
        }
        __syncthreads();

        u += take;
        if (u >= u1) break;
        blk = hi;
        if (blk == nb) {
            blk = 0;
            if (++g == p.Hkv) {
                g = 0;
                pre += nb;
                do {
                    ++b;
                } while (b < B && p.lens[b] <= 0);
                if (b >= B) break;   // unreachable: units remain after the current pair
                L = uniform(p.lens[b]);
                nb = (int)blocks_of(L, kBlockSize);
            }
        }
    }
}

}  // namespace apex
