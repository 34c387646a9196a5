// attend_simd.cpp -- inner loops of the host paged decode attention for one
// instruction set.  Built twice: with -mavx512f -mavx512bw -mavx512vl
// -mavx512dq -mf16c -mfma into namespace simd_avx512 (16-lane vectors) and
// with -mavx2 -mfma -mf16c into namespace simd_avx2 (8-lane vectors).
//
// Per (request, kv-head) range the G query rows are a G x d fp32 matrix kept
// in cache.  Tokens are taken in tiles of one vector width W (never crossing
// a cache block); the tile's K and V rows are widened to fp32 once into
// scratch.  Scores: per head, W accumulators (one per tile row) run over the
// d-chunks and are reduced together by one transposing sum, which yields the
// head's W scores as one vector.  The online softmax updates (m, l) per head
// and rescales that head's accumulator only when its running max grows.
// Values: per head, the W weights are broadcast once and the d-chunks of the
// accumulator are updated in independent groups.  Scores are kept in base 2
// (q is pre-scaled by scale * log2 e), so the exponentials are 2^x.
#include <immintrin.h>
#include <math.h>
#include <stdint.h>

#include "attend.h"

#ifndef APEX_SIMD_NS
#error "define APEX_SIMD_NS (simd_avx512 or simd_avx2)"
#endif

namespace apex_cpu {
namespace APEX_SIMD_NS {
namespace {

#if defined(__AVX512F__)

constexpr int W = 16;
typedef __m512 vf;
inline vf load_h(const uint16_t* p) { return _mm512_cvtph_ps(_mm256_loadu_si256((const __m256i*)p)); }
inline void store_h(uint16_t* p, vf x)
{
    _mm256_storeu_si256((__m256i*)p, _mm512_cvtps_ph(x, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC));
}
inline vf loadf(const float* p) { return _mm512_loadu_ps(p); }
inline void storef(float* p, vf x) { _mm512_storeu_ps(p, x); }
inline vf set1(float x) { return _mm512_set1_ps(x); }
inline vf zero() { return _mm512_setzero_ps(); }
inline vf fmadd(vf a, vf b, vf c) { return _mm512_fmadd_ps(a, b, c); }
inline vf mul(vf a, vf b) { return _mm512_mul_ps(a, b); }
inline vf sub(vf a, vf b) { return _mm512_sub_ps(a, b); }
inline vf vmax(vf a, vf b) { return _mm512_max_ps(a, b); }
inline float hsum(vf x) { return _mm512_reduce_add_ps(x); }
inline float hmax(vf x) { return _mm512_reduce_max_ps(x); }
inline vf round_nearest(vf x) { return _mm512_roundscale_ps(x, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC); }
// 2^n for integral n in [-127, 127]
inline vf pow2i(vf n) { return _mm512_scalef_ps(set1(1.0f), n); }
// lanes [0, n) of x, the others set to fill
inline vf first_n(vf x, int n, float fill)
{
    const __mmask16 k = (__mmask16)((1u << n) - 1u);
    return _mm512_mask_blend_ps(k, set1(fill), x);
}
// lane j of the result = sum of the lanes of a[j] (16 vectors): pairs are
// folded 256, 128, 64 and 32 bits at a time, so the 16 horizontal sums cost
// 15 adds and 30 shuffles.  The inputs are taken in the order that leaves
// the sums in natural lane order.
inline vf transpose_sum(const vf* a)
{
    vf x[16], t[8], w[4], e[2];
    for (int k = 0; k < 4; ++k)
        for (int c = 0; c < 4; ++c) x[4 * k + c] = a[4 * c + k];
    for (int k = 0; k < 8; ++k)
        t[k] = _mm512_add_ps(_mm512_shuffle_f32x4(x[2 * k], x[2 * k + 1], _MM_SHUFFLE(1, 0, 1, 0)),
                             _mm512_shuffle_f32x4(x[2 * k], x[2 * k + 1], _MM_SHUFFLE(3, 2, 3, 2)));
    for (int m = 0; m < 4; ++m)
        w[m] = _mm512_add_ps(_mm512_shuffle_f32x4(t[2 * m], t[2 * m + 1], _MM_SHUFFLE(2, 0, 2, 0)),
                             _mm512_shuffle_f32x4(t[2 * m], t[2 * m + 1], _MM_SHUFFLE(3, 1, 3, 1)));
    for (int q = 0; q < 2; ++q)
        e[q] = _mm512_add_ps(_mm512_shuffle_ps(w[2 * q], w[2 * q + 1], _MM_SHUFFLE(2, 0, 2, 0)),
                             _mm512_shuffle_ps(w[2 * q], w[2 * q + 1], _MM_SHUFFLE(3, 1, 3, 1)));
    return _mm512_add_ps(_mm512_shuffle_ps(e[0], e[1], _MM_SHUFFLE(2, 0, 2, 0)),
                         _mm512_shuffle_ps(e[0], e[1], _MM_SHUFFLE(3, 1, 3, 1)));
}

#elif defined(__AVX2__)

constexpr int W = 8;
typedef __m256 vf;
inline vf load_h(const uint16_t* p) { return _mm256_cvtph_ps(_mm_loadu_si128((const __m128i*)p)); }
inline void store_h(uint16_t* p, vf x)
{
    _mm_storeu_si128((__m128i*)p, _mm256_cvtps_ph(x, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC));
}
inline vf loadf(const float* p) { return _mm256_loadu_ps(p); }
inline void storef(float* p, vf x) { _mm256_storeu_ps(p, x); }
inline vf set1(float x) { return _mm256_set1_ps(x); }
inline vf zero() { return _mm256_setzero_ps(); }
inline vf fmadd(vf a, vf b, vf c) { return _mm256_fmadd_ps(a, b, c); }
inline vf mul(vf a, vf b) { return _mm256_mul_ps(a, b); }
inline vf sub(vf a, vf b) { return _mm256_sub_ps(a, b); }
inline vf vmax(vf a, vf b) { return _mm256_max_ps(a, b); }
inline float hsum(vf x)
{
    __m128 s = _mm_add_ps(_mm256_castps256_ps128(x), _mm256_extractf128_ps(x, 1));
    s = _mm_add_ps(s, _mm_movehl_ps(s, s));
    s = _mm_add_ss(s, _mm_movehdup_ps(s));
    return _mm_cvtss_f32(s);
}
inline float hmax(vf x)
{
    __m128 s = _mm_max_ps(_mm256_castps256_ps128(x), _mm256_extractf128_ps(x, 1));
    s = _mm_max_ps(s, _mm_movehl_ps(s, s));
    s = _mm_max_ss(s, _mm_movehdup_ps(s));
    return _mm_cvtss_f32(s);
}
inline vf round_nearest(vf x) { return _mm256_round_ps(x, _MM_FROUND_TO_NEAREST_INT | _MM_FROUND_NO_EXC); }
// 2^n for integral n in [-127, 127] (n = -127 gives 0)
inline vf pow2i(vf n)
{
    const __m256i e = _mm256_add_epi32(_mm256_cvtps_epi32(n), _mm256_set1_epi32(127));
    return _mm256_castsi256_ps(_mm256_slli_epi32(e, 23));
}
inline vf first_n(vf x, int n, float fill)
{
    const __m256i iota = _mm256_setr_epi32(0, 1, 2, 3, 4, 5, 6, 7);
    const __m256 keep = _mm256_castsi256_ps(_mm256_cmpgt_epi32(_mm256_set1_epi32(n), iota));
    return _mm256_blendv_ps(set1(fill), x, keep);
}
// lane j of the result = sum of the lanes of a[j] (8 vectors), folded 128,
// 64 and 32 bits at a time; inputs reordered so the sums land in lane order.
inline vf transpose_sum(const vf* a)
{
    vf x[8], t[4], w[2];
    for (int h = 0; h < 2; ++h)
        for (int k = 0; k < 4; ++k) x[2 * k + h] = a[4 * h + k];
    for (int k = 0; k < 4; ++k)
        t[k] = _mm256_add_ps(_mm256_permute2f128_ps(x[2 * k], x[2 * k + 1], 0x20),
                             _mm256_permute2f128_ps(x[2 * k], x[2 * k + 1], 0x31));
    for (int m = 0; m < 2; ++m)
        w[m] = _mm256_add_ps(_mm256_shuffle_ps(t[2 * m], t[2 * m + 1], _MM_SHUFFLE(2, 0, 2, 0)),
                             _mm256_shuffle_ps(t[2 * m], t[2 * m + 1], _MM_SHUFFLE(3, 1, 3, 1)));
    return _mm256_add_ps(_mm256_shuffle_ps(w[0], w[1], _MM_SHUFFLE(2, 0, 2, 0)),
                         _mm256_shuffle_ps(w[0], w[1], _MM_SHUFFLE(3, 1, 3, 1)));
}

#else
#error "attend_simd.cpp needs AVX-512F or AVX2"
#endif

// Coefficients of the Taylor series of 2^f = e^(f ln 2): c_k = (ln 2)^k / k!.
// On |f| <= 1/2 the first omitted term is below 2^-27 relative, under fp32
// rounding, so degree 7 is enough.
constexpr double kLn2 = 0.69314718055994530942;
constexpr float kC1 = (float)(kLn2);
constexpr float kC2 = (float)(kLn2 * kLn2 / 2);
constexpr float kC3 = (float)(kLn2 * kLn2 * kLn2 / 6);
constexpr float kC4 = (float)(kLn2 * kLn2 * kLn2 * kLn2 / 24);
constexpr float kC5 = (float)(kLn2 * kLn2 * kLn2 * kLn2 * kLn2 / 120);
constexpr float kC6 = (float)(kLn2 * kLn2 * kLn2 * kLn2 * kLn2 * kLn2 / 720);
constexpr float kC7 = (float)(kLn2 * kLn2 * kLn2 * kLn2 * kLn2 * kLn2 * kLn2 / 5040);

// 2^x for x <= 0 (x below -127 gives 0 or a subnormal): x = n + f with n the
// nearest integer, 2^f from the series above, times 2^n.
inline vf exp2v(vf x)
{
    x = vmax(x, set1(-127.0f));
    const vf n = round_nearest(x);
    const vf f = sub(x, n);
    vf p = set1(kC7);
    p = fmadd(p, f, set1(kC6));
    p = fmadd(p, f, set1(kC5));
    p = fmadd(p, f, set1(kC4));
    p = fmadd(p, f, set1(kC3));
    p = fmadd(p, f, set1(kC2));
    p = fmadd(p, f, set1(kC1));
    p = fmadd(p, f, set1(1.0f));
    return mul(p, pow2i(n));
}

// acc[h0 + i][:] += sum_j w[h0 + i][j] * V_j for HB heads, CB d-chunks at a
// time: HB x CB accumulators stay in registers while each V chunk is widened
// once and used by the HB heads.
template <int HB, int CB>
inline void pv_block(const uint16_t* vr, int n, int d, const float* pw, int h0, float* acc,
                     int c_begin, int c_end)
{
    for (int c0 = c_begin; c0 + CB <= c_end; c0 += CB) {
        vf a[HB][CB];
        for (int i = 0; i < HB; ++i)
            for (int u = 0; u < CB; ++u) a[i][u] = loadf(acc + (int64_t)(h0 + i) * d + (c0 + u) * W);
        for (int j = 0; j < n; ++j) {
            vf v[CB];
            for (int u = 0; u < CB; ++u) v[u] = load_h(vr + (int64_t)j * d + (c0 + u) * W);
            for (int i = 0; i < HB; ++i) {
                const vf w = set1(pw[(h0 + i) * 16 + j]);
                for (int u = 0; u < CB; ++u) a[i][u] = fmadd(w, v[u], a[i][u]);
            }
        }
        for (int i = 0; i < HB; ++i)
            for (int u = 0; u < CB; ++u) storef(acc + (int64_t)(h0 + i) * d + (c0 + u) * W, a[i][u]);
    }
}

// Partial score vectors of a full tile (all W rows valid): for HB heads and
// TB rows at a time, HB x TB accumulators run over the d-chunks with each K
// chunk widened once in registers; the accumulators go to sacc[h][j] for the
// transposing sum.
template <int HB, int TB>
inline void qk_block(const uint16_t* kr, int d, const float* qs, int h0, vf* sacc)
{
    const int dc = d / W;
    for (int j0 = 0; j0 < W; j0 += TB) {
        vf a[HB][TB];
        for (int i = 0; i < HB; ++i)
            for (int t = 0; t < TB; ++t) a[i][t] = zero();
        for (int c = 0; c < dc; ++c) {
            vf k[TB];
            for (int t = 0; t < TB; ++t) k[t] = load_h(kr + (int64_t)(j0 + t) * d + c * W);
            for (int i = 0; i < HB; ++i) {
                const vf q = loadf(qs + (int64_t)(h0 + i) * d + c * W);
                for (int t = 0; t < TB; ++t) a[i][t] = fmadd(q, k[t], a[i][t]);
            }
        }
        for (int i = 0; i < HB; ++i)
            for (int t = 0; t < TB; ++t) sacc[(h0 + i) * W + j0 + t] = a[i][t];
    }
}

// accumulators per register block of the score update
constexpr int kQkAcc = W == 16 ? 16 : 8;

// register block of the value update: heads x d-chunks accumulators (16 of
// the 32 zmm registers with AVX-512, 8 of the 16 ymm registers with AVX2)
constexpr int kPvHeads = W == 16 ? 4 : 2;
constexpr int kPvChunks = 4;

template <int HB>
inline void pv_heads(const uint16_t* vr, int n, int d, const float* pw, int h0, float* acc)
{
    const int dc = d / W;
    const int full = dc / kPvChunks * kPvChunks;
    pv_block<HB, kPvChunks>(vr, n, d, pw, h0, acc, 0, full);
    pv_block<HB, 1>(vr, n, d, pw, h0, acc, full, dc);
}

// attend() for GT heads of dimension DT (0 = the values in p): the common
// shapes get compile-time trip counts, so the head and chunk loops unroll and
// the heads' softmax chains can overlap.
template <int GT, int DT>
inline void attend_impl(const Problem& p, int b, int g, int t0, int t1, State st, float* scratch)
{
    const int G = GT > 0 ? GT : p.G, d = DT > 0 ? DT : p.d, dc = d / W;
    float* qs = scratch;                   // [G][d] query rows, pre-scaled
    float* pw = qs + (int64_t)G * d;       // [G][16] weights of the tile
    float* kt = pw + (int64_t)G * 16;      // [W][d] K tile widened to fp32 (partial tiles)
    // [G][W] partial score vectors, 64-byte aligned
    vf* sacc = (vf*)(((uintptr_t)(kt + (int64_t)W * d) + 63) & ~(uintptr_t)63);
    const uint16_t* qrow = p.q + ((int64_t)b * p.Hq + (int64_t)g * G) * d;
    const vf qscale = set1(p.scale_log2);
    for (int h = 0; h < G; ++h) {
        st.m[h] = -INFINITY;
        st.l[h] = 0.0f;
        for (int c = 0; c < dc; ++c) {
            storef(qs + (int64_t)h * d + c * W, mul(load_h(qrow + (int64_t)h * d + c * W), qscale));
            storef(st.acc + (int64_t)h * d + c * W, zero());
        }
    }
    const int32_t* row = p.block_table + (int64_t)b * p.stride;
    const int bs = p.bs;
    int t = t0;
    while (t < t1) {
        const int bi = t / bs;
        const int pos = t - bi * bs;
        int n = bs - pos;
        if (n > t1 - t) n = t1 - t;
        if (n > W) n = W;
        const int64_t phys = row[bi];
        const int64_t off = ((phys * p.Hkv + g) * bs + pos) * (int64_t)d;
        const uint16_t* kr = p.k + off;
        const uint16_t* vr = p.v + off;
        if (pos == 0 && t + bs < t1) {
            // the next block is a different physical block: start its lines early
            const int64_t nphys = row[bi + 1];
            const int64_t noff = (nphys * p.Hkv + g) * (int64_t)bs * d;
            const int64_t nbytes = (int64_t)bs * d * 2;
            for (int64_t x = 0; x < nbytes; x += 64) {
                _mm_prefetch((const char*)(p.k + noff) + x, _MM_HINT_T0);
                _mm_prefetch((const char*)(p.v + noff) + x, _MM_HINT_T0);
            }
        }
        if (n == W) {
            // full tile: register-blocked scores straight from the fp16 rows
            int h0 = 0;
            for (; h0 + 4 <= G; h0 += 4) qk_block<4, kQkAcc / 4>(kr, d, qs, h0, sacc);
            for (; h0 + 2 <= G; h0 += 2) qk_block<2, kQkAcc / 2>(kr, d, qs, h0, sacc);
            for (; h0 < G; ++h0) qk_block<1, kQkAcc>(kr, d, qs, h0, sacc);
        } else {
            // partial tile (end of a block or of the range): widen the n valid
            // K rows once, zero the rest, then one accumulator per row
            for (int j = 0; j < n; ++j)
                for (int c = 0; c < dc; ++c) storef(kt + (int64_t)j * d + c * W, load_h(kr + (int64_t)j * d + c * W));
            for (int j = n; j < W; ++j)
                for (int c = 0; c < dc; ++c) storef(kt + (int64_t)j * d + c * W, zero());
            for (int h = 0; h < G; ++h) {
                const float* qh = qs + (int64_t)h * d;
                vf acc[W];
                for (int j = 0; j < W; ++j) acc[j] = zero();
                for (int c = 0; c < dc; ++c) {
                    const vf qv = loadf(qh + c * W);
                    for (int j = 0; j < W; ++j) acc[j] = fmadd(qv, loadf(kt + (int64_t)j * d + c * W), acc[j]);
                }
                for (int j = 0; j < W; ++j) sacc[h * W + j] = acc[j];
            }
        }
        for (int h = 0; h < G; ++h) {
            const vf s = first_n(transpose_sum(sacc + h * W), n, -INFINITY);
            // online softmax
            const float mx = hmax(s);
            if (mx > st.m[h]) {
                const float alpha = st.m[h] == -INFINITY ? 0.0f : exp2f(st.m[h] - mx);
                st.l[h] *= alpha;
                const vf av = set1(alpha);
                float* ah = st.acc + (int64_t)h * d;
                for (int c = 0; c < dc; ++c) storef(ah + c * W, mul(loadf(ah + c * W), av));
                st.m[h] = mx;
            }
            const vf w = first_n(exp2v(sub(s, set1(st.m[h]))), n, 0.0f);
            st.l[h] += hsum(w);
            storef(pw + h * 16, w);
        }
        // values: acc[h] += sum_j w[h][j] * V_j
        int h0 = 0;
        for (; h0 + kPvHeads <= G; h0 += kPvHeads) pv_heads<kPvHeads>(vr, n, d, pw, h0, st.acc);
        for (; h0 < G; ++h0) pv_heads<1>(vr, n, d, pw, h0, st.acc);
        t += n;
    }
}

}  // namespace

void attend(const Problem& p, int b, int g, int t0, int t1, State st, float* scratch)
{
    if (p.d == 128) {
        switch (p.G) {
            case 1: return attend_impl<1, 128>(p, b, g, t0, t1, st, scratch);
            case 2: return attend_impl<2, 128>(p, b, g, t0, t1, st, scratch);
            case 4: return attend_impl<4, 128>(p, b, g, t0, t1, st, scratch);
            case 8: return attend_impl<8, 128>(p, b, g, t0, t1, st, scratch);
            default: break;
        }
    }
    attend_impl<0, 0>(p, b, g, t0, t1, st, scratch);
}

void finish(const float* m, const float* l, const float* acc, int G, int d, uint16_t* out, float* lse)
{
    const int dc = d / W;
    for (int h = 0; h < G; ++h) {
        const vf inv = set1(1.0f / l[h]);
        for (int c = 0; c < dc; ++c)
            store_h(out + (int64_t)h * d + c * W, mul(loadf(acc + (int64_t)h * d + c * W), inv));
        if (lse) lse[h] = (float)(((double)m[h] + log2((double)l[h])) * kLn2);
    }
}

void merge(const float* const* m, const float* const* l, const float* const* acc, int n, int G,
           int d, float* m_out, float* l_out, float* acc_out)
{
    const int dc = d / W;
    for (int h = 0; h < G; ++h) {
        float M = -INFINITY;
        for (int s = 0; s < n; ++s) M = m[s][h] > M ? m[s][h] : M;
        float* oh = acc_out + (int64_t)h * d;
        for (int c = 0; c < dc; ++c) storef(oh + c * W, zero());
        float L = 0.0f;
        for (int s = 0; s < n; ++s) {
            if (m[s][h] == -INFINITY) continue;   // an empty range
            const float w = exp2f(m[s][h] - M);
            L += w * l[s][h];
            const vf wv = set1(w);
            const float* ah = acc[s] + (int64_t)h * d;
            for (int c = 0; c < dc; ++c) storef(oh + c * W, fmadd(wv, loadf(ah + c * W), loadf(oh + c * W)));
        }
        m_out[h] = M;
        l_out[h] = L;
    }
}

}  // namespace APEX_SIMD_NS
}  // namespace apex_cpu
