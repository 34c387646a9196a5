/*
 * oracle/ref_decode.c -- fp64 CPU oracle for batched paged decode attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark load it.  It shares no code, header, table or helper with
 * the HIP path.
 *
 * What it computes (APEX, Sec. 3.1 "System Overview" and Sec. 3.3
 * "Asynchronous Overlap"): in the decode phase every request contributes one
 * new query token per iteration, and the GPU performs self-attention for the
 * requests assigned to it, over their KV pairs held in GPU memory; APEX moves
 * attention between devices without changing the mathematics or the
 * precision.  Sec. 4.1 states that the KV cache is paged.  The paper never
 * writes the attention formula down; the oracle uses the standard
 * scaled-dot-product softmax attention of the attention works it cites
 * (Sec. 2.1), with no masking beyond the request's length:
 *
 *     z_t   = scale * sum_i q[b][h][i] * K_t[i]          t in [0, L_b)
 *     w_t   = exp(z_t - max_t z_t) / sum_t exp(z_t - max_t z_t)
 *     out   = sum_t w_t * V_t
 *     lse   = max_t z_t + log(sum_t exp(z_t - max_t z_t))
 *
 * It is the plain definition: two passes over the tokens, no splitting, no
 * online rescaling, no blocking.  Readings where the paper is silent:
 *   - K/V cache layout [num_blocks][Hkv][block_size][d], token t of request b
 *     lives in physical block block_table[b*stride + t/block_size] at slot
 *     t % block_size;
 *   - q-head h reads kv-head h / (Hq/Hkv) (consecutive grouping);
 *   - context_lens[b] counts the current token; L_b <= 0 gives a zero row
 *     (softmax over an empty set is undefined) and lse = -inf;
 *   - the scale is the fp32 value passed in, widened to fp64.
 *
 * fp16 inputs are decoded with f16_to_f64 below, written from the IEEE-754
 * binary16 definition (1 sign bit, 5 exponent bits with bias 15, 10 fraction
 * bits; exponent 0 = zero/subnormal, exponent 31 = Inf/NaN).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

double apex_oracle_f16_to_f64(uint16_t bits)
{
    const int sign = (bits >> 15) & 1;
    const int expo = (bits >> 10) & 0x1f;
    const int frac = bits & 0x3ff;
    double mag;
    if (expo == 0) {
        mag = ldexp((double)frac, -24);               /* 0.frac * 2^-14 */
    } else if (expo == 31) {
        mag = frac ? NAN : INFINITY;
    } else {
        mag = ldexp((double)(1024 + frac), expo - 25); /* 1.frac * 2^(e-15) */
    }
    return sign ? -mag : mag;
}

void apex_oracle_f16_to_f64_array(const uint16_t* in, double* out, size_t n)
{
    for (size_t i = 0; i < n; ++i) out[i] = apex_oracle_f16_to_f64(in[i]);
}

/* Address (in elements) of K/V row for token t of request b, kv-head g. */
static size_t kv_row(const int32_t* block_table, long stride, int b, int t,
                     int g, int Hkv, int block_size, int d)
{
    const int32_t blk = block_table[(size_t)b * (size_t)stride + (size_t)(t / block_size)];
    const int slot = t % block_size;
    return (((size_t)blk * (size_t)Hkv + (size_t)g) * (size_t)block_size + (size_t)slot) * (size_t)d;
}

/*
 * One (request, q-head) pair.  w must hold L doubles of scratch.  On return
 * w[t] holds the normalised softmax weight of token t.
 */
static void attend_one(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                       const int32_t* block_table, long stride, int L,
                       int b, int h, int Hq, int Hkv, int d, int block_size, double scale,
                       double* w, double* out_row, double* lse_out)
{
    const int group = Hq / Hkv;
    const int g = h / group;
    const uint16_t* qrow = q + ((size_t)b * (size_t)Hq + (size_t)h) * (size_t)d;

    for (int i = 0; i < d; ++i) out_row[i] = 0.0;
    if (L <= 0) {
        if (lse_out) *lse_out = -INFINITY;
        return;
    }

    /* pass 1: logits and their maximum */
    double zmax = -INFINITY;
    for (int t = 0; t < L; ++t) {
        const uint16_t* krow = k_cache + kv_row(block_table, stride, b, t, g, Hkv, block_size, d);
        double dot = 0.0;
        for (int i = 0; i < d; ++i)
            dot += apex_oracle_f16_to_f64(qrow[i]) * apex_oracle_f16_to_f64(krow[i]);
        w[t] = scale * dot;
        if (w[t] > zmax) zmax = w[t];
    }

    /* pass 2: exponentials, normaliser, weighted sum of values */
    double Z = 0.0;
    for (int t = 0; t < L; ++t) {
        w[t] = exp(w[t] - zmax);
        Z += w[t];
    }
    for (int t = 0; t < L; ++t) {
        w[t] /= Z;
        const uint16_t* vrow = v_cache + kv_row(block_table, stride, b, t, g, Hkv, block_size, d);
        for (int i = 0; i < d; ++i) out_row[i] += w[t] * apex_oracle_f16_to_f64(vrow[i]);
    }
    if (lse_out) *lse_out = zmax + log(Z);
}

/*
 * Decode attention for a whole batch.
 *   q            fp16 bits [B][Hq][d]
 *   k_cache      fp16 bits [num_blocks][Hkv][block_size][d]
 *   v_cache      same layout as k_cache
 *   block_table  int32 [B][stride]
 *   context_lens int32 [B]
 *   out          double [B][Hq][d]
 *   lse          double [B][Hq] or NULL (natural log)
 * Returns 0, or -1 on an invalid shape.
 */
int apex_oracle_decode_attention_f64(const uint16_t* q, const uint16_t* k_cache,
                                     const uint16_t* v_cache, const int32_t* block_table,
                                     long block_table_stride, const int32_t* context_lens,
                                     int B, int Hq, int Hkv, int d, int block_size, float scale,
                                     double* out, double* lse, int num_threads)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || block_size <= 0)
        return -1;
    int maxL = 0;
    for (int b = 0; b < B; ++b)
        if (context_lens[b] > maxL) maxL = context_lens[b];
    const long pairs = (long)B * (long)Hq;
    int failed = 0;
#ifdef _OPENMP
    if (num_threads <= 0) num_threads = omp_get_max_threads();
#pragma omp parallel num_threads(num_threads) reduction(| : failed)
#endif
    {
        double* w = (double*)malloc(sizeof(double) * (size_t)(maxL > 0 ? maxL : 1));
        if (!w) {
            failed = 1;
        } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
            for (long p = 0; p < pairs; ++p) {
                const int b = (int)(p / Hq), h = (int)(p % Hq);
                attend_one(q, k_cache, v_cache, block_table, block_table_stride, context_lens[b],
                           b, h, Hq, Hkv, d, block_size, (double)scale, w,
                           out + (size_t)p * (size_t)d, lse ? lse + p : NULL);
            }
            free(w);
        }
    }
    return failed ? -1 : 0;
}

/*
 * Softmax weights of one (request, q-head): w[0..L) with L = context_lens[b].
 * Exposed so that tests can check that the weights sum to one.
 */
int apex_oracle_softmax_weights_f64(const uint16_t* q, const uint16_t* k_cache,
                                    const uint16_t* v_cache, const int32_t* block_table,
                                    long block_table_stride, const int32_t* context_lens,
                                    int b, int h, int Hq, int Hkv, int d, int block_size,
                                    float scale, double* w)
{
    if (Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || block_size <= 0) return -1;
    double* row = (double*)malloc(sizeof(double) * (size_t)d);
    if (!row) return -1;
    attend_one(q, k_cache, v_cache, block_table, block_table_stride, context_lens[b], b, h, Hq,
               Hkv, d, block_size, (double)scale, w, row, NULL);
    free(row);
    return 0;
}

int apex_oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
