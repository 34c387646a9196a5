/*
 * apex_cpu_attention.h -- C ABI of the host (CPU) paged decode-attention
 * backend.
 *
 * The operation is the one of apex_decode.h, computed by the host cores over
 * KV caches held in host memory.  APEX runs the attention of the requests it
 * offloads on the CPU, over their KV pairs kept in pinned host memory, with a
 * paged-attention kernel of its own built from matrix-multiplication kernels
 * (Sec. 4.1 "Integration of Llamafile Kernels"; Sec. 3.3 sends the new
 * token's Q/K/V of those requests to the host each layer).  Only where the
 * attention runs changes, not its mathematics (Sec. 3.1):
 *
 *     out[b][h] = sum_t softmax_t(scale * q[b][h] . K_t) * V_t,  t in [0, L_b)
 *
 * with the same paged layout and head grouping as apex_decode.h:
 *   q            fp16 [B][Hq][d]
 *   k_cache,     fp16 [num_blocks][Hkv][block_size][d]
 *   v_cache
 *   block_table  int32 [B][stride] (stride = block_table_stride, or
 *                ceil(max_b L_b / block_size) when 0)
 *   context_lens int32 [B]; counts the current token; L_b <= 0 gives a zero row
 *   out          fp16 [B][Hq][d], rounded to nearest even
 *   lse_out      optional fp32 [B][Hq], natural-log log-sum-exp of the scaled
 *                logits (-inf for L_b <= 0)
 * All pointers are HOST memory (pageable or pinned, e.g. hipHostMalloc).
 *
 * How it computes.  For every (request, kv-head) pair the G = Hq / Hkv query
 * rows form a G x d matrix; each block of up to block_size tokens is one
 * small matrix product for the scores (G x d times d x block_size), an online
 * softmax in fp32, and one small product for the values (G x block_size
 * times block_size x d), so every K/V row is read once for all G heads.
 * Pairs are cut into token chunks when there are fewer pairs than threads
 * can balance; chunks are merged with the log-sum-exp identity.  fp16 is
 * widened to fp32 on load; scores, softmax statistics and accumulators are
 * fp32.  The inner loops use AVX-512 (with F16C conversions) when the CPU has
 * it, else AVX2 + FMA + F16C; apex_cpu_isa() says which.
 *
 * Supported: d a multiple of 16 up to 512, block_size >= 1, Hq % Hkv == 0
 * with G <= 64.  Anything else returns APEX_ERR_UNSUPPORTED.
 *
 * Threads: a persistent pool owned by the library, sized on first use (or by
 * num_threads in apex_cpu_args); calls are synchronous -- they return when
 * the output is written -- and calls from several host threads are
 * serialised.  The calling thread takes part in the work.
 *
 * Errors: the apex_status codes of apex_decode.h; messages through
 * apex_cpu_last_error() (thread-local).  Block ids are not range-checked.
 */
#ifndef APEX_CPU_ATTENTION_H
#define APEX_CPU_ATTENTION_H

#include <stddef.h>
#include <stdint.h>

#include "apex_decode.h"   /* apex_status codes */

#ifdef __cplusplus
extern "C" {
#endif

/* Same arguments as apex_decode_attention, minus the stream; host pointers. */
int apex_cpu_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                              const int32_t* block_table, const int32_t* context_lens, void* out,
                              int B, int Hq, int Hkv, int d, int block_size, float scale);

typedef struct apex_cpu_args {
    const void* q;
    const void* k_cache;
    const void* v_cache;
    const int32_t* block_table;
    const int32_t* context_lens;
    void* out;
    int B, Hq, Hkv, d, block_size;
    float scale;
    /* entries per block_table row; 0 = ceil(max_b L_b / block_size) */
    int64_t block_table_stride;
    /* optional fp32 [B][Hq] */
    float* lse_out;
    /* threads taking part (including the caller); 0 = the pool's size */
    int num_threads;
    /* smallest token chunk a pair is cut into; 0 = library default (512) */
    int min_chunk_tokens;
    /* APEX_CPU_FLAG_* bits; other bits must be 0 */
    uint32_t flags;
} apex_cpu_args;

/* Use the AVX2 path even where AVX-512 is available (both paths stay testable). */
#define APEX_CPU_FLAG_FORCE_AVX2 1u

int apex_cpu_decode_attention_ex(const apex_cpu_args* args);

/* Resizes the thread pool (n >= 1; 0 = all cores the process may run on). */
int apex_cpu_set_threads(int n);

/* Threads in the pool (including the calling thread). */
int apex_cpu_threads(void);

/* SIMD path in use: 2 = AVX-512 + F16C, 1 = AVX2 + FMA + F16C, 0 = none. */
int apex_cpu_isa(void);

/* Host read bandwidth in GB/s: `threads` threads read a library-allocated
 * buffer of `bytes` bytes `reps` times (the host-memory roofline of the
 * backend).  Negative on failure. */
double apex_cpu_read_bandwidth(size_t bytes, int threads, int reps);

/* Message for the last failed call on this thread ("" if none). */
const char* apex_cpu_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* APEX_CPU_ATTENTION_H */
