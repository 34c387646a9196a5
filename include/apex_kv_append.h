/*
 * apex_kv_append.h -- C ABI of the paged KV-cache append (MI355X, gfx950).
 *
 * The operation.  Each decode iteration produces one new token per request,
 * and its Key and Value vectors are cached at every layer so that later
 * iterations reuse them instead of recomputing them (APEX, Sec. 2.1); the
 * cache is paged (Sec. 4.1) and holds, in GPU memory, the KV pairs of the
 * requests the GPU attends (Sec. 3.1).  Before the decode attention of
 * apex_decode.h reads a request with context_lens[b] = L_b tokens, the new
 * token's K/V must sit at position L_b - 1; this call puts it there:
 *
 *     for every t in [0, T) with 0 <= slot_mapping[t] < num_blocks * block_size,
 *     and every kv-head g:
 *         k_cache[slot / block_size][g][slot % block_size][:] = k_new[t][g][:]
 *         v_cache[slot / block_size][g][slot % block_size][:] = v_new[t][g][:]
 *
 * Other slots are left untouched.  A negative slot marks a padding token and
 * a slot at or past num_blocks * block_size is skipped as well, so the kernel
 * never writes outside the pool the caller described.
 *
 * Layouts (device memory, row-major, 16-byte aligned):
 *   k_new, v_new   fp16, token t / kv-head g / element i at
 *                  [t * new_token_stride + g * d + i]; new_token_stride is in
 *                  elements, 0 means Hkv * d (tight [T][Hkv][d]); a wider
 *                  stride reads K and V straight out of a fused projection
 *                  buffer.  Each must hold (T - 1) * stride + Hkv * d elements.
 *   k_cache,       fp16 [num_blocks][Hkv][block_size][d], the layout of
 *   v_cache        apex_decode.h
 *   slot_mapping   int64 [T], slot = physical block * block_size + position
 *
 * Supported: d a multiple of 8 up to 2048, any block_size >= 1 (the
 * attention reads block_size 16, d 128), T * Hkv < 2^31.  The slots of one
 * call must be distinct; with duplicates, which row ends up in the slot is
 * unspecified.
 *
 * Ownership and errors as in apex_decode.h: the caller owns every buffer,
 * the call validates on the host, enqueues one kernel on `stream` (NULL =
 * legacy default stream) and returns without synchronising; on failure it
 * enqueues nothing and apex_decode_last_error() says why.  T == 0 is a
 * successful no-op.
 */
#ifndef APEX_KV_APPEND_H
#define APEX_KV_APPEND_H

#include <stddef.h>
#include <stdint.h>

#include "apex_decode.h"

#ifdef __cplusplus
extern "C" {
#endif

int apex_kv_append(const void* k_new, const void* v_new, int64_t new_token_stride,
                   void* k_cache, void* v_cache, const int64_t* slot_mapping, int T, int Hkv,
                   int d, int block_size, int64_t num_blocks, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* APEX_KV_APPEND_H */
