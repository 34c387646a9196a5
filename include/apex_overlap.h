/*
 * apex_overlap.h -- C ABI of the Asynchronous Overlap runtime (MI355X +
 * host), in libapex_overlap.so.
 *
 * The mechanism (APEX, Sec. 3.3 "Asynchronous Overlap Mechanism" and
 * Sec. 4.2 "Asynchronous GPU-CPU Overlap Runtime").  Linear layers run once
 * per iteration on one unified GPU batch; after a layer's pre-attention
 * linears, the Q/K/V rows of the requests attended on the CPU are copied to
 * host memory while the GPU attends its own requests.  A dedicated compute
 * thread appends the new K/V rows to the host KV cache (pinned, Sec. 4.1)
 * and runs the host attention.  The result is not awaited: it is copied back
 * just before the post-attention linears of the same layer in the next
 * iteration, after a readiness check that never blocks -- if the CPU is not
 * done, the GPU carries on and the check is repeated in the following
 * iteration (Sec. 3.4, last paragraph).
 *
 * Use, per layer l and iteration:
 *   apex_overlap_submit(rt, l, q, k_new, v_new, slots, table, stride, lens,
 *                       B, stream, &ticket)   -- after the projections on `stream`
 *   ... later (next iteration) ...
 *   apex_overlap_poll(rt, ticket, out, stream, &ready)   -- non-blocking
 *   apex_overlap_wait(rt, ticket, out, stream)           -- blocking
 *
 * Device buffers (on the current device, fp16, contiguous):
 *   q [B][Hq][d]; k_new, v_new [B][Hkv][d] (this token's rows); out [B][Hq][d]
 *   When k_new starts right after q's B rows and v_new right after k_new's,
 *   the three are copied to the host as one transfer.
 * Host arrays (copied at submit, the caller may reuse them at once):
 *   slot_mapping int64 [B] (host cache slot of the new token: block *
 *   block_size + position, negative = no append), block_table int32
 *   [B][stride], context_lens int32 [B] (counts the new token).
 * The host KV cache of layer l ([num_blocks][Hkv][block_size][d] fp16, K and
 * V) is owned by the runtime (pinned, hipHostMalloc) and reachable through
 * apex_overlap_host_cache for filling it (e.g. with KV swapped out of the
 * GPU).  The compute thread appends to a layer's cache while that layer has
 * jobs pending (apex_overlap_pending, or after apex_overlap_hold): write into
 * it only when none is.  The attention is the one of apex_cpu_attention.h
 * (its supported set -- d a multiple of 16 up to 512, G <= 64 -- is checked
 * at create).
 *
 * Every layer has `slots_per_layer` result slots (default 2: one result in
 * flight while the next iteration submits).  A slot can be reused as soon as
 * its result has been collected by poll or wait: the new submit's copies are
 * ordered on the device after the copy-back of the previous result
 * (hipStreamWaitEvent), so the host never blocks.  Submitting into a slot
 * whose result has not been collected returns APEX_ERR_BUSY.  Calls on one
 * runtime must come from one host thread (the engine's main thread); the
 * compute thread is internal.
 *
 * Errors: apex_status codes of apex_decode.h, messages through
 * apex_overlap_last_error() (thread-local).  A failure of the host attention
 * or of a copy is reported by the poll/wait that collects that ticket.
 */
#ifndef APEX_OVERLAP_H
#define APEX_OVERLAP_H

#include <stddef.h>
#include <stdint.h>

#include "apex_decode.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct apex_overlap apex_overlap;

typedef struct apex_overlap_config {
    int layers;            /* layers sharing the runtime (one host KV cache each) */
    int max_requests;      /* largest B of one submit */
    int Hq, Hkv, d, block_size;
    float scale;
    int64_t num_blocks;    /* host KV cache blocks per layer */
    int max_blocks_per_request;   /* widest block-table row accepted */
    int threads;           /* host attention threads; 0 = the backend's pool size */
    int slots_per_layer;   /* result slots per layer; 0 = 2 */
} apex_overlap_config;

/* Allocates the pinned host caches and staging buffers, starts the compute thread. */
int apex_overlap_create(const apex_overlap_config* cfg, apex_overlap** out);

/* Host K and V cache of `layer` ([num_blocks][Hkv][block_size][d] fp16, pinned). */
int apex_overlap_host_cache(apex_overlap* rt, int layer, void** k_cache, void** v_cache);

/* Copies this layer's CPU-request rows to the host (ordered after the work
 * already on `stream`) and queues the append + host attention. */
int apex_overlap_submit(apex_overlap* rt, int layer, const void* q, const void* k_new,
                        const void* v_new, const int64_t* slot_mapping,
                        const int32_t* block_table, int64_t block_table_stride,
                        const int32_t* context_lens, int B, void* stream, int64_t* ticket);

/* Readiness check: if the ticket's result is ready, enqueues its copy into
 * `out` on `stream` and sets *ready = 1; otherwise sets *ready = 0 and
 * enqueues nothing.  Never blocks. */
int apex_overlap_poll(apex_overlap* rt, int64_t ticket, void* out, void* stream, int* ready);

/* Blocks until the ticket's result is ready, then enqueues its copy like poll. */
int apex_overlap_wait(apex_overlap* rt, int64_t ticket, void* out, void* stream);

/* Pauses (hold != 0) or resumes the compute thread between jobs. */
int apex_overlap_hold(apex_overlap* rt, int hold);

/* Jobs submitted and not yet finished by the compute thread. */
int apex_overlap_pending(apex_overlap* rt);

/* Finishes queued jobs, waits for outstanding copies, frees everything. */
int apex_overlap_destroy(apex_overlap* rt);

/* Message for the last failed call on this thread ("" if none). */
const char* apex_overlap_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* APEX_OVERLAP_H */
