/*
 * apex_decode.h -- C ABI of the MI355X (gfx950) batched paged decode-attention
 * library.
 *
 * The operation.  In the decode phase each request contributes one query
 * token per iteration, and the GPU performs self-attention for the requests
 * assigned to it over their KV pairs resident in GPU memory (APEX, Sec. 3.1
 * "System Overview" and Sec. 3.3 "Asynchronous Overlap Mechanism"); the KV
 * cache is paged (Sec. 4.1) and the bandwidth-bound nature of this decode
 * attention is what APEX's placement decisions revolve around (Sec. 2.2).
 * APEX changes only where attention runs, never its mathematics (Sec. 3.1).
 * For request b with L_b = context_lens[b] cached tokens and q-head h:
 *
 *     out[b][h] = sum_t softmax_t(scale * q[b][h] . K_t) * V_t,  t in [0, L_b)
 *
 * where token t lives in physical block block_table[b][t / block_size] at slot
 * t % block_size, and q-head h reads kv-head h / (Hq / Hkv).
 *
 * Layouts (all device memory, row-major, contiguous, 16-byte aligned):
 *   q            fp16  [B][Hq][d]          (rotary embedding already applied)
 *   k_cache      fp16  [num_blocks][Hkv][block_size][d]
 *   v_cache      fp16  same layout as k_cache
 *   block_table  int32 [B][stride]; in apex_decode_attention the stride is
 *                tight, ceil(max_b L_b / block_size), and is derived on the
 *                device; entries past ceil(L_b / block_size) are never read
 *   context_lens int32 [B]; counts the current token (its K/V must already be
 *                in the cache); L_b <= 0 yields a zero output row
 *   out          fp16  [B][Hq][d]; must not overlap any input.  Checked on
 *                the host against q, context_lens, the new rows of the fused
 *                append, and the extents of k_cache, v_cache and block_table
 *                the call knows: num_blocks blocks when apex_decode_args
 *                gives them (else the first block), B rows of an explicit
 *                block_table_stride (else one entry per request)
 *
 * Supported: d = 128, block_size = 16, Hq % Hkv == 0 with Hq / Hkv in
 * {1, 2, 4, 8}.  Anything else returns APEX_ERR_UNSUPPORTED.  The batch's
 * block count, sum over b of ceil(L_b / block_size), must stay below 2^31
 * (about 34 G context tokens): the kernel sums it in 32 bits.  The lengths
 * are device data, so this is not checked.
 *
 * Precision: fp16 inputs, fp32 scores, softmax statistics and accumulation,
 * fp16 output rounded to nearest even.
 *
 * Ownership: the caller owns every buffer; the library never retains or
 * frees caller pointers.  Calls are asynchronous: they validate arguments on
 * the host, enqueue kernels on `stream` (a hipStream_t; NULL = the legacy
 * default stream) and return without synchronising.  Nothing is printed and
 * no C++ exception crosses this boundary.
 *
 * Errors: every entry point returns an apex_status; on failure nothing has
 * been enqueued and apex_decode_last_error() returns a message
 * (thread-local).  Block ids out of range are not checked on the device
 * unless apex_decode_attention_ex is asked to (APEX_DECODE_FLAG_CHECK_INPUTS).
 *
 * Work partition: one persistent kernel launch per call.  Each work group
 * derives the partition from context_lens itself, takes an equal-cost share
 * of the (request, kv-head, block) units (a pair's cost is its blocks plus a
 * fixed start-up cost), and (request, kv-head) pairs shared by several work
 * groups are merged by a log-sum-exp combine done by the last work group to
 * finish its share of the pair.
 */
#ifndef APEX_DECODE_H
#define APEX_DECODE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum apex_status {
    APEX_OK = 0,
    APEX_ERR_INVALID_ARG = -1,   /* null/misaligned pointer, B < 0, Hq % Hkv != 0, aliasing */
    APEX_ERR_UNSUPPORTED = -2,   /* d, block_size or group size outside the supported set */
    APEX_ERR_OUT_OF_MEMORY = -3, /* workspace allocation failed or caller workspace too small */
    APEX_ERR_HIP = -4,           /* a HIP runtime call or kernel launch failed */
    APEX_ERR_BUSY = -5           /* a resource is still in use (apex_overlap.h: result slot) */
} apex_status;

/*
 * Batched paged decode attention for one layer-step (the formula above).
 * B == 0 is a successful no-op.  Uses library-owned workspaces, one set per
 * device, grown on demand (growing waits for the device); concurrent calls on
 * different streams of one device must use apex_decode_attention_ex with
 * caller-owned workspaces.  The call only enqueues one kernel (no host
 * synchronisation, no memset; the arrival counters are left zero by every
 * launch), so apex_decode_attention_ex with a caller workspace and no events
 * can be captured in a HIP graph and replayed.
 */
int apex_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                          const int32_t* block_table, const int32_t* context_lens, void* out,
                          int B, int Hq, int Hkv, int d, int block_size, float scale,
                          void* stream);

/* Extended arguments.  Zero-initialise and fill the first group; every
 * extension field has "off" as its zero value. */
typedef struct apex_decode_args {
    /* same meaning as the apex_decode_attention arguments */
    const void* q;
    const void* k_cache;
    const void* v_cache;
    const int32_t* block_table;
    const int32_t* context_lens;
    void* out;
    int B, Hq, Hkv, d, block_size;
    float scale;
    void* stream;

    /* entries per block_table row; 0 = tight (derived on the device) */
    int64_t block_table_stride;
    /* work groups of the persistent launch; 0 = as many as the device keeps
     * resident.  The work (one unit = one 16-token block of one kv-head) is
     * cut into contiguous ranges, one per work group.  With 0 the ranges are
     * of equal cost, where every non-empty (request, kv-head) pair costs its
     * units plus 8 (the latency of starting and finishing a pair, so that a
     * run of short pairs is spread over several work groups); about 16 units
     * per work group, but never fewer work groups than non-empty pairs, and a
     * batch of at most one pair per CU (and at most 1024 units per CU) uses
     * one work group per CU.  With n > 0 the ranges hold equal numbers of
     * units, at least one each (tests use this to force split requests) */
    int num_workers;
    /* caller-owned device workspace of at least apex_decode_workspace_bytes()
     * bytes and 256-byte aligned, or NULL for the library-owned one.  Its
     * first apex_decode_counter_bytes(B, Hkv) bytes must be zero when the call
     * is enqueued; every call leaves them zero again when it completes. */
    void* workspace;
    size_t workspace_bytes;
    /* optional fp32 [B][Hq]: natural-log log-sum-exp of the scaled logits
     * (max + log of the normaliser); -inf for L_b <= 0 */
    float* lse_out;
    /* optional pair of hipEvent_t recorded on `stream` immediately before and
     * after the attention kernel (for per-kernel timing); NULL = none */
    void* attn_kernel_events[2];
    /* APEX_DECODE_FLAG_* bits; other bits must be 0 */
    uint32_t flags;
    /* physical blocks in k_cache/v_cache (0 = not given; negative is an
     * error); needed by APEX_DECODE_FLAG_CHECK_INPUTS, and when given the
     * overlap check of out covers the whole caches */
    int64_t num_blocks;
    /* Fused append (both NULL = off): the current token's K and V rows, fp16
     * [B][Hkv][d] with new_token_stride elements between tokens (0 = Hkv * d;
     * otherwise a multiple of 8, >= Hkv * d), 16-byte aligned.  context_lens
     * still counts the current token, but the caches need to hold only its
     * first L_b - 1 tokens: the current token is attended from these rows and
     * written to its slot -- the block_table entry of position L_b - 1, slot
     * (L_b - 1) % block_size -- during the call (no request may share that
     * slot).  Equivalent to apex_kv_append of these rows followed by the
     * plain call, in one launch.  With APEX_DECODE_FLAG_CHECK_INPUTS, a
     * current token whose table entry is outside the pool is attended but
     * not stored (APEX_DEVICE_ERR_BLOCK_ID); a context longer than its
     * explicit table row keeps every cached token of the row, and its
     * current token, whose position then lies past the row, is attended but
     * not stored, so the row's last slot keeps its cached token
     * (APEX_DEVICE_ERR_TABLE_ROW). */
    const void* k_new;
    const void* v_new;
    int64_t new_token_stride;
} apex_decode_args;

/*
 * Input check (for debugging engines; a separate kernel build, the default
 * path is unchanged): block ids outside [0, num_blocks) are never read --
 * their blocks are skipped as if absent -- and a context longer than an
 * explicit block_table_stride row is cut to the row.  Each case sets a bit
 * of a per-device error word that apex_decode_check_device_error() returns.
 */
#define APEX_DECODE_FLAG_CHECK_INPUTS 1u
#define APEX_DEVICE_ERR_BLOCK_ID 1u    /* a block id outside [0, num_blocks) */
#define APEX_DEVICE_ERR_TABLE_ROW 2u   /* a context past its block-table row */

int apex_decode_attention_ex(const apex_decode_args* args);

/*
 * No-allocation variant of apex_decode_attention, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments and, on a device whose
 * default grid fits the scratch below (MI355X: 512 work groups), the same
 * launch and the same result bit for bit.  The arrival counters and the
 * partial results live in a static device array of the library instead of a
 * workspace: 4.3 MiB on every device that loads the library, held until the
 * process ends.  The call allocates nothing (no hipMalloc, no hipFree, no
 * allocating library routine).
 *   Limits: B * Hkv <= 65536 (request, kv-head) pairs, else
 *   APEX_ERR_UNSUPPORTED and nothing is enqueued; the launch uses at most
 *   4096 / (Hq / Hkv) work groups.
 *   The first call on a device looks the array up and clears its counters
 *   with a kernel on `stream`; every launch leaves them zero.
 *   Every call on a device shares that device's array: calls that overlap on
 *   one device (streams with no ordering between them) race and give wrong
 *   results.  Order them on one stream, or use apex_decode_attention_ex with
 *   a workspace per stream.
 */
int apex_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                  const int32_t* block_table, const int32_t* context_lens, void* out,
                                  int B, int Hq, int Hkv, int d, int block_size, float scale,
                                  void* stream);

/* Workspace bytes a call with these shapes needs on the current device
 * (num_workers as in apex_decode_args).  0 on bad shapes. */
size_t apex_decode_workspace_bytes(int B, int Hq, int Hkv, int d, int block_size, int num_workers);

/* Leading workspace bytes (arrival counters) that must be zero before a call. */
size_t apex_decode_counter_bytes(int B, int Hkv);

/*
 * Host mirror of the work partition, for inspection and tests (no GPU
 * needed).  Inputs: host context_lens[B], Hkv, block_size, the number of
 * launched work groups, whether that number was forced (num_workers > 0 in
 * apex_decode_args: forced grids cut equal units, the default grid equal
 * costs), and the device's compute units (the default grid uses only one
 * work group per CU for a batch of at most one (request, kv-head) pair per
 * CU and at most 1024 units per CU; 0 leaves that rule out).
 * Outputs (any may be NULL): contributors_out[B * Hkv] = work groups that
 * share each (request, kv-head) pair (1 = written directly, more = combined
 * from partials), *units_out = blocks x kv-heads, *active_out = work groups
 * that get units, *partials_out = partial results written.
 */
int apex_decode_plan_host(const int32_t* context_lens, int B, int Hkv, int block_size,
                          int launched_workers, int forced, int cus, int32_t* contributors_out,
                          int64_t* units_out, int64_t* active_out, int64_t* partials_out);

/* Waits for the current device, returns the input-check error bits that
 * checked calls on it set since the last read (0 if none), and clears them. */
int apex_decode_check_device_error(uint32_t* error_bits);

/* Message for the last failed call on this thread ("" if none). */
const char* apex_decode_last_error(void);

/* Frees the library-owned workspaces (waits for the devices first). */
int apex_decode_release_workspace(void);

/* Library version: major * 10000 + minor * 100 + patch. */
int apex_decode_version(void);

#ifdef __cplusplus
}
#endif

#endif /* APEX_DECODE_H */
