/*
 * apex_hbm_probe.h -- HBM read-bandwidth probes for one MI355X (gfx950).
 *
 * Measures the bandwidth that the decode-attention access pattern can reach on
 * the device it runs on, as a ceiling to read its own numbers against: decode
 * attention streams every cached K/V row once (APEX Sec. 2.2, Sec. 2.3), in
 * 4 KiB chunks (one block of one kv-head) scattered through the cache.
 *
 * Both calls enqueue one kernel on `stream` (hipStream_t, NULL = legacy
 * default stream) and return without synchronising.  Buffers are device
 * memory owned by the caller.  Return 0 on success, -1 on bad arguments, -4
 * on a launch failure.
 */
#ifndef APEX_HBM_PROBE_H
#define APEX_HBM_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` (a multiple of 16) of `buf` once with 128-bit loads using
 * `blocks` work groups of 256 threads (0 = 8 per compute unit).  flags bit 0
 * = non-temporal loads.  `sink` is a 4-byte device word the kernel writes
 * only if the data XOR to a sentinel. */
int apex_hbm_probe_stream(const void* buf, size_t bytes, int blocks, int flags, uint32_t* sink,
                          void* stream);

/* Reads `n_chunks` chunks of 4096 bytes, chunk i starting at byte
 * chunk_ids[i] * 4096 of `buf` (int32 ids, device memory), a 64-lane wave
 * per chunk with 128-bit loads, `blocks` work groups of 256 threads
 * (0 = 8 per compute unit).  flags bit 0 = non-temporal loads, bits 1-3 =
 * chunks each wave has in flight (1, 2 or 4), bit 4 = the attention kernel's
 * access form instead: a buffer resource per chunk and non-temporal buffer
 * loads (bit 0 is then ignored). */
int apex_hbm_probe_gather(const void* buf, const int32_t* chunk_ids, int64_t n_chunks, int blocks,
                          int flags, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* APEX_HBM_PROBE_H */
