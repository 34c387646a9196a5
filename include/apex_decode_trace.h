/*
 * apex_decode_trace.h -- work-group timeline of the decode-attention kernel,
 * exported only by the diagnostic build libapex_decode_trace.so (the same
 * sources compiled with APEX_TRACE_WORK_GROUPS; the product library
 * libapex_decode.so has none of it, and its kernel code is unchanged).
 *
 * Decode attention streams every cached K/V row once and is bound by memory
 * bandwidth (APEX, Sec. 2.2 and Sec. 2.3); the timeline shows where a launch
 * loses time against that bound: each work group's start, the end of its
 * partition prologue, the arrival of its first K/V tiles, and its end.
 */
#ifndef APEX_DECODE_TRACE_H
#define APEX_DECODE_TRACE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Sets the device buffer every later attention launch of this library (any
 * entry point, any device) writes its timeline into: uint64
 * [max_work_groups][8], caller-owned, 8-byte aligned; NULL turns the
 * recording off.  Work group w < max_work_groups writes row w when it ends:
 *   [0] first instruction, [1] end of the partition prologue (0 if it got
 *   no units), [2] wave 0's first tiles complete (0 if no units), [3] end --
 *   all in ticks of the GPU's 100 MHz real-time clock --, [4] segments
 *   (request, kv-head pieces) it attended, [5] those of them shared with
 *   other work groups (split), [6] its units (16-token blocks of one
 *   kv-head), [7] zero.
 * Rows of work groups past max_work_groups are not written.  Returns
 * APEX_OK, or APEX_ERR_INVALID_ARG for a negative count or a misaligned
 * buffer.
 */
int apex_decode_trace_buffer(void* device_words, int64_t max_work_groups);

#ifdef __cplusplus
}
#endif

#endif /* APEX_DECODE_TRACE_H */
