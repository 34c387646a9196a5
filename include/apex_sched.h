/*
 * apex_sched.h -- C ABI of APEX's profiling-informed strategy selection
 * (host logic, in libapex_cpu.so).
 *
 * APEX decides per iteration how decode requests whose KV does not fit in GPU
 * memory are served (Sec. 3.4): GPU-only when no request waits for the CPU,
 * otherwise Asymmetric Pipelining (two sub-batches, CPU attention overlapped
 * with the GPU's) or its own Asynchronous Overlap (one unified batch, CPU
 * results taken one iteration later).  The choice compares throughputs from
 * an analytical model fed by offline profiles (Sec. 3.2):
 *
 *   Eq. 1  T_gpuonly = T_glinear + T_gatt
 *   Eq. 2  T_overlap = 2 T_glinear + T_gatt                 (decode only)
 *   Eq. 5  pipelining pays iff
 *          (N_G T_gatt + N_C T_overlap) / T_overlap > N_G T_gatt / T_gpuonly
 *   Eq. 6  equivalently N_G / N_C < 2 T_glinear / T_gatt + 3 + T_gatt / T_glinear
 *   Eq. 7  T_overlap = T_glinear_pref + T_gatt_pref + T_glinear + T_gatt  (mixed)
 *   Eq. 8  mixed: (N_G T_gatt + N_C T_overlap) / (T_glinear + T_gatt) > N_G T_gatt / T_gatt
 *   Alg. 2 StrategySelection: pipelining if its throughput is strictly higher,
 *          else Asynchronous Overlap
 *   Alg. 1 MainScheduler: GPU-only / Asynchronous Overlap / Alg. 2
 *
 * N_G and N_C are attention rates in tokens per second (context tokens read
 * per second by one layer's attention), times are seconds per layer.
 * Eq. 8 is used as printed by default; APEX_MIXED_EQ5 selects the reading
 * that keeps Eq. 5's shape with Eq. 7's cycle time:
 *   (N_G T_gatt + N_C T_overlap) / T_overlap > N_G T_gatt / (T_glinear + T_gatt).
 *
 * Profiled inputs: apex_sched_inputs_from_profile reads times off sample
 * tables by piecewise-linear interpolation (bilinear over the CPU's batch x
 * tokens grid), extended past the ends along the end segments and clamped at
 * zero; N_G = GPU tokens / T_gatt(GPU tokens), N_C = CPU tokens /
 * T_cpu(CPU batch, CPU tokens), T_glinear = T_glinear(GPU batch).
 *
 * All functions are pure and thread-safe; they return an apex_status code
 * (apex_decode.h) and leave a message in apex_cpu_last_error() on failure.
 */
#ifndef APEX_SCHED_H
#define APEX_SCHED_H

#include <stdint.h>

#include "apex_decode.h"   /* apex_status codes */

#ifdef __cplusplus
extern "C" {
#endif

typedef enum apex_strategy {
    APEX_GPU_ONLY = 0,
    APEX_ASYNC_OVERLAP = 1,
    APEX_ASYM_PIPELINE = 2
} apex_strategy;

typedef enum apex_mixed_form {
    APEX_MIXED_PAPER = 0,   /* Eq. 8 / Alg. 2 as printed */
    APEX_MIXED_EQ5 = 1      /* Eq. 5's shape with Eq. 7's cycle time */
} apex_mixed_form;

typedef struct apex_sched_inputs {
    double n_g, n_c;                    /* tokens / s; n_g > 0, n_c >= 0 */
    double t_glinear, t_gatt;           /* s per layer, > 0 */
    double t_glinear_pref, t_gatt_pref; /* s per layer of the prefill part, >= 0 */
    int prefill;                        /* nonzero: mixed prefill + decode branch */
    int mixed_form;                     /* apex_mixed_form */
} apex_sched_inputs;

typedef struct apex_sched_result {
    int strategy;              /* apex_strategy */
    double throughput_pipe;    /* tokens / s, Alg. 2 */
    double throughput_gpu;
    double t_overlap;          /* Eq. 2 or Eq. 7 */
    double ratio_bound;        /* Eq. 6 right-hand side (decode-only branch; 0 otherwise) */
} apex_sched_result;

/* Alg. 2. */
int apex_sched_select(const apex_sched_inputs* in, apex_sched_result* out);

/* Alg. 1 on queue sizes: n_cpu_decode requests wait for CPU attention and
 * n_cpu_scheduled of them were placed in the pipelining sub-batches by the
 * caller's sub-batch policy (the paper leaves that policy to the pipelining
 * baseline), n_prefill_scheduled prefill requests likewise.  `in` is read only
 * when Alg. 2 is reached (its `prefill` field is set from
 * n_prefill_scheduled > 0). */
int apex_sched_main(int n_prefill_scheduled, int n_gpu_decode, int n_cpu_decode,
                    int n_cpu_scheduled, const apex_sched_inputs* in, apex_sched_result* out);

/* Eq. 6 right-hand side: the largest N_G / N_C at which pipelining pays. */
double apex_sched_ratio_bound(double t_glinear, double t_gatt);

/* Offline profile tables (all arrays host memory, x values strictly increasing). */
typedef struct apex_sched_profile {
    int gatt_n;                  /* GPU decode attention, seconds per layer vs total context tokens */
    const double* gatt_tokens;
    const double* gatt_seconds;
    int glin_n;                  /* GPU decode linears, seconds per layer vs batch size */
    const double* glin_batch;
    const double* glin_seconds;
    int cpu_nb, cpu_nt;          /* CPU attention, seconds per layer on a batch x tokens grid */
    const double* cpu_batch;     /* [cpu_nb] */
    const double* cpu_tokens;    /* [cpu_nt] */
    const double* cpu_seconds;   /* [cpu_nb][cpu_nt] */
    int pref_n;                  /* prefill, seconds per layer vs prefill tokens (may be 0) */
    const double* pref_tokens;
    const double* pref_linear_seconds;
    const double* pref_attn_seconds;
} apex_sched_profile;

/* Fills `out` for a GPU decode batch (gpu_batch requests, gpu_tokens context
 * tokens) and a CPU batch (cpu_batch, cpu_tokens); prefill_tokens > 0 selects
 * the mixed branch (needs pref_n > 0). */
int apex_sched_inputs_from_profile(const apex_sched_profile* p, double gpu_batch, double gpu_tokens,
                                   double cpu_batch, double cpu_tokens, double prefill_tokens,
                                   int mixed_form, apex_sched_inputs* out);

/* Piecewise-linear interpolation as used above (exposed for tests). */
double apex_sched_interp1(int n, const double* xs, const double* ys, double x);

/* Decode-attention tokens whose KV fits in `free_bytes` of GPU memory
 * (K and V of every layer: 2 * layers * Hkv * d * bytes_per_element per
 * token) -- the GPU-first rule admits requests to the GPU while this lasts. */
int64_t apex_sched_gpu_token_capacity(double free_bytes, int layers, int Hkv, int d,
                                      int bytes_per_element);

#ifdef __cplusplus
}
#endif

#endif /* APEX_SCHED_H */
