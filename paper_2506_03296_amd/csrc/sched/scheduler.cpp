// scheduler.cpp -- APEX's analytical model and strategy selection
// (include/apex_sched.h): Eq. 1-8, Alg. 1 and Alg. 2 of the paper, plus the
// profile-table lookups that feed them.  Pure host arithmetic in double.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include "apex_sched.h"

namespace apex_cpu {
__attribute__((visibility("hidden"), format(printf, 2, 3))) int sched_fail(int code, const char* fmt, ...);
}

namespace {

using apex_cpu::sched_fail;

bool finite_pos(double x) { return isfinite(x) && x > 0.0; }
bool finite_nonneg(double x) { return isfinite(x) && x >= 0.0; }

double interp1(int n, const double* xs, const double* ys, double x)
{
    if (n == 1) return ys[0] > 0.0 ? ys[0] : 0.0;
    int i = 0;
    while (i < n - 2 && x > xs[i + 1]) ++i;
    const double y = ys[i] + (ys[i + 1] - ys[i]) * (x - xs[i]) / (xs[i + 1] - xs[i]);
    return y > 0.0 ? y : 0.0;
}

bool increasing(int n, const double* xs)
{
    for (int i = 0; i < n; ++i) {
        if (!isfinite(xs[i])) return false;
        if (i > 0 && !(xs[i] > xs[i - 1])) return false;
    }
    return true;
}

int check_table(const char* what, int n, const double* xs, const double* ys)
{
    if (n < 1 || !xs || !ys) return sched_fail(APEX_ERR_INVALID_ARG, "%s table is empty", what);
    if (!increasing(n, xs)) return sched_fail(APEX_ERR_INVALID_ARG, "%s sample points must increase", what);
    for (int i = 0; i < n; ++i)
        if (!finite_nonneg(ys[i])) return sched_fail(APEX_ERR_INVALID_ARG, "%s times must be finite and >= 0", what);
    return APEX_OK;
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" {

double apex_sched_ratio_bound(double t_glinear, double t_gatt)
{
    return 2.0 * t_glinear / t_gatt + 3.0 + t_gatt / t_glinear;
}

int apex_sched_select(const apex_sched_inputs* in, apex_sched_result* out)
{
    if (!in || !out) return sched_fail(APEX_ERR_INVALID_ARG, "NULL argument");
    const apex_sched_inputs& a = *in;
    if (!finite_pos(a.n_g) || !finite_nonneg(a.n_c) || !finite_pos(a.t_glinear) || !finite_pos(a.t_gatt))
        return sched_fail(APEX_ERR_INVALID_ARG, "rates and decode times must be finite, n_g and times > 0");
    if (a.prefill && (!finite_nonneg(a.t_glinear_pref) || !finite_nonneg(a.t_gatt_pref)))
        return sched_fail(APEX_ERR_INVALID_ARG, "prefill times must be finite and >= 0");
    if (a.mixed_form != APEX_MIXED_PAPER && a.mixed_form != APEX_MIXED_EQ5)
        return sched_fail(APEX_ERR_INVALID_ARG, "unknown mixed_form %d", a.mixed_form);
    const double ng = a.n_g, nc = a.n_c, tl = a.t_glinear, ta = a.t_gatt;
    double t_ov, gpu, pipe;
    if (!a.prefill) {
        // decode only: Eq. 2 cycle, Eq. 5 throughputs
        t_ov = 2.0 * tl + ta;
        gpu = ng * ta / (tl + ta);
        pipe = (ng * ta + nc * t_ov) / (2.0 * tl + ta);
        out->ratio_bound = apex_sched_ratio_bound(tl, ta);
    } else {
        // mixed: Eq. 7 cycle, Eq. 8 (or its Eq.-5-shaped reading)
        t_ov = a.t_glinear_pref + a.t_gatt_pref + tl + ta;
        if (a.mixed_form == APEX_MIXED_PAPER) {
            gpu = ng * ta / ta;
            pipe = (ng * ta + nc * t_ov) / (tl + ta);
        } else {
            gpu = ng * ta / (tl + ta);
            pipe = (ng * ta + nc * t_ov) / t_ov;
        }
        out->ratio_bound = 0.0;
    }
    out->t_overlap = t_ov;
    out->throughput_gpu = gpu;
    out->throughput_pipe = pipe;
    out->strategy = pipe > gpu ? APEX_ASYM_PIPELINE : APEX_ASYNC_OVERLAP;
    return APEX_OK;
}

int apex_sched_main(int n_prefill_scheduled, int n_gpu_decode, int n_cpu_decode, int n_cpu_scheduled,
                    const apex_sched_inputs* in, apex_sched_result* out)
{
    if (!out) return sched_fail(APEX_ERR_INVALID_ARG, "NULL result");
    if (n_prefill_scheduled < 0 || n_gpu_decode < 0 || n_cpu_decode < 0 || n_cpu_scheduled < 0 ||
        n_cpu_scheduled > n_cpu_decode)
        return sched_fail(APEX_ERR_INVALID_ARG, "queue sizes must be >= 0 and scheduled <= waiting");
    out->throughput_pipe = out->throughput_gpu = out->t_overlap = out->ratio_bound = 0.0;
    if (n_cpu_decode == 0) {
        out->strategy = APEX_GPU_ONLY;   // the GPU holds every request's KV
        return APEX_OK;
    }
    if (n_cpu_scheduled == 0) {
        out->strategy = APEX_ASYNC_OVERLAP;   // pipelining found no CPU work
        return APEX_OK;
    }
    if (!in) return sched_fail(APEX_ERR_INVALID_ARG, "NULL inputs");
    apex_sched_inputs a = *in;
    a.prefill = n_prefill_scheduled > 0;
    return apex_sched_select(&a, out);
}

double apex_sched_interp1(int n, const double* xs, const double* ys, double x)
{
    if (n < 1 || !xs || !ys) return 0.0;
    return interp1(n, xs, ys, x);
}

int apex_sched_inputs_from_profile(const apex_sched_profile* p, double gpu_batch, double gpu_tokens,
                                   double cpu_batch, double cpu_tokens, double prefill_tokens,
                                   int mixed_form, apex_sched_inputs* out)
{
    if (!p || !out) return sched_fail(APEX_ERR_INVALID_ARG, "NULL argument");
    int rc;
    if ((rc = check_table("gatt", p->gatt_n, p->gatt_tokens, p->gatt_seconds)) != APEX_OK) return rc;
    if ((rc = check_table("glin", p->glin_n, p->glin_batch, p->glin_seconds)) != APEX_OK) return rc;
    if (p->cpu_nb < 1 || p->cpu_nt < 1 || !p->cpu_batch || !p->cpu_tokens || !p->cpu_seconds ||
        !increasing(p->cpu_nb, p->cpu_batch) || !increasing(p->cpu_nt, p->cpu_tokens))
        return sched_fail(APEX_ERR_INVALID_ARG, "cpu grid must be non-empty with increasing axes");
    for (int i = 0; i < p->cpu_nb * p->cpu_nt; ++i)
        if (!finite_nonneg(p->cpu_seconds[i])) return sched_fail(APEX_ERR_INVALID_ARG, "cpu times must be >= 0");
    if (!(gpu_tokens > 0.0) || !(gpu_batch > 0.0) || !(cpu_tokens >= 0.0) || !(cpu_batch >= 0.0) ||
        !(prefill_tokens >= 0.0))
        return sched_fail(APEX_ERR_INVALID_ARG, "batch sizes and token counts must be >= 0 (GPU ones > 0)");
    const double t_gatt = interp1(p->gatt_n, p->gatt_tokens, p->gatt_seconds, gpu_tokens);
    const double t_glin = interp1(p->glin_n, p->glin_batch, p->glin_seconds, gpu_batch);
    if (!(t_gatt > 0.0) || !(t_glin > 0.0))
        return sched_fail(APEX_ERR_INVALID_ARG, "profile gives a zero GPU time at this batch");
    // bilinear: interpolate each batch row at cpu_tokens, then across batch
    double rows_stack[64];
    double* rows = rows_stack;
    if (p->cpu_nb > 64) return sched_fail(APEX_ERR_UNSUPPORTED, "cpu grid has more than 64 batch rows");
    for (int i = 0; i < p->cpu_nb; ++i)
        rows[i] = interp1(p->cpu_nt, p->cpu_tokens, p->cpu_seconds + (int64_t)i * p->cpu_nt, cpu_tokens);
    const double t_cpu = interp1(p->cpu_nb, p->cpu_batch, rows, cpu_batch);
    out->n_g = gpu_tokens / t_gatt;
    if (cpu_tokens > 0.0) {
        if (!(t_cpu > 0.0)) return sched_fail(APEX_ERR_INVALID_ARG, "profile gives a zero CPU time at this batch");
        out->n_c = cpu_tokens / t_cpu;
    } else {
        out->n_c = 0.0;
    }
    out->t_glinear = t_glin;
    out->t_gatt = t_gatt;
    out->prefill = prefill_tokens > 0.0;
    out->mixed_form = mixed_form;
    out->t_glinear_pref = out->t_gatt_pref = 0.0;
    if (out->prefill) {
        if (p->pref_n < 1) return sched_fail(APEX_ERR_INVALID_ARG, "prefill tokens given but no prefill table");
        if ((rc = check_table("prefill linear", p->pref_n, p->pref_tokens, p->pref_linear_seconds)) != APEX_OK ||
            (rc = check_table("prefill attention", p->pref_n, p->pref_tokens, p->pref_attn_seconds)) != APEX_OK)
            return rc;
        out->t_glinear_pref = interp1(p->pref_n, p->pref_tokens, p->pref_linear_seconds, prefill_tokens);
        out->t_gatt_pref = interp1(p->pref_n, p->pref_tokens, p->pref_attn_seconds, prefill_tokens);
    }
    return APEX_OK;
}

int64_t apex_sched_gpu_token_capacity(double free_bytes, int layers, int Hkv, int d, int bytes_per_element)
{
    if (!(free_bytes > 0.0) || layers <= 0 || Hkv <= 0 || d <= 0 || bytes_per_element <= 0) return 0;
    const double per_token = 2.0 * layers * Hkv * (double)d * bytes_per_element;
    return (int64_t)floor(free_bytes / per_token);
}

}  // extern "C"
#pragma GCC visibility pop
