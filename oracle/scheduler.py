"""APEX's analytical model and scheduler, as plain Python -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline
may import this; it shares no code with the library's C++ scheduler.

It follows Sec. 3.2 ("Analytical Model for Scheduling Decisions") and
Sec. 3.4 ("Scheduling Algorithm", Alg. 1 and Alg. 2) in the paper's order and
notation:

  N_G, N_C      GPU and CPU attention rates (tokens per unit time)
  T_glinear     GPU time of a layer's linear operations (decode batch)
  T_gatt        GPU time of the same batch's self-attention
  Eq. 1         T_gpuonly = T_glinear + T_gatt
  Eq. 2         T_overlap = 2 T_glinear + T_gatt   (decode-only pipelining)
  Eq. 3         N_Gtotal  = N_G T_gatt
  Eq. 4         N_Ctotal  = N_C T_overlap
  Eq. 5         pipelining pays iff (N_Gtotal + N_Ctotal) / T_overlap
                                      > N_Gtotal / T_gpuonly
  Eq. 6         the same, solved: N_G / N_C < 2 T_glinear/T_gatt + 3
                                               + T_gatt/T_glinear
  Eq. 7         T_overlap = T_glinear_pref + T_gatt_pref + T_glinear + T_gatt
                (mixed prefill + decode)
  Eq. 8         mixed: (N_G T_gatt + N_C T_overlap) / (T_glinear + T_gatt)
                       > N_G T_gatt / T_gatt
  Alg. 2        StrategySelection: the two throughputs above, pick the larger
  Alg. 1        MainScheduler: GPU-only when no request waits for the CPU;
                Asynchronous Overlap when pipelining schedules no CPU request;
                else StrategySelection.

Readings (the paper is silent or reads two ways):
  - Eq. 8 is taken as printed (Alg. 2 repeats it).  ``mixed_form="eq5"``
    gives the alternative that keeps Eq. 5's shape with Eq. 7's cycle time:
    (N_G T_gatt + N_C T_overlap) / T_overlap > N_G T_gatt / (T_glinear + T_gatt).
  - AsymPipeStrat (the sub-batch choice of the pipelining baseline) is not
    defined by the paper; main_scheduler takes it as a function argument.
  - Ties (equal throughputs) choose Asynchronous Overlap, since Alg. 2 picks
    pipelining only when its throughput is strictly higher.
"""

GPU_ONLY = "gpu_only"
ASYNC_OVERLAP = "async_overlap"
ASYM_PIPELINE = "asym_pipeline"


def t_gpuonly(t_glinear, t_gatt):
    """Eq. 1."""
    return t_glinear + t_gatt


def t_overlap_decode(t_glinear, t_gatt):
    """Eq. 2."""
    return 2 * t_glinear + t_gatt


def n_gtotal(n_g, t_gatt):
    """Eq. 3."""
    return n_g * t_gatt


def n_ctotal(n_c, t_overlap):
    """Eq. 4."""
    return n_c * t_overlap


def pipelining_pays_decode(n_g, n_c, t_glinear, t_gatt):
    """Eq. 5: throughput of pipelining above that of GPU-only."""
    t_ov = t_overlap_decode(t_glinear, t_gatt)
    pipe = (n_gtotal(n_g, t_gatt) + n_ctotal(n_c, t_ov)) / t_ov
    gpu = n_gtotal(n_g, t_gatt) / t_gpuonly(t_glinear, t_gatt)
    return pipe > gpu


def ratio_bound(t_glinear, t_gatt):
    """Right-hand side of Eq. 6: the largest N_G / N_C for which pipelining pays."""
    return 2 * t_glinear / t_gatt + 3 + t_gatt / t_glinear


def t_overlap_mixed(t_glinear_pref, t_gatt_pref, t_glinear, t_gatt):
    """Eq. 7."""
    return t_glinear_pref + t_gatt_pref + t_glinear + t_gatt


def strategy_selection(n_g, n_c, t_glinear, t_gatt, prefill=False, t_glinear_pref=0.0,
                       t_gatt_pref=0.0, mixed_form="paper"):
    """Alg. 2.  Returns (strategy, throughput_pipe, throughput_gpu)."""
    if not prefill:
        t_ov = 2 * t_glinear + t_gatt
        throughput_gpu = n_g * t_gatt / (t_glinear + t_gatt)
        throughput_pipe = (n_g * t_gatt + n_c * t_ov) / (2 * t_glinear + t_gatt)
    else:
        t_ov = t_glinear_pref + t_gatt_pref + t_glinear + t_gatt
        if mixed_form == "paper":
            throughput_gpu = n_g * t_gatt / t_gatt
            throughput_pipe = (n_g * t_gatt + n_c * t_ov) / (t_glinear + t_gatt)
        elif mixed_form == "eq5":
            throughput_gpu = n_g * t_gatt / (t_glinear + t_gatt)
            throughput_pipe = (n_g * t_gatt + n_c * t_ov) / t_ov
        else:
            raise ValueError(mixed_form)
    strategy = ASYM_PIPELINE if throughput_pipe > throughput_gpu else ASYNC_OVERLAP
    return strategy, throughput_pipe, throughput_gpu


def main_scheduler(p_in, d_gpu_in, d_cpu_in, asym_pipe_strat, selection_inputs):
    """Alg. 1.  ``asym_pipe_strat(p_in, d_gpu_in, d_cpu_in)`` returns the
    sub-batches (p_sch, d_gpu_sch, d_cpu_sch); ``selection_inputs(p_sch,
    d_gpu_sch, d_cpu_sch)`` returns the keyword arguments of
    strategy_selection for them (the profiled times and rates)."""
    if len(d_cpu_in) == 0:
        return GPU_ONLY
    p_sch, d_gpu_sch, d_cpu_sch = asym_pipe_strat(p_in, d_gpu_in, d_cpu_in)
    if len(d_cpu_sch) == 0:
        return ASYNC_OVERLAP
    kw = selection_inputs(p_sch, d_gpu_sch, d_cpu_sch)
    return strategy_selection(prefill=len(p_sch) > 0, **kw)[0]


# ---------------------------------------------------------------------------
# profiled inputs (Sec. 3.2 "Parameter Estimation via Offline Profiling"):
# times measured at sample points, read between them by linear interpolation
# ---------------------------------------------------------------------------

def interp1(xs, ys, x):
    """Piecewise-linear through (xs[i], ys[i]) (xs strictly increasing),
    extended past either end along the nearest segment, never below 0.
    A single sample is a constant."""
    n = len(xs)
    if n == 1:
        return max(ys[0], 0.0)
    i = 0
    while i < n - 2 and x > xs[i + 1]:
        i += 1
    y = ys[i] + (ys[i + 1] - ys[i]) * (x - xs[i]) / (xs[i + 1] - xs[i])
    return max(y, 0.0)


def interp2(bs, ts, table, b, t):
    """Bilinear over a batch x tokens grid (table[i][j] at bs[i], ts[j]),
    extended like interp1 along each axis."""
    rows = [interp1(ts, table[i], t) for i in range(len(bs))]
    return interp1(bs, rows, b)


def inputs_from_profile(profile, gpu_batch, gpu_tokens, cpu_batch, cpu_tokens, prefill_tokens=0.0):
    """Rates and times for strategy_selection from a profile dict:
    gatt_tokens/gatt_seconds, glin_batch/glin_seconds, cpu_batch/cpu_tokens/
    cpu_seconds (grid), pref_tokens/pref_linear_seconds/pref_attn_seconds.
    N_G = GPU tokens / T_gatt(GPU tokens); N_C = CPU tokens / T_cpu(batch, tokens)."""
    t_gatt = interp1(profile["gatt_tokens"], profile["gatt_seconds"], gpu_tokens)
    t_glinear = interp1(profile["glin_batch"], profile["glin_seconds"], gpu_batch)
    t_cpu = interp2(profile["cpu_batch"], profile["cpu_tokens"], profile["cpu_seconds"], cpu_batch, cpu_tokens)
    out = dict(n_g=gpu_tokens / t_gatt, n_c=cpu_tokens / t_cpu if cpu_tokens > 0 else 0.0,
               t_glinear=t_glinear, t_gatt=t_gatt)
    if prefill_tokens > 0:
        out["t_glinear_pref"] = interp1(profile["pref_tokens"], profile["pref_linear_seconds"], prefill_tokens)
        out["t_gatt_pref"] = interp1(profile["pref_tokens"], profile["pref_attn_seconds"], prefill_tokens)
    return out
