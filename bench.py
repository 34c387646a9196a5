"""Benchmark: batched paged decode attention, one layer-step, on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c4]

A step is one apex_decode_attention call (one persistent kernel that plans,
attends and combines) over the whole batch with inputs resident in HBM.  Whole
steps for --prewarm-ms (200 ms: the GPU reaches its steady clocks; calls after
an idle spell run up to 3-4 % slower), then W untimed steps, then K steps back
to back between two device synchronisations.  Prints one JSON line:

  value      algorithmic HBM GB/s of the whole step: (KV + Q + O bytes of valid
             tokens) / (ms per step); us_per_layer_step alongside
  roofline   the attention kernel alone: algorithmic bytes / its mean duration,
             timed with HIP events recorded by the library on the launch stream
             around that kernel, against the 8 TB/s HBM peak; "traffic" is the
             HBM bytes per launch from the committed rocprofv3 counter summary
             when it was taken on the current kernel source, else null
  cpu_baseline  the fp64 CPU oracle on the host cores over a bounded sample of
             the same workload (the first requests), in the same unit; its
             single_thread entry is the same on one thread (about 2 s)
  cpu_attention  the library's own host backend (libapex_cpu.so, SIMD +
             thread pool) on a host copy of the same workload, against the
             host read bandwidth measured with the same threads
  overlap    the Asynchronous Overlap runtime (libapex_overlap.so) in a
             synthetic decode iteration of 8 Llama-3.1-8B layers: bf16
             linears on the unified batch, this workload's attention on the
             GPU, 16 extra requests attended on the host; iteration time
             GPU-only (without the extra requests; and with their rows in
             the linears but no attention for them, the floor of the
             overlap), with the overlap (results collected by a readiness
             check that never blocks; a layer whose previous result is still
             out gets no new host work that iteration, so the host-attended
             requests advance at the host's pace and the GPU never waits for
             them; their tokens are counted from the collected jobs) and with
             a blocking wait in every layer; every iteration ends with a host
             synchronisation, as sampling the next tokens requires
  kv_append  the paged KV append that precedes each step (apex_kv_append),
             timed alone with events around its kernel: the step's own append
             (one token per request at position L_b - 1 of the workload's
             cache) and a prompt-sized bulk append (65536 tokens) against the
             HBM peak; bytes = new K/V rows read + cache rows written + slots
  fused_append  one layer-step as apex_kv_append + attention (two launches)
             and as one fused call (k_new/v_new), back to back
  scheduler  Alg. 2's decision for this GPU batch plus a host batch, from
             the committed MI355X profile, and the cost of one decision
  host       CPU model, sockets, NUMA nodes and usable cores of the host
  parity     the output of the last timed step against the fp64 oracle over
             the cpu_baseline sample (the whole batch of the default
             workload): max-abs, relative L2, finite, against the attention
             bar; the run exits non-zero after printing when it fails
  workloads  every named workload (c1-c5) timed like the headline one:
             whole step, kernel alone (events) and kernel with cold caches,
             algorithmic GB/s and fraction of the HBM peak, and the committed
             counter traffic when it matches the kernel source (c1, 13 MB,
             fits in the caches: a latency figure); with the CPU baseline on,
             each also carries cpu_baseline_1_thread, the fp64 oracle on one
             host thread over a sample of that workload (about 2 s)
Inside roofline, kernel_us_cold_median / achieved_cold time the kernel after
a 512 MiB read has evicted the caches (the figure that relies on no K/V left
in a cache by the previous call).

The default workload is the Llama-3.1-8B GQA long-output decode batch (B=32,
32 q-heads over 8 kv-heads, d=128, block_size 16, context lengths lognormal
with median 12k clipped to [4096, 32768]).  Only one GPU is used: --gpus above
1 is refused.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode-attn µs/layer-step + achieved HBM GB/s (% peak), Llama-3.1-8B GQA"
PEAK_HBM_GBS = 8000.0
COLD_REPS = 20        # calls timed after evicting the caches
SINGLE_THREAD_SECONDS = 2.0   # the one-thread oracle sample of each workload
PARITY_MAX_ABS = 2e-3  # the attention bar: fp16 output, fp32 accumulation
PARITY_REL_L2 = 1e-3
WORKLOADS = ("c1", "c2", "c3", "c4", "c5")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")
# the files that define the attention kernel and its work partition: counter
# summaries stay valid while their code (comments aside) is unchanged
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2506_03296_amd", "csrc", f)
                  for f in ("kernels.h", "plan_policy.h")]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _code_only(text):
    """C++ source of the product build: comments and the blocks of the
    work-group trace build (APEX_TRACE_WORK_GROUPS, never defined in the
    product) removed and whitespace runs collapsed, so that editing a comment
    or the diagnostic build does not invalidate a counter summary."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = re.sub(r"#ifdef APEX_TRACE_WORK_GROUPS\b.*?#endif", " ", text, flags=re.S)
    return " ".join(text.split())


def kernel_source_digest():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p) as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def committed_traffic(workload):
    """HBM bytes per attention launch from the committed counter summary, if
    it was taken on the current kernel source and this workload."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    entry = t.get(workload)
    if not entry or entry.get("source_digest") != kernel_source_digest():
        return None
    return entry.get("hbm_bytes_per_launch")


def oracle_rate(wl, threads, target_s):
    """The fp64 oracle on `threads` host threads over the first requests of
    the batch: one request first, then as many as its time per context
    token puts at about target_s (at most the whole batch).  Returns the
    rate line, the host case, the oracle's output and the request count."""
    import numpy as np

    import oracle
    import apex_workloads as W
    cfg = wl.cfg

    def run(n):
        case = wl.host_request_case(range(n))
        t0 = time.perf_counter()
        ref = oracle.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale, num_threads=threads)
        return time.perf_counter() - t0, case, ref

    n = 1
    dt, case, ref = run(n)
    if dt < target_s and n < cfg.B:
        tokens = np.cumsum(np.maximum(np.asarray(wl.lens, dtype=np.int64), 0))
        per_token = dt / max(1, int(tokens[0]))
        n = int(max(1, min(cfg.B, np.searchsorted(tokens, target_s / per_token, side="right"))))
        dt, case, ref = run(n)
    nbytes = W.algorithmic_bytes(case.context_lens, n, cfg.Hq, cfg.Hkv, cfg.d)
    line = {
        "value": round(nbytes / dt / 1e9, 4),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {n} of {cfg.B} requests ({int(np.sum(case.context_lens))} tokens, "
                  f"{nbytes / 1e6:.1f} MB algorithmic), fp64 plain-loop oracle, {dt:.2f} s",
    }
    return line, case, ref, n


def cpu_baseline(wl, target_s, timed_out=None):
    """Time the fp64 oracle on the host over the first requests of the batch,
    on up to 16 threads and on one.

    With ``timed_out`` (host copy of the output of the last timed step) the
    oracle's result over those requests is also compared with it: the parity
    of what the benchmark timed, against the attention bar (max-abs <= 2e-3,
    relative L2 <= 1e-3, all finite)."""
    import numpy as np

    cfg = wl.cfg
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    baseline, case, ref, n = oracle_rate(wl, threads, target_s)
    baseline["single_thread"] = oracle_rate(wl, 1, SINGLE_THREAD_SECONDS)[0]
    parity = None
    if timed_out is not None:
        got = np.asarray(timed_out[:n], dtype=np.float64)
        err = got - ref
        max_abs = float(np.max(np.abs(err)))
        rel = float(np.linalg.norm(err) / np.linalg.norm(ref))
        finite = bool(np.all(np.isfinite(got)))
        parity = {
            "against": "fp64 oracle (the cpu_baseline sample)",
            "output": "out of the last timed step",
            "requests": n, "of": cfg.B,
            "max_abs": max_abs, "rel_l2": rel, "finite": finite,
            "bar": {"max_abs": PARITY_MAX_ABS, "rel_l2": PARITY_REL_L2},
            "ok": finite and max_abs <= PARITY_MAX_ABS and rel <= PARITY_REL_L2,
        }
    return baseline, parity


def host_info():
    """The host the CPU legs ran on: model, sockets, NUMA nodes, cores usable."""
    model, sockets = "unknown", set()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                key, _, val = line.partition(":")
                key = key.strip()
                if key == "model name" and model == "unknown":
                    model = val.strip()
                elif key == "physical id":
                    sockets.add(val.strip())
    except OSError:
        pass
    try:
        numa = len([d for d in os.listdir("/sys/devices/system/node") if d.startswith("node") and d[4:].isdigit()])
    except OSError:
        numa = None
    return {"cpu_model": model, "sockets": len(sockets) or None, "numa_nodes": numa,
            "cores_usable": len(os.sched_getaffinity(0)), "cores_online": os.cpu_count()}


def time_append(A, torch, k_new, v_new, k_cache, v_cache, slots, reps):
    """Mean kernel time (ms) of apex_kv_append, from events around each call.

    A short kernel finishes before the host can enqueue the next one, so the
    stream is first held by a spin kernel while every (event, append, event)
    triple is enqueued; the appends then run back to back and each event
    pair brackets its kernel alone rather than the host's enqueue latency."""
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(reps)]
    for _ in range(3):
        A.kv_append(k_new, v_new, k_cache, v_cache, slots)
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    for a, b in pairs:
        a.record()
        A.kv_append(k_new, v_new, k_cache, v_cache, slots)
        b.record()
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in pairs) / reps


def time_copy(torch, nbytes, reps):
    """Mean time (ms) of a plain device copy of nbytes (reads and writes
    nbytes each): the read+write bandwidth a scatter can hope for."""
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def append_bytes(tokens, Hkv, d):
    return tokens * Hkv * d * 2 * 4 + tokens * 8


def measure_append(A, torch, W, wl, reps):
    cfg = wl.cfg
    # the step's own append: rewrite each request's newest row with its
    # current values, so the workload's cache is unchanged
    slots_np = W.append_slots(wl.layout)
    slots = torch.from_numpy(slots_np).cuda()
    valid = slots_np >= 0
    blk = torch.from_numpy(slots_np[valid] // cfg.block_size).cuda()
    pos = torch.from_numpy(slots_np[valid] % cfg.block_size).cuda()
    kn = torch.zeros((cfg.B, cfg.Hkv, cfg.d), dtype=torch.float16, device="cuda")
    vn = torch.zeros_like(kn)
    sel = torch.from_numpy(valid.nonzero()[0]).cuda()
    kn[sel] = wl.k_cache[blk, :, pos, :]
    vn[sel] = wl.v_cache[blk, :, pos, :]
    ms = time_append(A, torch, kn, vn, wl.k_cache, wl.v_cache, slots, reps)
    nb = append_bytes(int(valid.sum()), cfg.Hkv, cfg.d)
    step = {"tokens": int(valid.sum()), "us_mean": round(ms * 1e3, 2), "bytes": nb,
            "achieved": round(nb / (ms * 1e-3) / 1e9, 2)}
    # prompt-sized bulk append into a pool of its own
    T, pool = 65536, 4096
    gen = torch.Generator(device="cuda")
    gen.manual_seed(cfg.seed)
    kc = torch.zeros((pool, cfg.Hkv, cfg.block_size, cfg.d), dtype=torch.float16, device="cuda")
    vc = torch.zeros_like(kc)
    kn = torch.randn((T, cfg.Hkv, cfg.d), generator=gen, device="cuda").half()
    vn = torch.randn((T, cfg.Hkv, cfg.d), generator=gen, device="cuda").half()
    perm = torch.randperm(pool, generator=gen, device="cuda")
    slots = (perm[:, None] * cfg.block_size
             + torch.arange(cfg.block_size, device="cuda")[None, :]).reshape(-1)[:T].contiguous()
    ms = time_append(A, torch, kn, vn, kc, vc, slots, reps)
    nb = append_bytes(T, cfg.Hkv, cfg.d)
    achieved = nb / (ms * 1e-3) / 1e9
    del kc, vc, kn, vn
    copy_ms = time_copy(torch, nb // 2, reps)
    bulk = {"tokens": T, "us_mean": round(ms * 1e3, 2), "bytes": nb, "bound": "hbm",
            "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "device_copy_same_bytes_GBps": round(nb / (copy_ms * 1e-3) / 1e9, 2)}
    return {"kernel": "kv_append_kernel", "decode_step": step, "bulk": bulk}


def measure_cpu_attention(wl, threads, reps=5):
    """The host backend over a host copy of the whole workload."""
    from paper_2506_03296_amd import cpu
    cpu.set_threads(threads)
    q = wl.q.cpu().numpy()
    k = wl.k_cache.cpu().numpy()
    v = wl.v_cache.cpu().numpy()
    bt = wl.block_table.cpu().numpy()
    lens = wl.context_lens.cpu().numpy()
    out = cpu.decode_attention(q, k, v, bt, lens, wl.scale)
    best = float("inf")
    for _ in range(reps):
        t0 = time.perf_counter()
        cpu.decode_attention(q, k, v, bt, lens, wl.scale, out=out)
        best = min(best, time.perf_counter() - t0)
    del k, v
    read = cpu.read_bandwidth(1 << 30, num_threads=threads, reps=3)
    achieved = wl.algorithmic_bytes / best / 1e9
    return {"kernel": "apex_cpu_decode_attention", "isa": {2: "avx512", 1: "avx2"}.get(cpu.isa(), "none"),
            "threads": threads, "us_per_layer_step": round(best * 1e6, 1),
            "bound": "host-dram", "achieved": round(achieved, 2), "unit": "GB/s",
            "host_read_GBps": round(read, 2), "frac_of_host_read": round(achieved / read, 4),
            "timing": f"best of {reps} calls, wall clock"}


def measure_overlap(A, torch, wl, layers=8, b_cpu=16, l_cpu=512, iters=16, warmup=3):
    """Iteration times of a synthetic decode loop with and without host
    attention for b_cpu extra requests (see the module docstring)."""
    import numpy as np

    from paper_2506_03296_amd import cpu, overlap
    from paper_2506_03296_amd.profiler import layer_linears
    # leave cores to the thread that launches the GPU work
    threads = max(1, min(8, len(os.sched_getaffinity(0)) // 2))
    cpu.set_threads(threads)
    cfg = wl.cfg
    total = warmup + iters
    stride = -(-(l_cpu + total + 1) // cfg.block_size) + 1
    num_blocks = b_cpu * stride
    table = np.arange(num_blocks, dtype=np.int32).reshape(b_cpu, stride)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(cfg.seed + 1)
    # the host-attended requests' new rows, q | k | v back to back (one copy)
    nq, nkv = b_cpu * cfg.Hq * cfg.d, b_cpu * cfg.Hkv * cfg.d
    rows = torch.randn((nq + 2 * nkv,), generator=gen, device="cuda").half()
    q_c = rows[:nq].view(b_cpu, cfg.Hq, cfg.d)
    kn = rows[nq:nq + nkv].view(b_cpu, cfg.Hkv, cfg.d)
    vn = rows[nq + nkv:].view(b_cpu, cfg.Hkv, cfg.d)
    outs = [torch.empty_like(q_c) for _ in range(layers)]
    lin_gpu = layer_linears(torch, cfg.B, seed=1)
    lin_all = layer_linears(torch, cfg.B + b_cpu, seed=2)

    def attn():
        A.decode_attention_ex(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                              wl.scale, out=wl.out)

    # the host attention alone, for reference
    hk = np.zeros((num_blocks, cfg.Hkv, cfg.block_size, cfg.d), np.float16)
    lens0 = np.full(b_cpu, l_cpu, np.int32)
    qh = q_c.cpu().numpy()
    cpu.decode_attention(qh, hk, hk, table, lens0, wl.scale)
    t_cpu = min(_timed(lambda: cpu.decode_attention(qh, hk, hk, table, lens0, wl.scale))
                for _ in range(5))

    times, jobs = {}, {}
    for mode in ("gpu_only", "gpu_only_unified", "async_overlap", "sync_wait"):
        # two result slots per layer: one in flight, one being collected
        rt = overlap.Overlap(layers, b_cpu, cfg.Hq, cfg.Hkv, cfg.d, cfg.block_size, wl.scale,
                             num_blocks, stride, threads=threads)
        lens = np.full(b_cpu, l_cpu - 1, np.int32)
        pending = [[] for _ in range(layers)]   # tickets not yet collected, oldest first
        counts = {"done": 0, "skipped": 0}

        def slots_for(lens_now):
            pos = lens_now - 1
            return table[np.arange(b_cpu), pos // cfg.block_size].astype(np.int64) * cfg.block_size \
                + pos % cfg.block_size

        def iteration():
            nonlocal lens
            lens = lens + 1
            slots = slots_for(lens)
            for l in range(layers):
                if mode.startswith("gpu_only"):
                    (lin_gpu if mode == "gpu_only" else lin_all)()
                    attn()
                    continue
                lin_all()
                if mode == "sync_wait":
                    t = rt.submit(l, q_c, kn, vn, slots, table, lens)
                    attn()
                    rt.wait(t, outs[l])
                    counts["done"] += 1
                    continue
                # readiness check, never blocking: collect what the host has
                # finished; a layer whose previous result is still out gets no
                # new work this iteration (its requests wait), the GPU goes on
                while pending[l] and rt.poll(pending[l][0], outs[l]):
                    pending[l].pop(0)
                    counts["done"] += 1
                if not pending[l]:
                    pending[l].append(rt.submit(l, q_c, kn, vn, slots, table, lens))
                else:
                    counts["skipped"] += 1
                attn()
            # the iteration ends by sampling the next tokens: the host waits
            # for the GPU once per iteration, as a decode loop does
            torch.cuda.synchronize()

        for _ in range(warmup):
            iteration()
        torch.cuda.synchronize()
        counts["done"] = counts["skipped"] = 0
        t0 = time.perf_counter()
        for _ in range(iters):
            iteration()
        torch.cuda.synchronize()
        times[mode] = (time.perf_counter() - t0) / iters
        jobs[mode] = dict(counts)
        for l in range(layers):
            for t in pending[l]:
                rt.wait(t, outs[l])
        torch.cuda.synchronize()
        rt.close()
    # host-attended requests finish a token per `layers` collected jobs
    tok = {"gpu_only": cfg.B, "gpu_only_unified": cfg.B,
           "async_overlap": cfg.B + b_cpu * jobs["async_overlap"]["done"] / (layers * iters),
           "sync_wait": cfg.B + b_cpu}
    return {
        "runtime": "apex_overlap", "layers": layers, "gpu_requests": cfg.B, "cpu_requests": b_cpu,
        "cpu_context_tokens": l_cpu, "host_threads": threads,
        "iteration_ms": {k: round(v * 1e3, 3) for k, v in times.items()},
        "tokens_per_s": {k: round(tok[k] / v, 1) for k, v in times.items()},
        "host_attention_ms_per_layer": round(t_cpu * 1e3, 3),
        "host_jobs_done_per_layer_iteration": round(jobs["async_overlap"]["done"] / (layers * iters), 3),
        "overlap_cost_ms": round((times["async_overlap"] - times["gpu_only_unified"]) * 1e3, 3),
        "timing": f"wall clock over {iters} iterations after {warmup}",
    }


def measure_scheduler(wl, gpu_tokens, cpu_batch=16, cpu_tokens=16 * 4096, calls=20000):
    """Alg. 2 of the library on inputs interpolated from the committed MI355X
    profile (this GPU batch, a CPU batch of cpu_batch requests): the decision
    and the host time per call through the binding (ctypes included)."""
    from paper_2506_03296_amd import sched
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "sched_profile_mi355x.json")
    with open(path) as f:
        profile = json.load(f)
    kw = sched.inputs_from_profile(profile, wl.cfg.B, gpu_tokens, cpu_batch, cpu_tokens)
    r = sched.select(**kw)
    t0 = time.perf_counter()
    for _ in range(calls):
        sched.select(**kw)
    per = (time.perf_counter() - t0) / calls
    return {
        "algorithm": "Alg. 2 (decode), apex_sched_select",
        "profile": "profiles/sched_profile_mi355x.json",
        "gpu_batch": wl.cfg.B, "gpu_tokens": int(gpu_tokens), "cpu_batch": cpu_batch,
        "cpu_tokens": cpu_tokens, "n_g_tokens_per_s": round(kw["n_g"], 1), "n_c_tokens_per_s": round(kw["n_c"], 1),
        "ratio": round(kw["n_g"] / kw["n_c"], 2), "ratio_bound": round(r["ratio_bound"], 3),
        "strategy": r["strategy"], "us_per_decision": round(per * 1e6, 3),
        "timing": f"{calls} calls from Python, ctypes included",
    }


def measure_fused_step(A, torch, wl, steps=50, warmup=20):
    """One layer-step as two launches (apex_kv_append, then the attention) and
    as one fused call (k_new/v_new), back to back; the new rows are copies of
    each request's last cached token, so the caches do not change."""
    lens = wl.context_lens.to(torch.int64)
    last = (lens - 1).clamp(min=0)
    rows = torch.arange(wl.cfg.B, device=lens.device)
    blocks = wl.block_table[rows, last // 16].to(torch.int64)
    pos = last % 16
    slots = torch.where(lens > 0, blocks * 16 + pos, torch.full_like(blocks, -1))
    k_new = wl.k_cache[blocks, :, pos, :].contiguous()
    v_new = wl.v_cache[blocks, :, pos, :].contiguous()

    def separate():
        A.kv_append(k_new, v_new, wl.k_cache, wl.v_cache, slots)
        A.decode_attention(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens, wl.scale,
                           out=wl.out)

    def fused():
        A.decode_attention_ex(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens, wl.scale,
                              out=wl.out, k_new=k_new, v_new=v_new)

    res = {}
    for name, fn in (("separate", separate), ("fused", fused), ("separate_again", separate)):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        res[name] = a.elapsed_time(b) * 1e3 / steps
    sep = (res["separate"] + res["separate_again"]) / 2
    return {"us_per_step_append_then_attend": round(sep, 2), "us_per_step_fused": round(res["fused"], 2),
            "saved_us": round(sep - res["fused"], 2),
            "timing": f"{steps} back-to-back steps after {warmup}; the two-launch time is the mean of a run "
                      "before and one after the fused run"}


def time_workload(A, torch, wl, steps, warmup, workers=0, prewarm_ms=0.0):
    """The timings of one workload: whole steps for prewarm_ms (the GPU at its
    steady clocks: calls after an idle spell run up to 3-4 % slower), W
    untimed steps, K steps back to back between two synchronisations (whole
    step), K steps with events recorded by the library around the kernel
    (kernel alone), and COLD_REPS calls each after a 512 MiB read (cold
    caches).  Returns the figures and a host copy of the output of the last
    back-to-back step."""
    def step(events=None):
        A.decode_attention_ex(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                              wl.scale, out=wl.out, num_workers=workers, events=events)

    prewarm_calls = 0
    t_end = time.perf_counter() + prewarm_ms * 1e-3
    while time.perf_counter() < t_end:
        for _ in range(10):
            step()
        prewarm_calls += 10
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()

    # whole steps, back to back, no per-kernel events
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = start.elapsed_time(stop) / steps
    timed_out = wl.out.cpu().numpy()

    # the attention kernel alone: events recorded by the library around it,
    # on the launch stream
    ev_pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(steps)]
    for i in range(steps):
        step(ev_pairs[i])
    torch.cuda.synchronize()
    kern_ms = sorted(a.elapsed_time(b) for a, b in ev_pairs)

    # the same kernel with cold caches: before each call a 512 MiB read
    # (outside the events) evicts the 256 MB Infinity Cache and the L2s with
    # clean lines, so no K/V byte comes from a cache filled by the previous
    # call and no write-back competes with the kernel
    scratch = torch.ones(128 << 20, dtype=torch.int32, device="cuda")
    cold_pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(COLD_REPS)]
    torch.cuda.synchronize()
    for pair in cold_pairs:
        torch.amax(scratch)
        step(pair)
    torch.cuda.synchronize()
    cold_ms = sorted(a.elapsed_time(b) for a, b in cold_pairs)
    del scratch
    return {"ms_per_step": ms_per_step, "wall_s_per_step": wall / steps, "kern_ms": kern_ms,
            "cold_ms": cold_ms, "prewarm_calls": prewarm_calls}, timed_out


def workload_line(wl, t, traffic):
    """One workload's figures: whole step and kernel alone, algorithmic GB/s
    and their fraction of the 8 TB/s HBM peak."""
    nbytes = wl.algorithmic_bytes
    kern = sum(t["kern_ms"]) / len(t["kern_ms"])
    cold = t["cold_ms"][len(t["cold_ms"]) // 2]
    step_gbs = nbytes / (t["ms_per_step"] * 1e-3) / 1e9
    kern_gbs = nbytes / (kern * 1e-3) / 1e9
    cfg = wl.cfg
    return {
        "workload": cfg.title,
        "B": cfg.B, "Hq": cfg.Hq, "Hkv": cfg.Hkv,
        "total_tokens": int(wl.lens.sum()), "algorithmic_bytes": int(nbytes),
        "us_per_layer_step": round(t["ms_per_step"] * 1e3, 2),
        "step_GBps": round(step_gbs, 2),
        "step_frac": round(step_gbs / PEAK_HBM_GBS, 4),
        "kernel_us_mean": round(kern * 1e3, 2),
        "kernel_GBps": round(kern_gbs, 2),
        "kernel_frac": round(kern_gbs / PEAK_HBM_GBS, 4),
        "kernel_us_cold_median": round(cold * 1e3, 2),
        "kernel_frac_cold": round(nbytes / (cold * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "traffic": traffic,
    }


def measure_workloads(A, torch, W, names, steps, warmup, workers, done, prewarm_ms, oracle_1_thread=False,
                      headline_oracle=None):
    """The other named workloads, each generated, timed like the headline one
    and freed in turn (``done`` holds lines already measured).  With
    oracle_1_thread every line also gets the fp64 oracle's one-thread rate on
    a sample of its batch (``headline_oracle`` is the headline workload's)."""
    lines = dict(done)
    for name in names:
        if name in lines:
            continue
        log(f"workload {name}: generating")
        wl = W.DeviceWorkload(name)
        torch.cuda.synchronize()
        t, _ = time_workload(A, torch, wl, steps, warmup, workers, prewarm_ms)
        lines[name] = workload_line(wl, t, committed_traffic(name))
        if name == "c1":
            lines[name]["kind"] = "latency (13 MB: the batch fits in the caches)"
        if oracle_1_thread:
            lines[name]["cpu_baseline_1_thread"] = oracle_rate(wl, 1, SINGLE_THREAD_SECONDS)[0]
        log(f"workload {name}: {lines[name]['us_per_layer_step']} us/step, "
            f"kernel {lines[name]['kernel_us_mean']} us ({100 * lines[name]['kernel_frac']:.1f} %)")
        del wl
        torch.cuda.empty_cache()
    out = {k: lines[k] for k in names if k in lines}
    for k, v in out.items():
        if oracle_1_thread and headline_oracle is not None and "cpu_baseline_1_thread" not in v:
            v["cpu_baseline_1_thread"] = headline_oracle
    return out


def _timed(fn):
    t0 = time.perf_counter()
    fn()
    return time.perf_counter() - t0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=500,
                    help="untimed steps first; ~0.1 s of continuous calls brings the GPU to its "
                         "steady clocks (the first calls after idle run up to 3-4 %% slower)")
    ap.add_argument("--prewarm-ms", type=float, default=200.0,
                    help="whole steps for this long before the warmup steps, so the GPU is at its "
                         "steady clocks when the warmup steps begin (0 = none)")
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--workers", type=int, default=0,
                    help="work groups of the persistent launch (0 = device default)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (for counter scaling)")
    ap.add_argument("--hbm-probe", action="store_true",
                    help="only measure achievable HBM read bandwidth (stream and 4 KiB gather)")
    ap.add_argument("--probe-mib", type=int, default=4096,
                    help="buffer size of --hbm-probe in MiB")
    ap.add_argument("--no-append", action="store_true", help="skip the kv_append lines")
    ap.add_argument("--no-cpu-attention", action="store_true",
                    help="skip the host backend line")
    ap.add_argument("--no-overlap", action="store_true", help="skip the overlap runtime line")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the per-workload lines (c1-c5 timed like the headline one)")
    ap.add_argument("--overlap-sweep", action="store_true",
                    help="only run the overlap measurement over host-attended batch sizes")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import apex_workloads as W
    import paper_2506_03296_amd as A

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    A.load_library()

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "launches": args.warmup + args.steps}))
        return

    if args.hbm_probe:
        from paper_2506_03296_amd import hbm_probe
        props = torch.cuda.get_device_properties(0)
        cus = props.multi_processor_count
        res = hbm_probe.measure(nbytes=args.probe_mib << 20, blocks_list=(cus * 2, cus * 4, cus * 8))
        res["device"] = props.name
        res["cus"] = cus
        print(json.dumps(res), flush=True)
        return

    log(f"generating workload {args.workload}")
    wl = W.DeviceWorkload(args.workload)
    if args.overlap_sweep:
        for b_cpu, l_cpu in ((8, 512), (16, 512), (32, 512), (64, 512), (16, 2048), (32, 2048)):
            r = measure_overlap(A, torch, wl, b_cpu=b_cpu, l_cpu=l_cpu)
            print(json.dumps(r), flush=True)
        return
    cfg = wl.cfg
    nbytes = wl.algorithmic_bytes
    torch.cuda.synchronize()

    log(f"warmup {args.warmup}, timing {args.steps} steps")
    t, timed_out = time_workload(A, torch, wl, args.steps, args.warmup, args.workers, args.prewarm_ms)
    ms_per_step = t["ms_per_step"]
    kern_ms = t["kern_ms"]
    kern_mean = sum(kern_ms) / len(kern_ms)
    cold_med = t["cold_ms"][len(t["cold_ms"]) // 2]
    log(f"{ms_per_step * 1e3:.1f} us/step (wall {t['wall_s_per_step'] * 1e6:.1f} us), "
        f"attention kernel mean {kern_mean * 1e3:.1f} us")

    achieved = nbytes / (kern_mean * 1e-3) / 1e9
    traffic = committed_traffic(args.workload)
    result = {
        "metric": METRIC,
        "value": round(nbytes / (ms_per_step * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "prewarm": {"ms": args.prewarm_ms, "calls": t["prewarm_calls"],
                    "what": "whole steps before the W warmup steps, until the GPU is at its steady clocks"},
        "ms_per_step": round(ms_per_step, 5),
        "us_per_layer_step": round(ms_per_step * 1e3, 2),
        "pct_of_peak_hbm": round(100.0 * nbytes / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBS, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}: {cfg.title}",
            "B": cfg.B, "Hq": cfg.Hq, "Hkv": cfg.Hkv, "d": cfg.d, "block_size": cfg.block_size,
            "total_tokens": int(wl.lens.sum()),
            "algorithmic_bytes": int(nbytes),
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "attn_kernel",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "kernel_us_mean": round(kern_mean * 1e3, 2),
            "kernel_us_p10": round(kern_ms[len(kern_ms) // 10] * 1e3, 2),
            "kernel_us_p90": round(kern_ms[(9 * len(kern_ms)) // 10] * 1e3, 2),
            "kernel_us_cold_median": round(cold_med * 1e3, 2),
            "achieved_cold": round(nbytes / (cold_med * 1e-3) / 1e9, 2),
        },
        "cpu_baseline": None,
        "parity": None,
    }
    headline_line = workload_line(wl, t, traffic)
    if not args.no_cpu_attention:
        log("timing the host backend")
        threads = max(1, min(16, len(os.sched_getaffinity(0))))
        result["cpu_attention"] = measure_cpu_attention(wl, threads)
    if not args.no_overlap:
        log("timing the overlap runtime")
        result["overlap"] = measure_overlap(A, torch, wl)
    log("timing the fused append")
    result["fused_append"] = measure_fused_step(A, torch, wl)
    log("timing the strategy selection")
    result["scheduler"] = measure_scheduler(wl, int(wl.lens.sum()))
    if not args.no_append:
        log("timing kv_append")
        result["kv_append"] = measure_append(A, torch, W, wl, max(10, args.steps))
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (and checking the timed output against it)")
        result["cpu_baseline"], result["parity"] = cpu_baseline(wl, args.cpu_seconds, timed_out)
        p = result["parity"]
        log(f"parity of the timed output over {p['requests']} requests: max_abs {p['max_abs']:.3e}, "
            f"rel_l2 {p['rel_l2']:.3e} -> {'ok' if p['ok'] else 'FAILED'}")
    if not (args.no_cpu_baseline and args.no_cpu_attention and args.no_overlap):
        result["host"] = host_info()
    if not args.no_workloads:
        del wl
        torch.cuda.empty_cache()
        cb = result["cpu_baseline"]
        result["workloads"] = measure_workloads(A, torch, W, WORKLOADS, args.steps, args.warmup,
                                                args.workers, {args.workload: headline_line},
                                                args.prewarm_ms, oracle_1_thread=cb is not None,
                                                headline_oracle=cb["single_thread"] if cb else None)
    print(json.dumps(result), flush=True)
    if result["parity"] is not None and not result["parity"]["ok"]:
        print("bench.py: the timed output fails the parity bar against the oracle", file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
