"""Work-group timeline of the decode-attention kernel (diagnostic build).

    python -m paper_2506_03296_amd.wg_trace [--workload c3 ...] [--calls 8]

Decode attention reads every cached K/V row once and is bound by HBM
bandwidth (APEX, Sec. 2.2 and Sec. 2.3).  This tool shows where a launch
loses time against that bound.  It loads libapex_decode_trace.so -- the same
kernel compiled with per-work-group timestamps (include/apex_decode_trace.h)
-- runs a named workload's call after a warm-up, and reports, over `--calls`
traced calls (medians across calls):

  span        last work-group end - first work-group start (us), next to the
              call's kernel time from HIP events around it
  dispatch    when work groups start, relative to the first one: the first
              round (one group per CU) and the second (the CU's other group)
  prologue    partition prologue per work group (start -> its first segment)
  first_load  prologue end -> wave 0's first K/V tiles complete
  ends        work-group end times (p10, p50, p90, max), overall and per round
  tail        last end - median end
  by_segments mean end time of the groups by the number of segments they
              attended (pair boundaries in their range)
  ends_by_xcd mean end time per XCD (work groups are dealt round-robin over
              the 8 XCDs: w mod 8), per round

Times are in microseconds from the first work group's start (the GPU's
100 MHz real-time clock).  Output: one JSON line per workload.  The trace
build carries a few more instructions than the product kernel; its event
time is reported beside the product's for comparison.
"""
import argparse
import ctypes
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
TRACE_LIB_PATH = os.path.join(HERE, "libapex_decode_trace.so")
WORDS = 8
TICK_US = 0.01     # 100 MHz real-time clock


def load_trace_library():
    from . import load_library
    if not os.path.exists(TRACE_LIB_PATH):
        raise RuntimeError(f"{TRACE_LIB_PATH} is not built; run python -m paper_2506_03296_amd.build")
    lib = load_library(path=TRACE_LIB_PATH)
    lib.apex_decode_trace_buffer.restype = ctypes.c_int
    lib.apex_decode_trace_buffer.argtypes = [ctypes.c_void_p, ctypes.c_int64]
    return lib


def pct(x, q):
    return float(np.percentile(x, q)) if len(x) else float("nan")


def summarize(rows, cus):
    """Timeline statistics of one traced call (rows: int64 [W][8])."""
    rows = rows[rows[:, 3] > 0]
    W = rows.shape[0]
    t0 = rows[:, 0].min()
    start = (rows[:, 0] - t0) * TICK_US
    end = (rows[:, 3] - t0) * TICK_US
    act = rows[:, 6] > 0
    part = (rows[act, 1] - rows[act, 0]) * TICK_US
    first = (rows[act, 2] - rows[act, 1]) * TICK_US
    first_abs = (rows[act, 2] - t0) * TICK_US
    w = np.arange(W)
    r1, r2 = w < cus, w >= cus
    seg = rows[:, 4]
    by_seg = {}
    for n in np.unique(seg[act]):
        sel = act & (seg == n)
        by_seg[int(n)] = {"groups": int(sel.sum()), "end_mean": round(float(end[sel].mean()), 2),
                          "end_max": round(float(end[sel].max()), 2)}
    out = {
        "work_groups": int(W), "active": int(act.sum()),
        "span": float(end.max()),
        "dispatch": {"round1_start_max": pct(start[r1], 100),
                     "round2_start_min": pct(start[r2], 0) if r2.any() else None,
                     "round2_start_max": pct(start[r2], 100) if r2.any() else None},
        "prologue": {"p50": pct(part, 50), "p90": pct(part, 90), "max": pct(part, 100)},
        "first_load": {"p50": pct(first, 50), "p90": pct(first, 90), "max": pct(first, 100)},
        "first_data_at": {"p50": pct(first_abs, 50), "p90": pct(first_abs, 90), "max": pct(first_abs, 100)},
        "ends": {"p10": pct(end, 10), "p50": pct(end, 50), "p90": pct(end, 90), "max": pct(end, 100)},
        "ends_round1": {"p10": pct(end[r1], 10), "p50": pct(end[r1], 50), "max": pct(end[r1], 100)},
        "ends_round2": ({"p10": pct(end[r2], 10), "p50": pct(end[r2], 50), "max": pct(end[r2], 100)}
                        if r2.any() else None),
        "tail": float(end.max() - np.percentile(end, 50)),
        # work groups are dealt round-robin over the 8 XCDs: w mod 8
        "ends_by_xcd_round1": [round(float(end[act & r1 & (w % 8 == x)].mean()), 2)
                               if (act & r1 & (w % 8 == x)).any() else None for x in range(8)],
        "ends_by_xcd_round2": [round(float(end[act & r2 & (w % 8 == x)].mean()), 2)
                               if (act & r2 & (w % 8 == x)).any() else None for x in range(8)],
        "first_load_round2": {"p50": pct(first[r2[act]], 50), "p90": pct(first[r2[act]], 90)}
                             if (r2 & act).any() else None,
        "units_per_group": {"min": int(rows[act, 6].min()), "max": int(rows[act, 6].max())},
        "split_segments": int(rows[:, 5].sum()),
        "by_segments": by_seg,
    }
    return out


def median_of(dicts):
    """Element-wise median of nested dicts of numbers (same keys)."""
    d0 = dicts[0]
    if isinstance(d0, dict):
        return {k: median_of([d[k] for d in dicts]) if all(isinstance(d.get(k), (dict, list, int, float))
                                                            for d in dicts) else d0[k] for k in d0}
    if isinstance(d0, list):
        return [median_of([d[i] for d in dicts]) if all(d[i] is not None for d in dicts) else None
                for i in range(len(d0))]
    vals = [v for v in dicts if v is not None]
    v = float(np.median(vals))
    return round(v, 2)


def trace_workload(A, lib, torch, W, name, calls, warmup):
    wl = W.DeviceWorkload(name)
    props = torch.cuda.get_device_properties(0)
    cus = props.multi_processor_count
    max_groups = 1 << 16
    buf = torch.zeros((max_groups, WORDS), dtype=torch.int64, device="cuda")

    def call(events=None):
        A.decode_attention_ex(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                              wl.scale, out=wl.out, events=events)

    assert lib.apex_decode_trace_buffer(ctypes.c_void_p(buf.data_ptr()), max_groups) == 0
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    stats, kern = [], []
    for _ in range(calls):
        buf.zero_()
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        call(ev)
        torch.cuda.synchronize()
        kern.append(ev[0].elapsed_time(ev[1]) * 1e3)
        stats.append(summarize(buf.cpu().numpy(), cus))
    assert lib.apex_decode_trace_buffer(None, 0) == 0
    res = median_of(stats)
    res = {"workload": name, "calls": calls, "cus": cus,
           "kernel_us_events": round(float(np.median(kern)), 2),
           "algorithmic_bytes": int(wl.algorithmic_bytes), **res}
    del wl, buf
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", action="append", default=None)
    ap.add_argument("--calls", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=300)
    args = ap.parse_args()
    import torch

    sys.path.insert(0, os.path.dirname(HERE))
    import apex_workloads as W
    import paper_2506_03296_amd as A
    if not torch.cuda.is_available():
        print("wg_trace needs a GPU", file=sys.stderr)
        sys.exit(2)
    lib = load_trace_library()
    A._LIB = lib        # every binding call of this process goes to the trace build
    for name in args.workload or ["c3"]:
        print(json.dumps(trace_workload(A, lib, torch, W, name, args.calls, args.warmup)), flush=True)


if __name__ == "__main__":
    main()
