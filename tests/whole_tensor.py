"""Whole-tensor parity at full size: the fp64 oracle over every request of a
named workload, chunk by chunk, and the error statistics over the whole
[B][Hq][d] output.

The oracle's inputs are copies of the workload's device tensors taken before
the GPU call under test (the inputs the HIP path reads), never its outputs.
"""
import os

import numpy as np

MAX_ABS = 2e-3
REL_L2 = 1e-3


def host_threads():
    """Threads for the oracle: the host cores this job may use, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_reference(oracle_mod, wl, chunk=64, prepare=None):
    """fp64 reference [B][Hq][d] of workload ``wl`` (an apex_workloads
    DeviceWorkload), computed over chunks of ``chunk`` requests so that the
    host holds one chunk of K/V at a time.  ``prepare(case, requests)`` may
    return a modified host case first (e.g. the oracle's own KV append)."""
    cfg = wl.cfg
    ref = np.empty((cfg.B, cfg.Hq, cfg.d), dtype=np.float64)
    threads = host_threads()
    for c0 in range(0, cfg.B, chunk):
        reqs = list(range(c0, min(cfg.B, c0 + chunk)))
        case = wl.host_request_case(reqs)
        if prepare is not None:
            case = prepare(case, reqs)
        ref[c0:c0 + len(reqs)] = oracle_mod.decode_attention_f64(
            case.q, case.k_cache, case.v_cache, case.block_table, case.context_lens, case.scale,
            num_threads=threads)
    return ref


def whole_tensor_errors(got, ref):
    """max-abs and relative-L2 error over the whole tensor, plus the request
    with the largest error (logged, not gated)."""
    got = np.asarray(got, dtype=np.float64)
    err = got - ref
    per_req = np.abs(err).reshape(err.shape[0], -1).max(axis=1)
    worst = int(np.argmax(per_req))
    return {
        "finite": bool(np.all(np.isfinite(got))),
        "max_abs": float(per_req.max()),
        "rel_l2": float(np.linalg.norm(err) / np.linalg.norm(ref)),
        "worst_request": worst,
        "worst_request_max_abs": float(per_req[worst]),
        "requests": int(err.shape[0]),
    }


def assert_whole_tensor(got, ref, what):
    e = whole_tensor_errors(got, ref)
    print(f"[whole-tensor] {what}: requests={e['requests']} max_abs={e['max_abs']:.3e} "
          f"rel_l2={e['rel_l2']:.3e} worst request {e['worst_request']}", flush=True)
    assert e["finite"], f"{what}: non-finite outputs"
    assert e["max_abs"] <= MAX_ABS, f"{what}: max-abs {e['max_abs']:.3e}"
    assert e["rel_l2"] <= REL_L2, f"{what}: rel-L2 {e['rel_l2']:.3e}"
    return e
