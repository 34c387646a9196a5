"""Python binding of APEX's strategy selection (include/apex_sched.h, in
libapex_cpu.so).  Argument marshalling only.

    r = select(n_g, n_c, t_glinear, t_gatt)                  # Alg. 2, decode only
    r = select(..., prefill=True, t_glinear_pref=..., t_gatt_pref=...)
    r = main(n_prefill_scheduled, n_gpu, n_cpu, n_cpu_scheduled, inputs)   # Alg. 1
    kw = inputs_from_profile(profile, gpu_batch, gpu_tokens, cpu_batch, cpu_tokens)

Strategies are returned as the strings "gpu_only", "async_overlap" and
"asym_pipeline".
"""
import ctypes

import numpy as np

from . import cpu as _cpu

GPU_ONLY, ASYNC_OVERLAP, ASYM_PIPELINE = "gpu_only", "async_overlap", "asym_pipeline"
_NAMES = {0: GPU_ONLY, 1: ASYNC_OVERLAP, 2: ASYM_PIPELINE}
MIXED_FORMS = {"paper": 0, "eq5": 1}

EXPORTED_SYMBOLS = (
    "apex_sched_select", "apex_sched_main", "apex_sched_ratio_bound",
    "apex_sched_inputs_from_profile", "apex_sched_interp1", "apex_sched_gpu_token_capacity",
)


class Inputs(ctypes.Structure):
    """Mirror of apex_sched_inputs."""
    _fields_ = [("n_g", ctypes.c_double), ("n_c", ctypes.c_double),
                ("t_glinear", ctypes.c_double), ("t_gatt", ctypes.c_double),
                ("t_glinear_pref", ctypes.c_double), ("t_gatt_pref", ctypes.c_double),
                ("prefill", ctypes.c_int), ("mixed_form", ctypes.c_int)]


class Result(ctypes.Structure):
    """Mirror of apex_sched_result."""
    _fields_ = [("strategy", ctypes.c_int), ("throughput_pipe", ctypes.c_double),
                ("throughput_gpu", ctypes.c_double), ("t_overlap", ctypes.c_double),
                ("ratio_bound", ctypes.c_double)]


_DP = ctypes.POINTER(ctypes.c_double)


class Profile(ctypes.Structure):
    """Mirror of apex_sched_profile."""
    _fields_ = [("gatt_n", ctypes.c_int), ("gatt_tokens", _DP), ("gatt_seconds", _DP),
                ("glin_n", ctypes.c_int), ("glin_batch", _DP), ("glin_seconds", _DP),
                ("cpu_nb", ctypes.c_int), ("cpu_nt", ctypes.c_int), ("cpu_batch", _DP),
                ("cpu_tokens", _DP), ("cpu_seconds", _DP),
                ("pref_n", ctypes.c_int), ("pref_tokens", _DP), ("pref_linear_seconds", _DP),
                ("pref_attn_seconds", _DP)]


def _lib():
    lib = _cpu.load_library()
    if not getattr(lib, "_sched_ready", False):
        lib.apex_sched_select.restype = ctypes.c_int
        lib.apex_sched_select.argtypes = [ctypes.POINTER(Inputs), ctypes.POINTER(Result)]
        lib.apex_sched_main.restype = ctypes.c_int
        lib.apex_sched_main.argtypes = [ctypes.c_int] * 4 + [ctypes.POINTER(Inputs), ctypes.POINTER(Result)]
        lib.apex_sched_ratio_bound.restype = ctypes.c_double
        lib.apex_sched_ratio_bound.argtypes = [ctypes.c_double, ctypes.c_double]
        lib.apex_sched_inputs_from_profile.restype = ctypes.c_int
        lib.apex_sched_inputs_from_profile.argtypes = [ctypes.POINTER(Profile)] + [ctypes.c_double] * 5 + [
            ctypes.c_int, ctypes.POINTER(Inputs)]
        lib.apex_sched_interp1.restype = ctypes.c_double
        lib.apex_sched_interp1.argtypes = [ctypes.c_int, _DP, _DP, ctypes.c_double]
        lib.apex_sched_gpu_token_capacity.restype = ctypes.c_int64
        lib.apex_sched_gpu_token_capacity.argtypes = [ctypes.c_double] + [ctypes.c_int] * 4
        lib._sched_ready = True
    return lib


def _check(rc):
    if rc != 0:
        raise _cpu.CpuError(rc, _cpu.last_error())


def make_inputs(n_g, n_c, t_glinear, t_gatt, prefill=False, t_glinear_pref=0.0, t_gatt_pref=0.0,
                mixed_form="paper"):
    return Inputs(float(n_g), float(n_c), float(t_glinear), float(t_gatt), float(t_glinear_pref),
                  float(t_gatt_pref), int(bool(prefill)), MIXED_FORMS[mixed_form])


def _result(r):
    return {"strategy": _NAMES[r.strategy], "throughput_pipe": r.throughput_pipe,
            "throughput_gpu": r.throughput_gpu, "t_overlap": r.t_overlap, "ratio_bound": r.ratio_bound}


def select(n_g, n_c, t_glinear, t_gatt, **kw):
    """Alg. 2; returns a dict with the strategy and the two throughputs."""
    inp = make_inputs(n_g, n_c, t_glinear, t_gatt, **kw)
    r = Result()
    _check(_lib().apex_sched_select(ctypes.byref(inp), ctypes.byref(r)))
    return _result(r)


def main(n_prefill_scheduled, n_gpu_decode, n_cpu_decode, n_cpu_scheduled, inputs=None):
    """Alg. 1 on queue sizes; ``inputs`` is a dict for make_inputs (or None)."""
    r = Result()
    inp = make_inputs(**inputs) if inputs else None
    _check(_lib().apex_sched_main(n_prefill_scheduled, n_gpu_decode, n_cpu_decode, n_cpu_scheduled,
                                  ctypes.byref(inp) if inp is not None else None, ctypes.byref(r)))
    return _result(r)


def ratio_bound(t_glinear, t_gatt):
    return _lib().apex_sched_ratio_bound(float(t_glinear), float(t_gatt))


def _arr(xs):
    a = np.ascontiguousarray(np.asarray(xs, dtype=np.float64))
    return a, a.ctypes.data_as(_DP)


def interp1(xs, ys, x):
    xa, xp = _arr(xs)
    ya, yp = _arr(ys)
    return _lib().apex_sched_interp1(len(xa), xp, yp, float(x))


def inputs_from_profile(profile, gpu_batch, gpu_tokens, cpu_batch, cpu_tokens, prefill_tokens=0.0,
                        mixed_form="paper"):
    """Rates and times (a dict for select/make_inputs) from a profile dict
    with the keys of apex_sched_profile (cpu_seconds as a [batch][tokens] grid)."""
    keep = []

    def arr(k):
        a, p = _arr(profile[k])
        keep.append(a)
        return p

    pr = Profile()
    pr.gatt_n = len(profile["gatt_tokens"])
    pr.gatt_tokens, pr.gatt_seconds = arr("gatt_tokens"), arr("gatt_seconds")
    pr.glin_n = len(profile["glin_batch"])
    pr.glin_batch, pr.glin_seconds = arr("glin_batch"), arr("glin_seconds")
    pr.cpu_nb, pr.cpu_nt = len(profile["cpu_batch"]), len(profile["cpu_tokens"])
    pr.cpu_batch, pr.cpu_tokens = arr("cpu_batch"), arr("cpu_tokens")
    grid = np.ascontiguousarray(np.asarray(profile["cpu_seconds"], dtype=np.float64).reshape(-1))
    keep.append(grid)
    pr.cpu_seconds = grid.ctypes.data_as(_DP)
    if profile.get("pref_tokens"):
        pr.pref_n = len(profile["pref_tokens"])
        pr.pref_tokens = arr("pref_tokens")
        pr.pref_linear_seconds, pr.pref_attn_seconds = arr("pref_linear_seconds"), arr("pref_attn_seconds")
    out = Inputs()
    _check(_lib().apex_sched_inputs_from_profile(ctypes.byref(pr), float(gpu_batch), float(gpu_tokens),
                                                 float(cpu_batch), float(cpu_tokens), float(prefill_tokens),
                                                 MIXED_FORMS[mixed_form], ctypes.byref(out)))
    d = {"n_g": out.n_g, "n_c": out.n_c, "t_glinear": out.t_glinear, "t_gatt": out.t_gatt}
    if out.prefill:
        d.update(prefill=True, t_glinear_pref=out.t_glinear_pref, t_gatt_pref=out.t_gatt_pref,
                 mixed_form=mixed_form)
    return d


def gpu_token_capacity(free_bytes, layers, Hkv, d, bytes_per_element=2):
    return int(_lib().apex_sched_gpu_token_capacity(float(free_bytes), layers, Hkv, d, bytes_per_element))
