"""fp64 CPU oracle for batched paged decode attention -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it.

``decode_attention_f64`` wraps the plain C definition in ``ref_decode.c``
(scaled-dot-product softmax attention per request and q-head over that
request's paged KV; APEX Sec. 3.1 and Sec. 3.3 state that the GPU attends its
requests' cached KV with the same mathematics wherever it runs).
``brute_force`` holds an independent pure-Python restatement used to pin it.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build(quiet=True)
        lib = ctypes.CDLL(_build.LIB)
        lib.apex_oracle_f16_to_f64.restype = ctypes.c_double
        lib.apex_oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
        lib.apex_oracle_f16_to_f64_array.restype = None
        lib.apex_oracle_f16_to_f64_array.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]
        lib.apex_oracle_decode_attention_f64.restype = ctypes.c_int
        lib.apex_oracle_decode_attention_f64.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_long,
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
        lib.apex_oracle_softmax_weights_f64.restype = ctypes.c_int
        lib.apex_oracle_softmax_weights_f64.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_long,
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.c_int, ctypes.c_float, ctypes.c_void_p]
        lib.apex_oracle_max_threads.restype = ctypes.c_int
        lib.apex_oracle_max_threads.argtypes = []
        _LIB = lib
    return _LIB


def _bits(a):
    """fp16 array (numpy float16 or uint16 view) -> contiguous uint16 bits."""
    a = np.asarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError(f"expected float16/uint16 bits, got {a.dtype}")
    return np.ascontiguousarray(a)


def _i32(a):
    a = np.ascontiguousarray(np.asarray(a), dtype=np.int32)
    return a


def f16_bits_to_f64(bits):
    """Decode fp16 bit patterns with the oracle's own IEEE-754 binary16 decoder."""
    b = _bits(bits)
    out = np.empty(b.shape, dtype=np.float64)
    _lib().apex_oracle_f16_to_f64_array(b.ctypes.data, out.ctypes.data, b.size)
    return out


def max_threads():
    return _lib().apex_oracle_max_threads()


def decode_attention_f64(q, k_cache, v_cache, block_table, context_lens, scale,
                         num_threads=0, return_lse=False):
    """Exact fp64 decode attention.

    q [B][Hq][d], k_cache/v_cache [NB][Hkv][bs][d] as fp16 (or uint16 bits),
    block_table int32 [B][stride], context_lens int32 [B], scale as fp32.
    Returns out float64 [B][Hq][d] (and lse float64 [B][Hq], natural log).
    """
    qb, kb, vb = _bits(q), _bits(k_cache), _bits(v_cache)
    bt, lens = _i32(block_table), _i32(context_lens)
    if qb.ndim != 3 or kb.ndim != 4 or kb.shape != vb.shape:
        raise ValueError("q must be [B][Hq][d]; caches [NB][Hkv][bs][d]")
    B, Hq, d = qb.shape
    _, Hkv, bs, d2 = kb.shape
    if d2 != d or lens.shape != (B,) or bt.ndim != 2 or bt.shape[0] != B:
        raise ValueError("shape mismatch")
    out = np.zeros((B, Hq, d), dtype=np.float64)
    lse = np.zeros((B, Hq), dtype=np.float64)
    rc = _lib().apex_oracle_decode_attention_f64(
        qb.ctypes.data, kb.ctypes.data, vb.ctypes.data, bt.ctypes.data, bt.shape[1],
        lens.ctypes.data, B, Hq, Hkv, d, bs, float(np.float32(scale)), out.ctypes.data,
        lse.ctypes.data, int(num_threads))
    if rc != 0:
        raise ValueError("oracle rejected the shapes")
    return (out, lse) if return_lse else out


def softmax_weights_f64(q, k_cache, v_cache, block_table, context_lens, scale, b, h):
    """Softmax weights of (request b, q-head h) over its context_lens[b] tokens."""
    qb, kb, vb = _bits(q), _bits(k_cache), _bits(v_cache)
    bt, lens = _i32(block_table), _i32(context_lens)
    B, Hq, d = qb.shape
    _, Hkv, bs, _ = kb.shape
    L = max(int(lens[b]), 0)
    w = np.zeros(max(L, 1), dtype=np.float64)
    rc = _lib().apex_oracle_softmax_weights_f64(
        qb.ctypes.data, kb.ctypes.data, vb.ctypes.data, bt.ctypes.data, bt.shape[1],
        lens.ctypes.data, int(b), int(h), Hq, Hkv, d, bs, float(np.float32(scale)), w.ctypes.data)
    if rc != 0:
        raise ValueError("oracle rejected the shapes")
    return w[:L]
