"""Python binding of libapex_cpu.so: paged decode attention on the host cores.

Argument marshalling only; the attention runs in the library's C++/SIMD code.
Inputs are host arrays (numpy, or CPU torch tensors) in the layout of
include/apex_cpu_attention.h -- the same layout the GPU library reads:

    out = decode_attention(q, k_cache, v_cache, block_table, context_lens, scale)

q fp16 [B][Hq][d], caches fp16 [num_blocks][Hkv][block_size][d], block_table
int32 [B][stride], context_lens int32 [B].  Returns fp16 [B][Hq][d] (and the
natural-log LSE [B][Hq] with ``return_lse``).  The library releases nothing
of the caller's and the GIL is released for the duration of the call
(ctypes), so a Python thread can run it beside GPU work.
"""
import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libapex_cpu.so")

EXPORTED_SYMBOLS = (
    "apex_cpu_decode_attention", "apex_cpu_decode_attention_ex", "apex_cpu_set_threads",
    "apex_cpu_threads", "apex_cpu_isa", "apex_cpu_read_bandwidth", "apex_cpu_last_error",
)
FLAG_FORCE_AVX2 = 1


class CpuArgs(ctypes.Structure):
    """Mirror of apex_cpu_args (include/apex_cpu_attention.h)."""
    _fields_ = [
        ("q", ctypes.c_void_p), ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p), ("context_lens", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("B", ctypes.c_int), ("Hq", ctypes.c_int), ("Hkv", ctypes.c_int), ("d", ctypes.c_int),
        ("block_size", ctypes.c_int), ("scale", ctypes.c_float),
        ("block_table_stride", ctypes.c_int64), ("lse_out", ctypes.c_void_p),
        ("num_threads", ctypes.c_int), ("min_chunk_tokens", ctypes.c_int),
        ("flags", ctypes.c_uint32),
    ]


class CpuError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"apex_cpu error {code}: {msg}")
        self.code = code


_LIB = None


def load_library(path=None):
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise CpuError(-4, f"{p} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(p)
    vp, i32 = ctypes.c_void_p, ctypes.c_int
    lib.apex_cpu_decode_attention.restype = i32
    lib.apex_cpu_decode_attention.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                              ctypes.c_float]
    lib.apex_cpu_decode_attention_ex.restype = i32
    lib.apex_cpu_decode_attention_ex.argtypes = [ctypes.POINTER(CpuArgs)]
    lib.apex_cpu_set_threads.restype = i32
    lib.apex_cpu_set_threads.argtypes = [i32]
    lib.apex_cpu_threads.restype = i32
    lib.apex_cpu_threads.argtypes = []
    lib.apex_cpu_isa.restype = i32
    lib.apex_cpu_isa.argtypes = []
    lib.apex_cpu_read_bandwidth.restype = ctypes.c_double
    lib.apex_cpu_read_bandwidth.argtypes = [ctypes.c_size_t, i32, i32]
    lib.apex_cpu_last_error.restype = ctypes.c_char_p
    lib.apex_cpu_last_error.argtypes = []
    if path is None:
        _LIB = lib
    return lib


def last_error():
    return load_library().apex_cpu_last_error().decode()


def _check(rc):
    if rc != 0:
        raise CpuError(rc, last_error())


def isa():
    """2 = AVX-512, 1 = AVX2, 0 = unsupported CPU."""
    return load_library().apex_cpu_isa()


def threads():
    return load_library().apex_cpu_threads()


def set_threads(n):
    _check(load_library().apex_cpu_set_threads(int(n)))


def read_bandwidth(nbytes=1 << 30, num_threads=0, reps=5):
    """Host read bandwidth (GB/s) with the library's own threads."""
    n = num_threads or threads()
    v = load_library().apex_cpu_read_bandwidth(int(nbytes), int(n), int(reps))
    if v < 0:
        raise CpuError(-1, last_error())
    return v


def _host(a, dtype):
    if hasattr(a, "numpy"):          # CPU torch tensor
        a = a.numpy()
    a = np.asarray(a)
    if dtype == np.float16 and a.dtype == np.uint16:
        a = a.view(np.float16)
    if a.dtype != dtype:
        raise TypeError(f"expected {np.dtype(dtype)}, got {a.dtype}")
    if not a.flags.c_contiguous:
        raise ValueError("arrays must be C-contiguous")
    return a


def decode_attention(q, k_cache, v_cache, block_table, context_lens, scale, out=None,
                     return_lse=False, block_table_stride=0, num_threads=0,
                     min_chunk_tokens=0, force_avx2=False):
    """apex_cpu_decode_attention_ex over host arrays; returns out (fp16)."""
    q = _host(q, np.float16)
    k = _host(k_cache, np.float16)
    v = _host(v_cache, np.float16)
    bt = _host(block_table, np.int32)
    lens = _host(context_lens, np.int32)
    if q.ndim != 3 or k.ndim != 4 or v.shape != k.shape:
        raise ValueError("q must be [B][Hq][d]; caches [num_blocks][Hkv][block_size][d]")
    B, Hq, d = q.shape
    _, Hkv, bs, dk = k.shape
    if dk != d or lens.shape != (B,) or bt.ndim != 2 or bt.shape[0] != B:
        raise ValueError("shape mismatch")
    if out is None:
        out = np.empty((B, Hq, d), dtype=np.float16)
    out = _host(out, np.float16)
    lse = np.empty((B, Hq), dtype=np.float32) if return_lse else None
    a = CpuArgs()
    a.q, a.k_cache, a.v_cache = q.ctypes.data, k.ctypes.data, v.ctypes.data
    a.block_table, a.context_lens, a.out = bt.ctypes.data, lens.ctypes.data, out.ctypes.data
    a.B, a.Hq, a.Hkv, a.d, a.block_size = B, Hq, Hkv, d, bs
    a.scale = float(scale)
    a.block_table_stride = int(block_table_stride or bt.shape[1])
    a.lse_out = lse.ctypes.data if lse is not None else None
    a.num_threads = int(num_threads)
    a.min_chunk_tokens = int(min_chunk_tokens)
    a.flags = FLAG_FORCE_AVX2 if force_avx2 else 0
    _check(load_library().apex_cpu_decode_attention_ex(ctypes.byref(a)))
    return (out, lse) if return_lse else out
