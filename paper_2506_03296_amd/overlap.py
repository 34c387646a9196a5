"""Python binding of libapex_overlap.so: the Asynchronous Overlap runtime
(include/apex_overlap.h).  Argument marshalling only.

    rt = Overlap(layers=32, max_requests=64, Hq=32, Hkv=8, d=128, block_size=16,
                 scale=128 ** -0.5, num_blocks=..., max_blocks_per_request=...)
    k, v = rt.host_cache(layer)                 # numpy views of the pinned caches
    t = rt.submit(layer, q, k_new, v_new, slots, table, lens)   # device q/k/v rows
    ...
    if rt.poll(t, out):                         # non-blocking readiness check
        ...                                     # out gets the result (stream-ordered)
    rt.wait(t, out)                             # blocking
    rt.close()
"""
import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libapex_overlap.so")

EXPORTED_SYMBOLS = (
    "apex_overlap_create", "apex_overlap_host_cache", "apex_overlap_submit", "apex_overlap_poll",
    "apex_overlap_wait", "apex_overlap_hold", "apex_overlap_pending", "apex_overlap_destroy",
    "apex_overlap_last_error",
)

APEX_ERR_BUSY = -5


class Config(ctypes.Structure):
    """Mirror of apex_overlap_config."""
    _fields_ = [("layers", ctypes.c_int), ("max_requests", ctypes.c_int), ("Hq", ctypes.c_int),
                ("Hkv", ctypes.c_int), ("d", ctypes.c_int), ("block_size", ctypes.c_int),
                ("scale", ctypes.c_float), ("num_blocks", ctypes.c_int64),
                ("max_blocks_per_request", ctypes.c_int), ("threads", ctypes.c_int),
                ("slots_per_layer", ctypes.c_int)]


class OverlapError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"apex_overlap error {code}: {msg}")
        self.code = code


_LIB = None


def load_library(path=None):
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    try:
        import torch  # noqa: F401  (same HIP runtime as torch)
    except ImportError:
        pass
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise OverlapError(-4, f"{p} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(p)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.apex_overlap_create.restype = i32
    lib.apex_overlap_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(vp)]
    lib.apex_overlap_host_cache.restype = i32
    lib.apex_overlap_host_cache.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(vp)]
    lib.apex_overlap_submit.restype = i32
    lib.apex_overlap_submit.argtypes = [vp, i32, vp, vp, vp, vp, vp, i64, vp, i32, vp,
                                        ctypes.POINTER(i64)]
    lib.apex_overlap_poll.restype = i32
    lib.apex_overlap_poll.argtypes = [vp, i64, vp, vp, ctypes.POINTER(i32)]
    lib.apex_overlap_wait.restype = i32
    lib.apex_overlap_wait.argtypes = [vp, i64, vp, vp]
    lib.apex_overlap_hold.restype = i32
    lib.apex_overlap_hold.argtypes = [vp, i32]
    lib.apex_overlap_pending.restype = i32
    lib.apex_overlap_pending.argtypes = [vp]
    lib.apex_overlap_destroy.restype = i32
    lib.apex_overlap_destroy.argtypes = [vp]
    lib.apex_overlap_last_error.restype = ctypes.c_char_p
    lib.apex_overlap_last_error.argtypes = []
    if path is None:
        _LIB = lib
    return lib


def last_error():
    return load_library().apex_overlap_last_error().decode()


def _check(rc):
    if rc != 0:
        raise OverlapError(rc, last_error())


def _stream(stream, device):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _host(a, dtype):
    a = np.ascontiguousarray(np.asarray(a), dtype=dtype)
    return a


class Overlap:
    def __init__(self, layers, max_requests, Hq, Hkv, d, block_size, scale, num_blocks,
                 max_blocks_per_request, threads=0, slots_per_layer=0):
        self.cfg = Config(layers, max_requests, Hq, Hkv, d, block_size, float(scale), num_blocks,
                          max_blocks_per_request, threads, slots_per_layer)
        self._lib = load_library()
        h = ctypes.c_void_p()
        _check(self._lib.apex_overlap_create(ctypes.byref(self.cfg), ctypes.byref(h)))
        self._h = h

    def host_cache(self, layer):
        """(k, v) numpy float16 views [num_blocks][Hkv][block_size][d] of the
        runtime's pinned host cache of ``layer`` (valid until close())."""
        k, v = ctypes.c_void_p(), ctypes.c_void_p()
        _check(self._lib.apex_overlap_host_cache(self._h, layer, ctypes.byref(k), ctypes.byref(v)))
        c = self.cfg
        shape = (c.num_blocks, c.Hkv, c.block_size, c.d)
        n = int(np.prod(shape))
        mk = np.ctypeslib.as_array(ctypes.cast(k, ctypes.POINTER(ctypes.c_uint16)), shape=(n,))
        mv = np.ctypeslib.as_array(ctypes.cast(v, ctypes.POINTER(ctypes.c_uint16)), shape=(n,))
        return mk.view(np.float16).reshape(shape), mv.view(np.float16).reshape(shape)

    def submit(self, layer, q, k_new, v_new, slot_mapping, block_table, context_lens,
               stream=None, block_table_stride=0):
        slots = _host(slot_mapping, np.int64)
        table = _host(block_table, np.int32)
        lens = _host(context_lens, np.int32)
        B = int(q.shape[0])
        t = ctypes.c_int64()
        _check(self._lib.apex_overlap_submit(
            self._h, layer, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k_new.data_ptr()),
            ctypes.c_void_p(v_new.data_ptr()), slots.ctypes.data, table.ctypes.data,
            int(block_table_stride or table.shape[1]), lens.ctypes.data, B,
            _stream(stream, q.device), ctypes.byref(t)))
        return t.value

    def poll(self, ticket, out, stream=None):
        ready = ctypes.c_int()
        _check(self._lib.apex_overlap_poll(self._h, ticket, ctypes.c_void_p(out.data_ptr()),
                                           _stream(stream, out.device), ctypes.byref(ready)))
        return bool(ready.value)

    def wait(self, ticket, out, stream=None):
        _check(self._lib.apex_overlap_wait(self._h, ticket, ctypes.c_void_p(out.data_ptr()),
                                           _stream(stream, out.device)))

    def hold(self, flag=True):
        _check(self._lib.apex_overlap_hold(self._h, int(bool(flag))))

    def pending(self):
        return self._lib.apex_overlap_pending(self._h)

    def close(self):
        if getattr(self, "_h", None):
            h, self._h = self._h, None
            _check(self._lib.apex_overlap_destroy(h))

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
