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
        self._rows = {}   # ticket -> rows of its result, until collected

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

    def _check_rows(self, t, name, heads, B):
        """q/k_new/v_new/out: contiguous fp16 GPU tensors [B][heads][d] (the
        runtime copies them as raw device bytes)."""
        import torch
        if t.device.type != "cuda" or t.dtype != torch.float16 or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float16 GPU tensor")
        if tuple(t.shape) != (B, heads, self.cfg.d):
            raise ValueError(f"{name} must have shape {(B, heads, self.cfg.d)}, got {tuple(t.shape)}")

    def submit(self, layer, q, k_new, v_new, slot_mapping, block_table, context_lens,
               stream=None, block_table_stride=0):
        slots = _host(slot_mapping, np.int64)
        table = _host(block_table, np.int32)
        lens = _host(context_lens, np.int32)
        B = int(q.shape[0])
        self._check_rows(q, "q", self.cfg.Hq, B)
        self._check_rows(k_new, "k_new", self.cfg.Hkv, B)
        self._check_rows(v_new, "v_new", self.cfg.Hkv, B)
        if slots.shape != (B,) or lens.shape != (B,):
            raise ValueError(f"slot_mapping and context_lens must hold B = {B} entries")
        if table.ndim != 2 or table.shape[0] != B:
            raise ValueError(f"block_table must be [B = {B}][entries per row]")
        if block_table_stride and block_table_stride != table.shape[1]:
            raise ValueError("block_table_stride must equal the table's row length")
        t = ctypes.c_int64()
        _check(self._lib.apex_overlap_submit(
            self._h, layer, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k_new.data_ptr()),
            ctypes.c_void_p(v_new.data_ptr()), slots.ctypes.data, table.ctypes.data,
            int(block_table_stride or table.shape[1]), lens.ctypes.data, B,
            _stream(stream, q.device), ctypes.byref(t)))
        self._rows[t.value] = B
        return t.value

    def poll(self, ticket, out, stream=None):
        self._check_out(out, ticket)
        ready = ctypes.c_int()
        _check(self._lib.apex_overlap_poll(self._h, ticket, ctypes.c_void_p(out.data_ptr()),
                                           _stream(stream, out.device), ctypes.byref(ready)))
        if ready.value:
            self._rows.pop(ticket, None)
        return bool(ready.value)

    def wait(self, ticket, out, stream=None):
        self._check_out(out, ticket)
        _check(self._lib.apex_overlap_wait(self._h, ticket, ctypes.c_void_p(out.data_ptr()),
                                           _stream(stream, out.device)))
        self._rows.pop(ticket, None)

    def _check_out(self, out, ticket):
        """out receives the ticket's B rows [B][Hq][d] as raw device bytes."""
        import torch
        if out.device.type != "cuda" or out.dtype != torch.float16 or not out.is_contiguous():
            raise ValueError("out must be a contiguous float16 GPU tensor")
        if out.dim() != 3 or tuple(out.shape[1:]) != (self.cfg.Hq, self.cfg.d):
            raise ValueError(f"out must be [B][{self.cfg.Hq}][{self.cfg.d}], got {tuple(out.shape)}")
        rows = self._rows.get(ticket)
        if rows is not None and out.shape[0] < rows:
            raise ValueError(f"out holds {out.shape[0]} rows, the ticket's result has {rows}")

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
