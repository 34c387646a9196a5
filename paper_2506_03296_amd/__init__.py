"""Python binding of libapex_decode.so: batched paged decode attention on MI355X.

Argument marshalling only.  Every step of the attention runs in the HIP
kernels of the library; torch provides device memory and the current stream.
If the built library is missing, importing the binding's functions raises --
there is no fallback.

    out = decode_attention(q, k_cache, v_cache, block_table, context_lens, scale)
    kv_append(k_new, v_new, k_cache, v_cache, slot_mapping)      # before the step

q [B][Hq][128] fp16, caches [num_blocks][Hkv][16][128] fp16, block_table int32
[B][stride], context_lens int32 [B] (all on the same GPU).  The names and
argument order follow include/apex_decode.h and include/apex_kv_append.h.
"""
import ctypes
import os

__all__ = [
    "ApexError", "LIB_PATH", "load_library", "decode_attention", "decode_attention_ex",
    "workspace_bytes", "plan_host", "last_error", "release_workspace", "version",
    "APEX_OK", "APEX_ERR_INVALID_ARG", "APEX_ERR_UNSUPPORTED", "APEX_ERR_OUT_OF_MEMORY",
    "APEX_ERR_HIP", "EXPORTED_SYMBOLS", "counter_bytes", "kv_append", "check_device_error",
    "FLAG_CHECK_INPUTS", "DEVICE_ERR_BLOCK_ID", "DEVICE_ERR_TABLE_ROW", "decode_attention_noalloc",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libapex_decode.so")

APEX_OK = 0
APEX_ERR_INVALID_ARG = -1
APEX_ERR_UNSUPPORTED = -2
APEX_ERR_OUT_OF_MEMORY = -3
APEX_ERR_HIP = -4

EXPORTED_SYMBOLS = (
    "apex_decode_attention", "apex_decode_attention_ex", "apex_decode_workspace_bytes",
    "apex_decode_counter_bytes", "apex_decode_plan_host", "apex_decode_last_error",
    "apex_decode_release_workspace", "apex_decode_version", "apex_kv_append",
    "apex_decode_check_device_error", "apex_decode_attention_noalloc",
)
FLAG_CHECK_INPUTS = 1
DEVICE_ERR_BLOCK_ID = 1
DEVICE_ERR_TABLE_ROW = 2


class ApexError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"apex_decode error {code}: {msg}")
        self.code = code


class DecodeArgs(ctypes.Structure):
    """Mirror of apex_decode_args (include/apex_decode.h)."""
    _fields_ = [
        ("q", ctypes.c_void_p), ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p), ("context_lens", ctypes.c_void_p),
        ("out", ctypes.c_void_p),
        ("B", ctypes.c_int), ("Hq", ctypes.c_int), ("Hkv", ctypes.c_int), ("d", ctypes.c_int),
        ("block_size", ctypes.c_int), ("scale", ctypes.c_float), ("stream", ctypes.c_void_p),
        ("block_table_stride", ctypes.c_int64), ("num_workers", ctypes.c_int),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t), ("lse_out", ctypes.c_void_p),
        ("attn_kernel_events", ctypes.c_void_p * 2), ("flags", ctypes.c_uint32),
        ("num_blocks", ctypes.c_int64),
        ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p), ("new_token_stride", ctypes.c_int64),
    ]


_LIB = None


def load_library(path=None):
    """Load (once) and return the ctypes handle of libapex_decode.so."""
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    p = path or LIB_PATH
    try:
        # torch ships its own HIP runtime; loading it first lets this library
        # bind to that same runtime instead of a second copy from /opt/rocm
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(p):
        raise ApexError(APEX_ERR_HIP, f"{p} is not built; run __graft_entry__.build() "
                                      "(python -m paper_2506_03296_amd.build)")
    lib = ctypes.CDLL(p)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.apex_decode_attention.restype = i32
    lib.apex_decode_attention.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                          ctypes.c_float, vp]
    lib.apex_decode_attention_noalloc.restype = i32
    lib.apex_decode_attention_noalloc.argtypes = lib.apex_decode_attention.argtypes
    lib.apex_decode_attention_ex.restype = i32
    lib.apex_decode_attention_ex.argtypes = [ctypes.POINTER(DecodeArgs)]
    lib.apex_decode_workspace_bytes.restype = ctypes.c_size_t
    lib.apex_decode_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    lib.apex_decode_counter_bytes.restype = ctypes.c_size_t
    lib.apex_decode_counter_bytes.argtypes = [i32, i32]
    lib.apex_decode_plan_host.restype = i32
    lib.apex_decode_plan_host.argtypes = [vp, i32, i32, i32, i32, i32, i32, vp,
                                          ctypes.POINTER(i64), ctypes.POINTER(i64),
                                          ctypes.POINTER(i64)]
    lib.apex_decode_last_error.restype = ctypes.c_char_p
    lib.apex_decode_last_error.argtypes = []
    lib.apex_decode_release_workspace.restype = i32
    lib.apex_decode_release_workspace.argtypes = []
    lib.apex_decode_version.restype = i32
    lib.apex_decode_version.argtypes = []
    lib.apex_decode_check_device_error.restype = i32
    lib.apex_decode_check_device_error.argtypes = [ctypes.POINTER(ctypes.c_uint32)]
    lib.apex_kv_append.restype = i32
    lib.apex_kv_append.argtypes = [vp, vp, i64, vp, vp, vp, i32, i32, i32, i32, i64, vp]
    if path is None:
        _LIB = lib
    return lib


def last_error():
    return load_library().apex_decode_last_error().decode()


def _check(rc):
    if rc != APEX_OK:
        raise ApexError(rc, last_error())


def version():
    return load_library().apex_decode_version()


def release_workspace():
    _check(load_library().apex_decode_release_workspace())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _addr(t):
    return None if t is None else int(t.data_ptr())


def _event_handle(ev, stream):
    """Raw hipEvent_t of a torch.cuda.Event (created on first use)."""
    if not ev.cuda_event:
        ev.record(stream)
    return int(ev.cuda_event)


def _stream_obj(stream, device):
    import torch
    return stream if stream is not None else torch.cuda.current_stream(device)


def _stream_handle(stream, device):
    return ctypes.c_void_p(_stream_obj(stream, device).cuda_stream)


def _require(t, name, dtype, device, shape=None, contiguous=True):
    """The library reads raw device pointers: a tensor of another dtype, on
    the host or on another device, or with gaps would be read as garbage (or
    fault the GPU), so such arguments are refused here."""
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _shapes(q, k_cache):
    if q.dim() != 3 or k_cache.dim() != 4:
        raise ValueError("q must be [B][Hq][d] and the caches [num_blocks][Hkv][block_size][d]")
    B, Hq, d = q.shape
    _, Hkv, bs, dk = k_cache.shape
    if dk != d:
        raise ValueError("q and the caches disagree on the head dim")
    return B, Hq, Hkv, d, bs


def _check_tensors(q, k_cache, v_cache, block_table, context_lens, out, block_table_stride=0):
    """dtype, device, shape and layout of the attention's tensors."""
    import torch
    B, Hq, Hkv, d, bs = _shapes(q, k_cache)
    dev = q.device
    if dev.type != "cuda":
        raise ValueError(f"q must be a GPU tensor, got {dev}")
    _require(q, "q", torch.float16, dev)
    _require(k_cache, "k_cache", torch.float16, dev)
    _require(v_cache, "v_cache", torch.float16, dev, shape=k_cache.shape)
    _require(context_lens, "context_lens", torch.int32, dev, shape=(B,))
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError(f"block_table must be [B={B}][entries per row], got {tuple(block_table.shape)}")
    if block_table_stride and block_table.shape[1] != block_table_stride:
        raise ValueError(f"block_table rows hold {block_table.shape[1]} entries, "
                         f"block_table_stride says {block_table_stride}")
    _require(block_table, "block_table", torch.int32, dev)
    if out is not None:
        _require(out, "out", torch.float16, dev, shape=(B, Hq, d))
    return B, Hq, Hkv, d, bs


def decode_attention(q, k_cache, v_cache, block_table, context_lens, scale, out=None,
                     stream=None):
    """apex_decode_attention over torch tensors; returns ``out``.

    The block table must be tight ([B][ceil(max L / 16)]); use
    ``decode_attention_ex`` for wider rows."""
    import torch
    B, Hq, Hkv, d, bs = _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    lib = load_library()
    rc = lib.apex_decode_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                   _ptr(context_lens), _ptr(out), B, Hq, Hkv, d, bs,
                                   ctypes.c_float(scale), _stream_handle(stream, q.device))
    _check(rc)
    return out


def decode_attention_noalloc(q, k_cache, v_cache, block_table, context_lens, scale, out,
                             stream=None):
    """apex_decode_attention_noalloc over torch tensors (the library
    allocates nothing; ``out`` is the caller's); returns ``out``.  The block
    table must be tight, as for ``decode_attention``."""
    if out is None:
        raise ValueError("decode_attention_noalloc writes into the caller's out")
    B, Hq, Hkv, d, bs = _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    lib = load_library()
    rc = lib.apex_decode_attention_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_table),
                                           _ptr(context_lens), _ptr(out), B, Hq, Hkv, d, bs,
                                           ctypes.c_float(scale), _stream_handle(stream, q.device))
    _check(rc)
    return out


def decode_attention_ex(q, k_cache, v_cache, block_table, context_lens, scale, out=None,
                        block_table_stride=0, num_workers=0, workspace=None,
                        lse_out=None, events=None, stream=None, check_inputs=False,
                        k_new=None, v_new=None):
    """apex_decode_attention_ex over torch tensors; returns ``out``.

    ``workspace`` is an optional uint8 device tensor (caller-owned; its first
    counter_bytes(B, Hkv) bytes must be zero, e.g. from torch.zeros);
    ``events`` an optional pair of torch.cuda.Event recorded around the
    attention kernel; ``check_inputs`` runs the input-checking kernel (block
    ids against the caches' block count; see check_device_error);
    ``k_new``/``v_new`` (fp16 [B][Hkv][d], unit strides inside a token) turn
    on the fused append: the current token (position L - 1) is attended from
    them and written to its cache slot in the same launch."""
    import torch
    B, Hq, Hkv, d, bs = _check_tensors(q, k_cache, v_cache, block_table, context_lens, out,
                                       block_table_stride)
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    if lse_out is not None:
        _require(lse_out, "lse_out", torch.float32, q.device, shape=(B, Hq))
    if workspace is not None:
        _require(workspace, "workspace", torch.uint8, q.device)
    a = DecodeArgs()
    a.q, a.k_cache, a.v_cache = _addr(q), _addr(k_cache), _addr(v_cache)
    a.block_table, a.context_lens, a.out = _addr(block_table), _addr(context_lens), _addr(out)
    a.B, a.Hq, a.Hkv, a.d, a.block_size = B, Hq, Hkv, d, bs
    a.scale = float(scale)
    s = _stream_obj(stream, q.device)
    a.stream = int(s.cuda_stream)
    a.block_table_stride = int(block_table_stride)
    a.num_workers = int(num_workers)
    if workspace is not None:
        a.workspace = _addr(workspace)
        a.workspace_bytes = workspace.numel() * workspace.element_size()
    a.lse_out = _addr(lse_out)
    if events is not None:
        a.attn_kernel_events[0] = _event_handle(events[0], s)
        a.attn_kernel_events[1] = _event_handle(events[1], s)
    if check_inputs:
        a.flags = FLAG_CHECK_INPUTS
        a.num_blocks = k_cache.shape[0]
    if k_new is not None or v_new is not None:
        if k_new is None or v_new is None or k_new.shape != (B, Hkv, d) or v_new.shape != k_new.shape:
            raise ValueError("k_new and v_new must both be [B][Hkv][d]")
        _require(k_new, "k_new", torch.float16, q.device, contiguous=False)
        _require(v_new, "v_new", torch.float16, q.device, contiguous=False)
        if k_new.stride(2) != 1 or k_new.stride(1) != d or v_new.stride() != k_new.stride():
            raise ValueError("k_new/v_new need unit strides inside a token and equal strides")
        a.k_new, a.v_new = _addr(k_new), _addr(v_new)
        a.new_token_stride = int(k_new.stride(0))
    _check(load_library().apex_decode_attention_ex(ctypes.byref(a)))
    return out


def check_device_error():
    """Waits for the current device and returns (and clears) the error bits
    set by input-checking calls (DEVICE_ERR_*; 0 = none)."""
    bits = ctypes.c_uint32()
    _check(load_library().apex_decode_check_device_error(ctypes.byref(bits)))
    return bits.value


def workspace_bytes(B, Hq, Hkv, d=128, block_size=16, num_workers=0):
    return int(load_library().apex_decode_workspace_bytes(B, Hq, Hkv, d, block_size, num_workers))


def counter_bytes(B, Hkv):
    return int(load_library().apex_decode_counter_bytes(B, Hkv))


def plan_host(context_lens, Hkv, launched_workers, block_size=16, forced=False, cus=0):
    """Host mirror of the work partition (no GPU).  ``cus`` = the device's
    compute units for the one-group-per-CU rule of the default grid (0 = off).
    Returns a dict with 'contributors' (numpy int32 [B][Hkv]: work groups
    sharing each pair) and the scalars 'units', 'active' and 'partials'."""
    import numpy as np
    lens = np.ascontiguousarray(np.asarray(context_lens), dtype=np.int32)
    B = lens.shape[0]
    contrib = np.zeros(max(B * Hkv, 1), dtype=np.int32)
    units, active, partials = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    rc = load_library().apex_decode_plan_host(
        lens.ctypes.data if B else None, B, Hkv, block_size, launched_workers, int(bool(forced)),
        int(cus), contrib.ctypes.data, ctypes.byref(units), ctypes.byref(active), ctypes.byref(partials))
    _check(rc)
    return {"contributors": contrib[:B * Hkv].reshape(B, Hkv), "units": units.value,
            "active": active.value, "partials": partials.value}


def kv_append(k_new, v_new, k_cache, v_cache, slot_mapping, stream=None):
    """apex_kv_append over torch tensors (in place on the caches).

    k_new/v_new: fp16 [T][Hkv][d] with unit strides inside a token (the token
    stride may be wider, e.g. views into a fused QKV buffer, but must be the
    same for both); caches [num_blocks][Hkv][block_size][d]; slot_mapping
    int64 [T] (negative = padding)."""
    if k_new.dim() != 3 or v_new.shape != k_new.shape or k_cache.dim() != 4:
        raise ValueError("k_new/v_new must be [T][Hkv][d]; caches [num_blocks][Hkv][block_size][d]")
    T, Hkv, d = k_new.shape
    nb, hkv2, bs, d2 = k_cache.shape
    if (hkv2, d2) != (Hkv, d) or v_cache.shape != k_cache.shape:
        raise ValueError("new rows and caches disagree on Hkv or d")
    for t in (k_new, v_new):
        if t.stride(2) != 1 or t.stride(1) != d:
            raise ValueError("each token's rows must be contiguous [Hkv][d]")
    if T > 1 and k_new.stride(0) != v_new.stride(0):
        raise ValueError("k_new and v_new must share the token stride")
    import torch
    dev = k_cache.device
    if dev.type != "cuda":
        raise ValueError(f"the caches must be GPU tensors, got {dev}")
    _require(k_cache, "k_cache", torch.float16, dev)
    _require(v_cache, "v_cache", torch.float16, dev)
    _require(k_new, "k_new", torch.float16, dev, contiguous=False)
    _require(v_new, "v_new", torch.float16, dev, contiguous=False)
    _require(slot_mapping, "slot_mapping", torch.int64, dev, shape=(T,))
    stride = k_new.stride(0) if T > 1 else 0
    rc = load_library().apex_kv_append(_ptr(k_new), _ptr(v_new), stride, _ptr(k_cache),
                                       _ptr(v_cache), _ptr(slot_mapping), T, Hkv, d, bs, nb,
                                       _stream_handle(stream, k_cache.device))
    _check(rc)
