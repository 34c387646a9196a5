"""Binding of libapex_hbm_probe.so: achievable HBM read bandwidth on this GPU.

Two patterns, timed with HIP events on the current stream: a sequential
128-bit stream over a large buffer, and the decode-attention pattern -- 4 KiB
chunks (one block of one kv-head) read in a random order.
"""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libapex_hbm_probe.so")
_LIB = None


def load_library():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built")
        lib = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        lib.apex_hbm_probe_stream.restype = ctypes.c_int
        lib.apex_hbm_probe_stream.argtypes = [vp, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, vp, vp]
        lib.apex_hbm_probe_gather.restype = ctypes.c_int
        lib.apex_hbm_probe_gather.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                              vp, vp]
        _LIB = lib
    return _LIB


def _time(torch, fn, reps):
    fn()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps * 1e-3


def measure(nbytes=4 << 30, reps=10, blocks_list=(0,), seed=0):
    """Returns GB/s per (pattern, flags, blocks): "stream" (flags = nt),
    "gather4k" (flags = nt | chunks-in-flight << 1) and "gather4k_dev" (the
    attention kernel's access form: a buffer resource per chunk,
    non-temporal buffer loads)."""
    import torch
    lib = load_library()
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_chunks = nbytes // 4096
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    ids = torch.randperm(n_chunks, generator=g, device="cuda").to(torch.int32)
    stream = torch.cuda.current_stream().cuda_stream
    res = {"bytes": nbytes, "stream": {}, "gather4k": {}, "gather4k_dev": {}}
    for blocks in blocks_list:
        for nt in (0, 1):
            def f1():
                rc = lib.apex_hbm_probe_stream(buf.data_ptr(), nbytes, blocks, nt, sink.data_ptr(),
                                               stream)
                assert rc == 0
            res["stream"][f"nt{nt}_wg{blocks}"] = round(nbytes / _time(torch, f1, reps) / 1e9, 1)
            for unroll in (1, 2, 4):
                flags = nt | (unroll << 1)
                def f2():
                    rc = lib.apex_hbm_probe_gather(buf.data_ptr(), ids.data_ptr(), n_chunks, blocks,
                                                   flags, sink.data_ptr(), stream)
                    assert rc == 0
                res["gather4k"][f"nt{nt}_u{unroll}_wg{blocks}"] = round(
                    nbytes / _time(torch, f2, reps) / 1e9, 1)
        for unroll in (1, 2, 4):
            flags = 16 | (unroll << 1)

            def f3():
                rc = lib.apex_hbm_probe_gather(buf.data_ptr(), ids.data_ptr(), n_chunks, blocks,
                                               flags, sink.data_ptr(), stream)
                assert rc == 0
            res["gather4k_dev"][f"u{unroll}_wg{blocks}"] = round(nbytes / _time(torch, f3, reps) / 1e9, 1)
    return res
