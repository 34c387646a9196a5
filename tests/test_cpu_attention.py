"""Host (CPU) paged decode-attention backend against the fp64 oracle.

The backend (libapex_cpu.so) computes the same attention as the GPU library
on the host cores; it runs here, without a GPU.  Bar: the GPU's (every output
finite, max-abs <= 2e-3, relative L2 <= 1e-3 against the unrounded fp64
oracle), on both SIMD paths (AVX-512 and AVX2), with NaN poison in every slot
the attention must not read, forced token chunking, wide table strides,
empty requests and the natural-log LSE.  Closed forms and invariants are
checked exactly where they hold exactly.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import apex_workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apex_cpu_attention.h")

C = pytest.importorskip("paper_2506_03296_amd.cpu")

MAX_ABS = 2e-3
REL_L2 = 1e-3


@pytest.fixture(scope="module")
def cpu():
    if not os.path.exists(C.LIB_PATH):
        from paper_2506_03296_amd import build
        build.build_cpu(quiet=True)
    C.load_library()
    if C.isa() == 0:
        pytest.skip("CPU lacks AVX2 + FMA + F16C")
    return C


PATHS = [False, True]   # AVX2 forced or not


def run(cpu, case, **kw):
    return cpu.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                case.context_lens, case.scale, **kw)


def assert_parity(got, ref, what=""):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite outputs"
    err = np.abs(got - ref)
    max_abs = float(err.max()) if err.size else 0.0
    nrm = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(got - ref)) / nrm if nrm > 0 else float(np.linalg.norm(got))
    assert max_abs <= MAX_ABS, f"{what}: max-abs {max_abs:.3e}"
    assert rel <= REL_L2, f"{what}: rel-L2 {rel:.3e}"


SHAPES = [
    # lens, Hq, Hkv, d, block_size
    ([17, 64, 200, 511, 1, 3000, 0], 32, 8, 128, 16),
    ([17, 64, 200, 511], 32, 32, 128, 16),
    ([1, 2, 15, 16, 17, 33], 8, 2, 128, 16),
    ([100, 7, 0, 65], 6, 2, 64, 16),       # G = 3
    ([300, 129], 16, 1, 128, 16),          # G = 16
    ([90, 45], 64, 2, 32, 16),             # G = 32, d = 32
    ([77, 5], 4, 4, 16, 7),                # block size 7, d = 16
    ([257, 31], 8, 4, 256, 32),            # d = 256, block size 32
    ([40, 3], 4, 2, 48, 1),                # block size 1, d / 16 odd
]


@pytest.mark.parametrize("force_avx2", PATHS)
@pytest.mark.parametrize("lens,Hq,Hkv,d,bs", SHAPES)
def test_parity_with_poison(cpu, oracle_mod, lens, Hq, Hkv, d, bs, force_avx2):
    case = W.make_host_case(lens, Hq, Hkv, d=d, block_size=bs, seed=sum(lens) + d, poison=True)
    out, lse = run(cpu, case, return_lse=True, force_avx2=force_avx2)
    ref, rlse = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                                case.context_lens, case.scale, return_lse=True)
    assert_parity(out, ref, f"{lens} {Hq}/{Hkv} d={d} bs={bs}")
    fin = np.isfinite(rlse)
    assert np.array_equal(np.isfinite(lse), fin)
    np.testing.assert_allclose(lse[fin], rlse[fin], rtol=0, atol=1e-4)


@pytest.mark.parametrize("force_avx2", PATHS)
@pytest.mark.parametrize("threads,min_chunk", [(1, 0), (8, 16), (3, 32), (8, 1)])
def test_forced_chunking_matches(cpu, oracle_mod, threads, min_chunk, force_avx2):
    """Few pairs, so long requests are cut into block-aligned chunks that are
    merged with the log-sum-exp identity (min_chunk 1 still rounds up to a
    block)."""
    case = W.make_host_case([5000, 33, 1, 700], 8, 2, seed=41, poison=True)
    out = run(cpu, case, num_threads=threads, min_chunk_tokens=min_chunk, force_avx2=force_avx2)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    assert_parity(out, ref, f"threads={threads} chunk={min_chunk}")


def test_wide_block_table_stride(cpu, oracle_mod):
    case = W.make_host_case([40, 300, 17], 8, 2, seed=5, poison=True, stride=64)
    out = run(cpu, case)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    assert_parity(out, ref, "stride 64")


def test_single_token_returns_v_bitwise(cpu):
    case = W.make_host_case([1, 1, 1], 32, 8, seed=9, poison=True)
    out = run(cpu, case)
    for b in range(3):
        blk = case.block_table[b, 0]
        for h in range(32):
            assert np.array_equal(out[b, h].view(np.uint16), case.v_cache[blk, h // 4, 0].view(np.uint16))


def test_identical_keys_give_mean_of_v(cpu):
    case = W.make_host_case([7, 50, 129], 8, 2, seed=6)
    key = np.random.default_rng(0).standard_normal((2, 128)).astype(np.float16)
    for b, L in enumerate(case.context_lens):
        for t in range(int(L)):
            case.k_cache[case.block_table[b, t // 16], :, t % 16, :] = key
    out = run(cpu, case).astype(np.float64)
    from oracle import brute_force
    for b, L in enumerate(case.context_lens):
        V = brute_force.dense_kv(case.v_cache, case.block_table, b, int(L))
        for h in range(8):
            np.testing.assert_allclose(out[b, h], V[h // 4].mean(axis=0), rtol=0, atol=1e-3)


def test_unit_values_give_unit_output(cpu):
    case = W.make_host_case([3, 70, 1000], 32, 8, seed=8)
    case.v_cache[:] = np.float16(1.0)
    out = run(cpu, case)
    assert np.all(out == np.float16(1.0))


def test_empty_requests_and_empty_batch(cpu):
    case = W.make_host_case([0, 5, -3, 0], 8, 2, seed=10, poison=True)
    out, lse = run(cpu, case, return_lse=True)
    for b in (0, 2, 3):
        assert np.all(out[b] == 0)
        assert np.all(np.isneginf(lse[b]))
    assert np.all(np.isfinite(out[1]))
    q = np.zeros((0, 8, 128), np.float16)
    kc = np.zeros((1, 2, 16, 128), np.float16)
    r = cpu.decode_attention(q, kc, kc, np.zeros((0, 1), np.int32), np.zeros(0, np.int32), 0.1)
    assert r.shape == (0, 8, 128)


def test_block_permutation_and_thread_count_are_bitwise_invariant(cpu):
    lens = [150, 64, 1]
    a = W.make_host_case(lens, 32, 8, seed=12)
    ref = run(cpu, a, min_chunk_tokens=1 << 20)
    # move every block to another physical id
    rng = np.random.default_rng(1)
    nb = a.k_cache.shape[0]
    perm = rng.permutation(nb)
    k2 = np.empty_like(a.k_cache)
    v2 = np.empty_like(a.v_cache)
    k2[perm] = a.k_cache
    v2[perm] = a.v_cache
    bt2 = perm[a.block_table].astype(np.int32)
    out = cpu.decode_attention(a.q, k2, v2, bt2, a.context_lens, a.scale, min_chunk_tokens=1 << 20)
    assert np.array_equal(out.view(np.uint16), ref.view(np.uint16))
    for n in (1, 2, 5):
        o = run(cpu, a, num_threads=n, min_chunk_tokens=1 << 20)
        assert np.array_equal(o.view(np.uint16), ref.view(np.uint16))


def test_gqa_matches_mha_with_repeated_kv(cpu):
    G = 4
    case = W.make_host_case([33, 200], 16, 4, seed=13)
    out = run(cpu, case)
    rep = W.HostCase(case.q, np.repeat(case.k_cache, G, axis=1), np.repeat(case.v_cache, G, axis=1),
                     case.block_table, case.context_lens, case.scale)
    out2 = run(cpu, rep)
    np.testing.assert_allclose(out.astype(np.float64), out2.astype(np.float64), rtol=0, atol=2e-3)


def test_late_peaked_key_dominates(cpu, oracle_mod):
    case = W.make_host_case([3000], 8, 2, seed=14)
    blk = case.block_table[0, 2999 // 16]
    case.k_cache[blk, :, 2999 % 16, :] = (case.q[0, ::4] * 4).astype(np.float16)
    out = run(cpu, case)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    assert_parity(out, ref, "peaked")


def test_larger_batch_matches(cpu, oracle_mod):
    """A Llama-3.1-8B-shaped batch of 24 requests, lengths 1024-4096."""
    rng = np.random.default_rng(15)
    lens = rng.integers(1024, 4096, size=24, endpoint=True)
    case = W.make_host_case(lens, 32, 8, seed=15, poison=True)
    out = run(cpu, case)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    assert_parity(out, ref, "24 requests")


# ---------------------------------------------------------------------------
# ABI
# ---------------------------------------------------------------------------

def test_header_symbols_are_exported(cpu):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    declared = set(re.findall(r"\b(apex_cpu_\w+)\s*\(", text))
    assert declared == set(C.EXPORTED_SYMBOLS)
    lib = C.load_library()
    for name in declared:
        assert hasattr(lib, name)


def test_args_struct_matches_header(cpu):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct apex_cpu_args \{(.*?)\} apex_cpu_args;", text, re.S).group(1)
    fields = []
    for decl in body.split(";"):
        decl = decl.strip()
        if not decl:
            continue
        names = decl.split(None, 1)[1] if not decl.startswith("const") else decl.split(None, 2)[2]
        for n in names.split(","):
            fields.append(re.sub(r"[\s*]", "", n))
    assert fields == [f[0] for f in C.CpuArgs._fields_]


@pytest.mark.parametrize("field,value,code", [
    ("B", -1, -1), ("Hkv", 0, -1), ("Hq", 30, -1), ("d", 24, -2), ("d", 1024, -2),
    ("block_size", 0, -1), ("flags", 2, -1), ("num_threads", -1, -1),
    ("block_table_stride", -1, -1), ("Hq", 8 * 65, -2),
])
def test_invalid_arguments(cpu, field, value, code):
    case = W.make_host_case([20, 40], 8, 8, seed=1)
    a = C.CpuArgs()
    out = np.empty_like(case.q)
    a.q, a.k_cache, a.v_cache = case.q.ctypes.data, case.k_cache.ctypes.data, case.v_cache.ctypes.data
    a.block_table, a.context_lens = case.block_table.ctypes.data, case.context_lens.ctypes.data
    a.out = out.ctypes.data
    a.B, a.Hq, a.Hkv, a.d, a.block_size, a.scale = 2, 8, 8, 128, 16, 0.1
    setattr(a, field, value)
    assert C.load_library().apex_cpu_decode_attention_ex(ctypes.byref(a)) == code
    assert C.last_error() != ""


def test_table_too_narrow_and_aliasing_are_rejected(cpu):
    case = W.make_host_case([20, 40], 8, 8, seed=1)
    with pytest.raises(C.CpuError):
        cpu.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                             case.context_lens, case.scale, block_table_stride=1)
    with pytest.raises(C.CpuError):
        cpu.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                             case.context_lens, case.scale, out=case.q)


def test_threads_and_bandwidth_probe(cpu):
    n = cpu.threads()
    assert n >= 1
    cpu.set_threads(2)
    assert cpu.threads() == 2
    assert cpu.read_bandwidth(1 << 24, reps=2) > 0
    cpu.set_threads(0)
    assert cpu.threads() == n
