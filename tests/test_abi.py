"""C-ABI library checks that need no GPU: symbols, host planner, argument validation.

Validation failures return before any HIP call, so they run on a CPU-only host
with fake (never dereferenced) device addresses.
"""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apex_decode.h")
LIB_HEADERS = [HEADER, os.path.join(ROOT, "include", "apex_kv_append.h")]

A = pytest.importorskip("paper_2506_03296_amd")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(A.LIB_PATH):
        from paper_2506_03296_amd import build
        build.build(quiet=True)
    return A.load_library()


def declared_functions():
    names = set()
    for h in LIB_HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(apex_\w+)\s*\(", text))
    return sorted(names)


def test_header_declares_the_base_entry_point_with_its_argument_order():
    text = open(HEADER).read()
    sig = re.search(r"int apex_decode_attention\((.*?)\);", text, flags=re.S).group(1)
    names = [re.findall(r"(\w+)\s*$", p.strip())[0] for p in sig.split(",")]
    assert names == ["q", "k_cache", "v_cache", "block_table", "context_lens", "out", "B", "Hq",
                     "Hkv", "d", "block_size", "scale", "stream"]


def test_every_declared_symbol_is_exported(lib):
    decl = declared_functions()
    assert set(decl) == set(A.EXPORTED_SYMBOLS)
    for name in decl:
        assert hasattr(lib, name), name


def test_version(lib):
    assert A.version() >= 100


def test_args_struct_matches_header_field_order():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct apex_decode_args \{(.*?)\} apex_decode_args;", text, re.S).group(1)
    fields = []
    for decl in body.split(";"):
        decl = decl.strip()
        if not decl:
            continue
        names = decl.split(None, 1)[1] if not decl.startswith("const") else decl.split(None, 2)[2]
        for n in names.split(","):
            fields.append(re.sub(r"[\s*]|\[.*\]", "", n))
    assert fields == [f[0] for f in A.DecodeArgs._fields_]


# ---------------------------------------------------------------------------
# work partition (host mirror) against a brute-force assignment of units
# ---------------------------------------------------------------------------

SEG_COST = 8   # cost positions per pair of the default grid (plan_policy.h)


def _brute_partition(lens, Hkv, launched, forced, cus=0):
    """Owner of every unit, from an explicit line of positions: each non-empty
    (request, kv-head) pair's SEG_COST cost positions, then its blocks; worker
    w takes positions [w V / W, (w + 1) V / W).  Forced grids: no cost."""
    blocks = [(-(-int(L) // 16)) if L > 0 else 0 for L in lens]
    U = sum(blocks) * Hkv
    pairs = sum(1 for nb in blocks if nb > 0) * Hkv
    if not forced and cus > 0 and pairs <= cus and U <= 1024 * cus:
        launched = min(launched, cus)
    W = min(launched, max(1, U // (1 if forced else 16), pairs))
    K = 0 if forced else SEG_COST
    line = []                      # True = a block, False = a cost position
    for nb in blocks:
        for _ in range(Hkv if nb else 0):
            line += [False] * K + [True] * nb
    V = len(line)
    assert V == U + K * pairs
    starts = [w * V // W for w in range(W + 1)]
    owner = []
    for w in range(W):
        owner += [w] * sum(line[starts[w]:starts[w + 1]])
    assert len(owner) == U
    contrib = np.zeros((len(lens), Hkv), dtype=np.int64)
    per_worker_partials = np.zeros(W, dtype=np.int64)
    u = 0
    for b, nb in enumerate(blocks):
        for g in range(Hkv):
            ws = sorted(set(owner[u:u + nb]))
            contrib[b, g] = len(ws)
            if len(ws) > 1:
                for w in ws:
                    per_worker_partials[w] += 1
            u += nb
    return U, W, contrib, per_worker_partials


def _check_plan(lens, Hkv, launched, forced=False, cus=0):
    p = A.plan_host(lens, Hkv, launched, forced=forced, cus=cus)
    U, W, contrib, pwp = _brute_partition(lens, Hkv, launched, forced, cus)
    assert p["units"] == U
    assert p["active"] == (W if U else 0)
    assert np.array_equal(p["contributors"], contrib)
    assert p["partials"] == int(contrib[contrib > 1].sum())
    assert np.all(pwp <= 2)          # a worker has at most two partial segments
    return p


@pytest.mark.parametrize("seed", range(6))
def test_partition_random_batches(lib, seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 300))
    lens = rng.integers(-3, 5000, size=B)
    lens[rng.random(B) < 0.1] = 0
    Hkv = int(rng.choice([1, 2, 8, 32]))
    _check_plan(lens, Hkv, int(rng.choice([1, 7, 80, 1024])))
    _check_plan(lens, Hkv, int(rng.choice([1, 3, 64, 100000])), forced=True)


def test_partition_one_group_per_cu_rule(lib):
    # at most one pair per CU and at most 1024 units per CU: only `cus` groups
    p = _check_plan([2048] * 32, 8, 512, cus=256)
    assert p["active"] == 256 and p["partials"] == 0          # one pair per group
    p = _check_plan([16384] * 32, 8, 512, cus=256)            # 1024 units per CU: still
    assert p["active"] == 256
    p = _check_plan([16400] * 32, 8, 512, cus=256)            # one block more per pair: off
    assert p["active"] == 512
    p = _check_plan([4096] * 64, 8, 512, cus=256)             # two pairs per CU: off
    assert p["active"] == 512
    p = _check_plan([2048] * 32, 8, 512, forced=True, cus=256)   # forced grids: off
    assert p["active"] == 512
    rng = np.random.default_rng(4)
    for _ in range(20):
        B = int(rng.integers(1, 40))
        _check_plan(rng.integers(0, 9000, size=B), int(rng.choice([1, 2, 8])), 512, cus=256)


def test_partition_past_the_cached_lengths(lib):
    rng = np.random.default_rng(9)
    for B in (2048, 2049, 5000):
        lens = rng.integers(0, 48, size=B)
        _check_plan(lens, 2, 768)
        _check_plan(lens, 2, 3, forced=True)


def test_partition_edge_lengths(lib):
    for L in (0, 1, 15, 16, 17, 31, 32, 33, 16 * 8, 16 * 8 + 1, 32768):
        _check_plan([L], 8, 1024)
        _check_plan([L], 8, 5, forced=True)
    p = _check_plan([], 8, 1024)
    assert p["units"] == 0 and p["active"] == 0
    p = _check_plan([0, 0, -1], 8, 1024)
    assert p["units"] == 0


def test_partition_one_worker_writes_everything_directly(lib):
    p = _check_plan([17, 64, 200, 511, 0], 32, 1, forced=True)
    assert p["partials"] == 0
    assert np.all(p["contributors"][:4] == 1)


def test_partition_one_unit_per_worker_splits_every_multi_block_pair(lib):
    lens = [17, 64, 200, 511]
    p = _check_plan(lens, 4, 10 ** 6, forced=True)
    blocks = [-(-L // 16) for L in lens]
    for b, nb in enumerate(blocks):
        assert np.all(p["contributors"][b] == nb)


def test_partition_named_workloads_partial_traffic_is_small(lib):
    import apex_workloads as W
    for name in ("c2", "c3", "c4", "c5"):
        cfg = W.CONFIGS[name]
        lay, _ = W.config_layout(cfg)
        p = _check_plan(lay.lens, cfg.Hkv, 1024)
        G = cfg.Hq // cfg.Hkv
        partial_bytes = 2 * p["partials"] * G * (128 + 2) * 4
        assert partial_bytes < 0.01 * W.algorithmic_bytes(lay.lens, cfg.B, cfg.Hq, cfg.Hkv, 128)


# ---------------------------------------------------------------------------
# argument validation (returns before any HIP call)
# ---------------------------------------------------------------------------

FAKE = 1 << 40   # 16-byte aligned, never dereferenced


def call(lib, B=2, Hq=32, Hkv=8, d=128, bs=16, q=FAKE, k=FAKE + (1 << 30), v=FAKE + (2 << 30),
         bt=FAKE + (3 << 30), lens=FAKE + (4 << 30), out=FAKE + (5 << 30)):
    return lib.apex_decode_attention(q, k, v, bt, lens, out, B, Hq, Hkv, d, bs, 0.1, None)


@pytest.mark.parametrize("kw,code", [
    (dict(Hq=30, Hkv=8), A.APEX_ERR_INVALID_ARG),
    (dict(B=-1), A.APEX_ERR_INVALID_ARG),
    (dict(Hkv=0), A.APEX_ERR_INVALID_ARG),
    (dict(d=64), A.APEX_ERR_UNSUPPORTED),
    (dict(bs=32), A.APEX_ERR_UNSUPPORTED),
    (dict(Hq=6, Hkv=2), A.APEX_ERR_UNSUPPORTED),
    (dict(Hq=32, Hkv=2), A.APEX_ERR_UNSUPPORTED),
    (dict(q=0), A.APEX_ERR_INVALID_ARG),
    (dict(out=0), A.APEX_ERR_INVALID_ARG),
    (dict(lens=0), A.APEX_ERR_INVALID_ARG),
    (dict(q=FAKE + 2), A.APEX_ERR_INVALID_ARG),
    (dict(k=FAKE + (1 << 30) + 8), A.APEX_ERR_INVALID_ARG),
    (dict(bt=FAKE + (3 << 30) + 2), A.APEX_ERR_INVALID_ARG),
    (dict(out=FAKE + 64), A.APEX_ERR_INVALID_ARG),     # overlaps q
    (dict(out=FAKE + (1 << 30)), A.APEX_ERR_INVALID_ARG),             # out = k_cache
    (dict(out=FAKE + (2 << 30) + 4096), A.APEX_ERR_INVALID_ARG),      # inside v_cache's first block
    (dict(out=FAKE + (1 << 30) - 4096), A.APEX_ERR_INVALID_ARG),      # runs into k_cache
    (dict(out=FAKE + (3 << 30)), A.APEX_ERR_INVALID_ARG),             # out = block_table
    (dict(out=FAKE + (4 << 30)), A.APEX_ERR_INVALID_ARG),             # out = context_lens
])
def test_invalid_arguments_are_rejected(lib, kw, code):
    assert call(lib, **kw) == code
    assert A.last_error() != ""


def test_empty_batch_is_a_noop(lib):
    assert call(lib, B=0, q=0, out=0) == A.APEX_OK
    assert A.last_error() == ""


def test_ex_rejects_flags_and_negative_fields(lib):
    for field, value in (("flags", 2), ("flags", 1), ("num_workers", -1), ("num_workers", 1 << 21),
                         ("block_table_stride", -5)):
        a = A.DecodeArgs()
        a.q, a.k_cache, a.v_cache = FAKE, FAKE + (1 << 30), FAKE + (2 << 30)
        a.block_table, a.context_lens, a.out = FAKE + (3 << 30), FAKE + (4 << 30), FAKE + (5 << 30)
        a.B, a.Hq, a.Hkv, a.d, a.block_size, a.scale = 2, 32, 8, 128, 16, 0.1
        setattr(a, field, value)
        assert lib.apex_decode_attention_ex(ctypes.byref(a)) == A.APEX_ERR_INVALID_ARG
    assert lib.apex_decode_attention_ex(None) == A.APEX_ERR_INVALID_ARG


@pytest.mark.parametrize("field,where,needle", [
    ("num_blocks", 1 << 20, "k_cache"),          # 1 MiB into a cache of 100 blocks (3.2 MB)
    ("num_blocks", (1 << 30) + (3 << 20), "v_cache"),
    ("block_table_stride", (2 << 30) + 640, "block_table"),   # row 1 of a 100-entry stride
])
def test_ex_out_overlap_over_the_known_extents(lib, field, where, needle):
    """With num_blocks (or an explicit table stride) the whole caches (the
    whole table) are checked against out, not just their start."""
    a = _fake_args()
    setattr(a, field, 100)
    a.out = a.k_cache + where
    assert lib.apex_decode_attention_ex(ctypes.byref(a)) == A.APEX_ERR_INVALID_ARG
    assert needle in A.last_error()


def test_ex_rejects_a_negative_block_count(lib):
    a = _fake_args()
    a.num_blocks = -1
    assert lib.apex_decode_attention_ex(ctypes.byref(a)) == A.APEX_ERR_INVALID_ARG
    assert "num_blocks" in A.last_error()


def test_ex_check_flag_needs_the_block_count(lib):
    a = A.DecodeArgs()
    a.q, a.k_cache, a.v_cache = FAKE, FAKE + (1 << 30), FAKE + (2 << 30)
    a.block_table, a.context_lens, a.out = FAKE + (3 << 30), FAKE + (4 << 30), FAKE + (5 << 30)
    a.B, a.Hq, a.Hkv, a.d, a.block_size, a.scale = 2, 32, 8, 128, 16, 0.1
    a.flags = A.FLAG_CHECK_INPUTS
    a.num_blocks = 0
    assert lib.apex_decode_attention_ex(ctypes.byref(a)) == A.APEX_ERR_INVALID_ARG
    assert "num_blocks" in A.last_error()


def _fake_args():
    a = A.DecodeArgs()
    a.q, a.k_cache, a.v_cache = FAKE, FAKE + (1 << 30), FAKE + (2 << 30)
    a.block_table, a.context_lens, a.out = FAKE + (3 << 30), FAKE + (4 << 30), FAKE + (5 << 30)
    a.B, a.Hq, a.Hkv, a.d, a.block_size, a.scale = 2, 32, 8, 128, 16, 0.1
    return a


@pytest.mark.parametrize("case", ["k_only", "v_only", "stride_alone", "stride_short", "stride_odd",
                                  "misaligned", "out_overlaps_k_new"])
def test_ex_fused_append_arguments(lib, case):
    a = _fake_args()
    if case == "k_only":
        a.k_new = FAKE + (6 << 30)
    elif case == "v_only":
        a.v_new = FAKE + (6 << 30)
    elif case == "stride_alone":
        a.new_token_stride = 8 * 128
    else:
        a.k_new, a.v_new = FAKE + (6 << 30), FAKE + (7 << 30)
        if case == "stride_short":
            a.new_token_stride = 8 * 128 - 8
        elif case == "stride_odd":
            a.new_token_stride = 8 * 128 + 4
        elif case == "misaligned":
            a.k_new += 2
        else:
            a.k_new = a.out + 64
    assert lib.apex_decode_attention_ex(ctypes.byref(a)) == A.APEX_ERR_INVALID_ARG
    assert A.last_error() != ""


def test_plan_host_rejects_bad_arguments(lib):
    with pytest.raises(A.ApexError):
        A.plan_host([5], 0, 256)
    with pytest.raises(A.ApexError):
        A.plan_host([5], 8, 0)
    with pytest.raises(A.ApexError):
        A.plan_host([5], 8, 256, block_size=32)
    with pytest.raises(A.ApexError):
        A.plan_host([5], 8, 256, cus=-1)


def test_counter_bytes(lib):
    assert A.counter_bytes(512, 8) == 512 * 8 * 4
    assert A.counter_bytes(3, 1) == 256


# ---------------------------------------------------------------------------
# KV append: argument validation (returns before any HIP call)
# ---------------------------------------------------------------------------

def append_call(lib, T=4, Hkv=8, d=128, bs=16, nb=100, stride=0, kn=FAKE, vn=FAKE + (1 << 30),
                kc=FAKE + (2 << 30), vc=FAKE + (3 << 30), slots=FAKE + (4 << 30)):
    return lib.apex_kv_append(kn, vn, stride, kc, vc, slots, T, Hkv, d, bs, nb, None)


def test_kv_append_header_argument_order():
    text = open(LIB_HEADERS[1]).read()
    sig = re.search(r"int apex_kv_append\((.*?)\);", text, flags=re.S).group(1)
    names = [re.findall(r"(\w+)\s*$", p.strip())[0] for p in sig.split(",")]
    assert names == ["k_new", "v_new", "new_token_stride", "k_cache", "v_cache", "slot_mapping",
                     "T", "Hkv", "d", "block_size", "num_blocks", "stream"]


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), A.APEX_ERR_INVALID_ARG),
    (dict(Hkv=0), A.APEX_ERR_INVALID_ARG),
    (dict(bs=0), A.APEX_ERR_INVALID_ARG),
    (dict(nb=-1), A.APEX_ERR_INVALID_ARG),
    (dict(d=12), A.APEX_ERR_UNSUPPORTED),
    (dict(d=4096), A.APEX_ERR_UNSUPPORTED),
    (dict(stride=8 * 128 - 8), A.APEX_ERR_INVALID_ARG),
    (dict(stride=8 * 128 + 4), A.APEX_ERR_INVALID_ARG),
    (dict(T=1 << 28, Hkv=16), A.APEX_ERR_UNSUPPORTED),
    (dict(nb=1 << 50), A.APEX_ERR_INVALID_ARG),
    (dict(kn=0), A.APEX_ERR_INVALID_ARG),
    (dict(slots=0), A.APEX_ERR_INVALID_ARG),
    (dict(kn=FAKE + 8), A.APEX_ERR_INVALID_ARG),
    (dict(vc=FAKE + (3 << 30) + 2), A.APEX_ERR_INVALID_ARG),
    (dict(slots=FAKE + (4 << 30) + 4), A.APEX_ERR_INVALID_ARG),
    (dict(vc=FAKE + (2 << 30) + 4096), A.APEX_ERR_INVALID_ARG),     # caches overlap
    (dict(kn=FAKE + (2 << 30) + 256), A.APEX_ERR_INVALID_ARG),      # input inside a cache
    (dict(slots=FAKE + (3 << 30)), A.APEX_ERR_INVALID_ARG),         # slots inside a cache
])
def test_kv_append_invalid_arguments_are_rejected(lib, kw, code):
    assert append_call(lib, **kw) == code
    assert A.last_error() != ""


def test_kv_append_empty_or_poolless_calls_are_noops(lib):
    assert append_call(lib, T=0, kn=0, vn=0, kc=0, vc=0, slots=0) == A.APEX_OK
    assert A.last_error() == ""
    assert append_call(lib, nb=0) == A.APEX_OK


def test_kv_append_overlapping_fused_inputs_are_allowed(lib):
    # K and V views into one fused [T][Hq + 2 Hkv][d] buffer interleave
    d, Hq, Hkv = 128, 32, 8
    stride = (Hq + 2 * Hkv) * d
    base = FAKE
    kn, vn = base + Hq * d * 2, base + (Hq + Hkv) * d * 2
    assert append_call(lib, T=4, nb=0, stride=stride, kn=kn, vn=vn) == A.APEX_OK


# ---------------------------------------------------------------------------
# Python binding: tensors the library would misread are refused before the
# call (no GPU needed: host tensors and the checking helper itself)
# ---------------------------------------------------------------------------

def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    q = torch.zeros((2, 8, 128), dtype=torch.float16)
    kc = torch.zeros((4, 2, 16, 128), dtype=torch.float16)
    bt = torch.zeros((2, 2), dtype=torch.int32)
    lens = torch.tensor([5, 20], dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        A.decode_attention(q, kc, kc.clone(), bt, lens, 0.1)
    with pytest.raises(ValueError, match="GPU tensor"):
        A.decode_attention_ex(q, kc, kc.clone(), bt, lens, 0.1)
    kn = torch.zeros((2, 2, 128), dtype=torch.float16)
    with pytest.raises(ValueError, match="GPU tensors"):
        A.kv_append(kn, kn.clone(), kc, kc.clone(), torch.tensor([0, 1]))


@pytest.mark.parametrize("case", ["dtype", "device", "shape", "gaps"])
def test_binding_tensor_check(case):
    torch = pytest.importorskip("torch")
    cpu = torch.device("cpu")
    t = torch.zeros((4, 6), dtype=torch.float16)
    if case == "dtype":
        with pytest.raises(TypeError, match="must be torch.float16"):
            A._require(t.float(), "x", torch.float16, cpu)
    elif case == "device":
        with pytest.raises(ValueError, match="must be on cuda:0"):
            A._require(t, "x", torch.float16, torch.device("cuda", 0))
    elif case == "shape":
        with pytest.raises(ValueError, match=r"shape \(4, 5\)"):
            A._require(t, "x", torch.float16, cpu, shape=(4, 5))
    else:
        with pytest.raises(ValueError, match="contiguous"):
            A._require(t[:, ::2], "x", torch.float16, cpu)
        A._require(t[:, ::2], "x", torch.float16, cpu, contiguous=False)
    A._require(t, "x", torch.float16, cpu, shape=(4, 6))


def test_partition_huge_unit_counts_divide_exactly(lib):
    """Unit counts past 2^32 (the 32-bit division path no longer applies):
    contributors per pair against exact integer arithmetic."""
    lens = [2 ** 31 - 1, 5, 2 ** 30, 70000]
    Hkv = 32
    for launched in (1024, 7, 100000):
        p = A.plan_host(lens, Hkv, launched)
        blocks = [-(-L // 16) for L in lens]
        U = sum(blocks) * Hkv
        pairs = sum(1 for nb in blocks if nb > 0) * Hkv
        W = min(launched, max(1, U // 16, pairs))
        assert U > 2 ** 32 and p["units"] == U and p["active"] == W

        def worker_of(u):
            return ((u + 1) * W - 1) // U

        pre = 0
        for b, nb in enumerate(blocks):
            for g in range(Hkv):
                p0 = (pre * Hkv) + g * nb
                want = worker_of(p0 + nb - 1) - worker_of(p0) + 1
                assert p["contributors"][b, g] == want, (launched, b, g)
            pre += nb


# ---------------------------------------------------------------------------
# apex_decode_attention_noalloc: the same validation, plus the static
# scratch's pair limit (host checks, before any HIP call)
# ---------------------------------------------------------------------------

def noalloc_call(lib, B=2, Hq=32, Hkv=8, q=FAKE, out=FAKE + (5 << 30)):
    return lib.apex_decode_attention_noalloc(q, FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30),
                                             FAKE + (4 << 30), out, B, Hq, Hkv, 128, 16, 0.1, None)


def test_noalloc_refuses_more_pairs_than_its_scratch(lib):
    assert noalloc_call(lib, B=8193, Hq=8, Hkv=8) == A.APEX_ERR_UNSUPPORTED
    assert "65536" in A.last_error()
    assert noalloc_call(lib, B=2049, Hq=32, Hkv=32) == A.APEX_ERR_UNSUPPORTED


def test_noalloc_validates_like_the_base_call(lib):
    assert noalloc_call(lib, Hq=30) == A.APEX_ERR_INVALID_ARG
    assert noalloc_call(lib, q=0) == A.APEX_ERR_INVALID_ARG
    assert noalloc_call(lib, out=FAKE + 64) == A.APEX_ERR_INVALID_ARG
    assert noalloc_call(lib, B=0, q=0, out=0) == A.APEX_OK
    assert A.last_error() == ""


# ---------------------------------------------------------------------------
# the work-group trace build (libapex_decode_trace.so): the product library's
# symbols plus apex_decode_trace_buffer, which the product does not export
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def trace_lib(lib):
    from paper_2506_03296_amd import wg_trace
    return wg_trace.load_trace_library()


def test_trace_build_exports_the_trace_entry_point_and_the_product_does_not(lib, trace_lib):
    for name in declared_functions():
        assert hasattr(trace_lib, name), name
    assert hasattr(trace_lib, "apex_decode_trace_buffer")
    with pytest.raises(AttributeError):
        lib.apex_decode_trace_buffer


def test_trace_buffer_arguments(trace_lib):
    assert trace_lib.apex_decode_trace_buffer(FAKE + 4, 16) == A.APEX_ERR_INVALID_ARG
    assert trace_lib.apex_decode_trace_buffer(FAKE, -1) == A.APEX_ERR_INVALID_ARG
    assert trace_lib.apex_decode_trace_buffer(FAKE, 16) == A.APEX_OK
    assert trace_lib.apex_decode_trace_buffer(None, 0) == A.APEX_OK


def test_trace_summary_of_a_synthetic_timeline():
    from paper_2506_03296_amd import wg_trace
    rows = np.zeros((8, 8), dtype=np.int64)
    for w in range(8):
        s = 1000 + 10 * (w % 4) + 100 * (w >= 4)      # second round starts 1 us later
        rows[w] = [s, s + 200, s + 500, s + 10000 + 100 * w, 1 + w % 2, w % 2, 40, 0]
    r = wg_trace.summarize(rows, cus=4)
    assert r["work_groups"] == 8 and r["active"] == 8
    assert abs(r["prologue"]["p50"] - 2.0) < 1e-9 and abs(r["first_load"]["p50"] - 3.0) < 1e-9
    assert abs(r["span"] - (1130 + 10000 + 700 - 1000) * 0.01) < 1e-9     # group 7 ends last
    assert abs(r["dispatch"]["round2_start_min"] - 1.0) < 1e-9
    assert r["split_segments"] == 4
    assert set(r["by_segments"]) == {1, 2}
