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

A = pytest.importorskip("paper_2506_03296_amd")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(A.LIB_PATH):
        from paper_2506_03296_amd import build
        build.build(quiet=True)
    return A.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apex_\w+)\s*\(", text)))


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
# split-K planner policy (host mirror)
# ---------------------------------------------------------------------------

def _check_plan(lens, Hkv, num_cu, num_splits=0, items_per_cu=0):
    p = A.plan_host(lens, Hkv, num_cu, num_splits=num_splits, items_per_cu=items_per_cu)
    lens = np.asarray(lens, dtype=np.int64)
    blocks = np.where(lens > 0, -(-lens // 16), 0)
    n, per, chunk = p["splits"], p["blocks_per_split"], p["chunk"]
    assert chunk >= 8
    target = num_cu * (items_per_cu or 16)
    assert chunk >= -(-int(blocks.sum() * Hkv) // target)
    for b in range(len(lens)):
        if blocks[b] == 0:
            assert n[b] == 1 and per[b] == 0
            continue
        assert n[b] * per[b] >= blocks[b]           # every block covered
        assert (-(-blocks[b] // per[b])) <= n[b]
        if num_splits:
            assert n[b] == num_splits
        else:
            assert per[b] <= chunk
            assert (n[b] == 1) == (blocks[b] <= chunk)
            assert (n[b] - 1) * per[b] < blocks[b]   # no empty range
    assert p["items"] == int(n.sum()) * Hkv
    assert p["partial_slots"] == int(n[n > 1].sum()) * Hkv
    if not num_splits:
        assert p["items"] <= target + len(lens) * Hkv
    return p


@pytest.mark.parametrize("seed", range(6))
def test_plan_random_batches(lib, seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 700))
    lens = rng.integers(-3, 40000, size=B)
    lens[rng.random(B) < 0.1] = 0
    _check_plan(lens, int(rng.choice([1, 2, 8, 32])), int(rng.choice([1, 80, 256])))


def test_plan_edge_lengths(lib):
    for L in (0, 1, 15, 16, 17, 31, 32, 33, 16 * 8, 16 * 8 + 1, 32768):
        _check_plan([L], 8, 256)
    p = _check_plan([], 8, 256)
    assert p["items"] == 0


@pytest.mark.parametrize("n", [1, 2, 7, 64])
def test_plan_forced_splits(lib, n):
    p = _check_plan([17, 64, 200, 511, 0], 32, 256, num_splits=n)
    assert list(p["splits"]) == [n, n, n, n, 1]


def test_plan_short_requests_stay_whole_long_ones_split(lib):
    lens = [300] * 256 + [16000] * 256
    p = _check_plan(lens, 8, 256)
    assert np.all(p["splits"][:256] == 1) and np.all(p["splits"][256:] > 1)


def test_plan_named_workload_partial_traffic_is_small(lib):
    import apex_workloads as W
    for name in ("c2", "c3", "c4", "c5"):
        cfg = W.CONFIGS[name]
        lay, _ = W.config_layout(cfg)
        p = _check_plan(lay.lens, cfg.Hkv, 256)
        G = cfg.Hq // cfg.Hkv
        partial_bytes = 2 * p["partial_slots"] * G * (128 + 2) * 4
        assert partial_bytes < 0.03 * W.algorithmic_bytes(lay.lens, cfg.B, cfg.Hq, cfg.Hkv, 128)


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
])
def test_invalid_arguments_are_rejected(lib, kw, code):
    assert call(lib, **kw) == code
    assert A.last_error() != ""


def test_empty_batch_is_a_noop(lib):
    assert call(lib, B=0, q=0, out=0) == A.APEX_OK
    assert A.last_error() == ""


def test_ex_rejects_flags_and_negative_fields(lib):
    for field, value in (("flags", 1), ("num_splits", -1), ("items_per_cu", -2),
                         ("block_table_stride", -5)):
        a = A.DecodeArgs()
        a.q, a.k_cache, a.v_cache = FAKE, FAKE + (1 << 30), FAKE + (2 << 30)
        a.block_table, a.context_lens, a.out = FAKE + (3 << 30), FAKE + (4 << 30), FAKE + (5 << 30)
        a.B, a.Hq, a.Hkv, a.d, a.block_size, a.scale = 2, 32, 8, 128, 16, 0.1
        setattr(a, field, value)
        assert lib.apex_decode_attention_ex(ctypes.byref(a)) == A.APEX_ERR_INVALID_ARG
    assert lib.apex_decode_attention_ex(None) == A.APEX_ERR_INVALID_ARG


def test_plan_host_rejects_bad_arguments(lib):
    with pytest.raises(A.ApexError):
        A.plan_host([5], 0, 256)
    with pytest.raises(A.ApexError):
        A.plan_host([5], 8, 0)
    with pytest.raises(A.ApexError):
        A.plan_host([5], 8, 256, block_size=32)
