"""ABI checks of the overlap runtime library that need no GPU: exported
symbols, the config struct mirror, and configuration errors (returned before
any HIP call)."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apex_overlap.h")

ov = pytest.importorskip("paper_2506_03296_amd.overlap")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ov.LIB_PATH):
        from paper_2506_03296_amd import build
        build.build(quiet=True)
    return ov.load_library()


def test_header_symbols_are_exported(lib):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    declared = set(re.findall(r"\b(apex_overlap_\w+)\s*\(", text))
    assert declared == set(ov.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(lib, name)


def test_config_struct_matches_header(lib):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct apex_overlap_config \{(.*?)\} apex_overlap_config;", text, re.S).group(1)
    fields = []
    for decl in body.split(";"):
        decl = decl.strip()
        if decl:
            for n in decl.split(None, 1)[1].split(","):
                fields.append(n.strip())
    assert fields == [f[0] for f in ov.Config._fields_]


BASE = dict(layers=2, max_requests=4, Hq=32, Hkv=8, d=128, block_size=16, scale=0.1,
            num_blocks=16, max_blocks_per_request=8)


@pytest.mark.parametrize("field,value,code", [
    ("layers", 0, -1), ("layers", 1 << 16, -1), ("max_requests", 0, -1), ("Hq", 30, -1),
    ("Hkv", 0, -1), ("d", 24, -2), ("block_size", 0, -1), ("num_blocks", 0, -1),
    ("max_blocks_per_request", 0, -1), ("threads", -1, -1), ("slots_per_layer", -2, -1),
])
def test_bad_config_is_rejected_before_any_hip_call(lib, field, value, code):
    kw = dict(BASE, **{field: value})
    with pytest.raises(ov.OverlapError) as e:
        ov.Overlap(**kw)
    assert e.value.code == code
    assert ov.last_error() != ""


def test_group_size_beyond_the_host_backend_is_rejected(lib):
    with pytest.raises(ov.OverlapError) as e:
        ov.Overlap(**dict(BASE, Hq=128, Hkv=1))
    assert e.value.code == -2


def test_null_runtime_calls(lib):
    import ctypes
    assert lib.apex_overlap_destroy(None) == 0
    assert lib.apex_overlap_pending(None) == 0
    assert lib.apex_overlap_hold(None, 1) == -1
    r = ctypes.c_int()
    assert lib.apex_overlap_poll(None, 0, None, None, ctypes.byref(r)) == -1
