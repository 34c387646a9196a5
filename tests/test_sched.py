"""The library's strategy selection (libapex_cpu.so, include/apex_sched.h)
against the scheduler oracle (oracle/scheduler.py), CPU only.

Both sides compute in IEEE double.  Throughputs and times must agree to a
few ulps; the strategy must be identical wherever the two throughputs differ
by more than 1e-12 relative (at an exact tie either side may round its way;
the oracle's pins check the tie itself in exact arithmetic).
"""
import os
import random
import re

import numpy as np
import pytest

from oracle import scheduler as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apex_sched.h")

sched = pytest.importorskip("paper_2506_03296_amd.sched")


@pytest.fixture(scope="module")
def lib():
    from paper_2506_03296_amd import cpu
    if not os.path.exists(cpu.LIB_PATH):
        from paper_2506_03296_amd import build
        build.build_cpu(quiet=True)
    return sched._lib()


def lograndom(rng, lo=1e-6, hi=1e6):
    return 10 ** rng.uniform(np.log10(lo), np.log10(hi))


def close(a, b, rel=1e-13):
    return abs(a - b) <= rel * max(abs(a), abs(b), 1e-300)


def _case(rng, prefill, form):
    kw = dict(n_g=lograndom(rng), n_c=lograndom(rng) if rng.random() > 0.05 else 0.0,
              t_glinear=lograndom(rng), t_gatt=lograndom(rng))
    if prefill:
        kw.update(prefill=True, t_glinear_pref=lograndom(rng), t_gatt_pref=lograndom(rng) if rng.random() > 0.1 else 0.0,
                  mixed_form=form)
    return kw


@pytest.mark.parametrize("prefill,form", [(False, "paper"), (True, "paper"), (True, "eq5")])
def test_select_matches_oracle(lib, prefill, form):
    rng = random.Random(hash((prefill, form)) & 0xffff)
    decided = {O.ASYM_PIPELINE: 0, O.ASYNC_OVERLAP: 0}
    for _ in range(20000):
        kw = _case(rng, prefill, form)
        st, pipe, gpu = O.strategy_selection(**kw)
        r = sched.select(**kw)
        assert close(r["throughput_pipe"], pipe) and close(r["throughput_gpu"], gpu), kw
        if abs(pipe - gpu) > 1e-12 * max(pipe, gpu):
            assert r["strategy"] == st, kw
            decided[st] += 1
        if not prefill:
            assert close(r["ratio_bound"], O.ratio_bound(kw["t_glinear"], kw["t_gatt"]))
            assert close(r["t_overlap"], O.t_overlap_decode(kw["t_glinear"], kw["t_gatt"]))
        else:
            assert close(r["t_overlap"], O.t_overlap_mixed(kw["t_glinear_pref"], kw["t_gatt_pref"],
                                                           kw["t_glinear"], kw["t_gatt"]))
    assert min(decided.values()) > 1000    # both outcomes exercised


def test_decode_decision_follows_eq6(lib):
    rng = random.Random(7)
    for _ in range(20000):
        ng, nc, tl, ta = (lograndom(rng) for _ in range(4))
        bound = O.ratio_bound(tl, ta)
        if abs(ng / nc - bound) < 1e-9 * bound:
            continue
        expect = O.ASYM_PIPELINE if ng / nc < bound else O.ASYNC_OVERLAP
        assert sched.select(ng, nc, tl, ta)["strategy"] == expect


def test_papers_worked_numbers(lib):
    assert sched.ratio_bound(2.0, 1.0) == 7.5
    assert abs(sched.ratio_bound(2.0, 3.0) - 35 / 6) < 1e-15
    # CPU at 13 % of the GPU rate with T_gatt / T_glinear = 0.5: no; at 14 %: yes
    assert sched.select(1.0, 0.13, 2.0, 1.0)["strategy"] == O.ASYNC_OVERLAP
    assert sched.select(1.0, 0.14, 2.0, 1.0)["strategy"] == O.ASYM_PIPELINE


def test_main_scheduler_exits(lib):
    slow_cpu = dict(n_g=100.0, n_c=1.0, t_glinear=1.0, t_gatt=1.0)
    fast_cpu = dict(n_g=10.0, n_c=9.0, t_glinear=1.0, t_gatt=1.0)
    assert sched.main(0, 8, 0, 0)["strategy"] == O.GPU_ONLY
    assert sched.main(3, 8, 0, 0, fast_cpu)["strategy"] == O.GPU_ONLY
    assert sched.main(0, 8, 5, 0, fast_cpu)["strategy"] == O.ASYNC_OVERLAP
    assert sched.main(0, 8, 5, 2, fast_cpu)["strategy"] == O.ASYM_PIPELINE
    assert sched.main(0, 8, 5, 2, slow_cpu)["strategy"] == O.ASYNC_OVERLAP
    mixed = dict(slow_cpu, t_glinear_pref=200.0, t_gatt_pref=0.0)
    assert sched.main(1, 8, 5, 2, mixed)["strategy"] == O.ASYM_PIPELINE
    # the same queues through the oracle's Alg. 1
    asym = lambda p, g, c: (p, g, c[:2])
    for p, inp in (([], fast_cpu), ([], slow_cpu), ([1], mixed)):
        sel = lambda ps, gs, cs, inp=inp: {k: v for k, v in inp.items()}
        assert O.main_scheduler(p, [0] * 8, [0] * 5, asym, sel) == \
            sched.main(len(p), 8, 5, 2, inp)["strategy"]


@pytest.mark.parametrize("bad", [
    dict(n_g=0.0, n_c=1.0, t_glinear=1.0, t_gatt=1.0),
    dict(n_g=1.0, n_c=-1.0, t_glinear=1.0, t_gatt=1.0),
    dict(n_g=1.0, n_c=1.0, t_glinear=0.0, t_gatt=1.0),
    dict(n_g=1.0, n_c=1.0, t_glinear=1.0, t_gatt=float("nan")),
    dict(n_g=1.0, n_c=1.0, t_glinear=1.0, t_gatt=1.0, prefill=True, t_glinear_pref=-1.0),
])
def test_select_rejects_bad_inputs(lib, bad):
    from paper_2506_03296_amd.cpu import CpuError
    with pytest.raises(CpuError):
        sched.select(**bad)


def test_main_rejects_bad_queues(lib):
    from paper_2506_03296_amd.cpu import CpuError
    with pytest.raises(CpuError):
        sched.main(0, 1, 2, 3)
    with pytest.raises(CpuError):
        sched.main(-1, 1, 0, 0)


# ---------------------------------------------------------------------------
# profile tables
# ---------------------------------------------------------------------------

def random_profile(rng):
    def axis(n, lo, hi):
        return sorted(rng.sample(range(lo, hi), n))
    gt = axis(rng.randint(1, 6), 100, 10 ** 6)
    gb = axis(rng.randint(1, 5), 1, 2048)
    cb = axis(rng.randint(1, 4), 1, 512)
    ct = axis(rng.randint(1, 5), 16, 10 ** 6)
    pt = axis(rng.randint(1, 4), 16, 10 ** 5)
    return dict(
        gatt_tokens=[float(x) for x in gt], gatt_seconds=sorted(rng.uniform(1e-6, 1e-2) for _ in gt),
        glin_batch=[float(x) for x in gb], glin_seconds=sorted(rng.uniform(1e-5, 1e-2) for _ in gb),
        cpu_batch=[float(x) for x in cb], cpu_tokens=[float(x) for x in ct],
        cpu_seconds=[sorted(rng.uniform(1e-5, 1.0) for _ in ct) for _ in cb],
        pref_tokens=[float(x) for x in pt], pref_linear_seconds=sorted(rng.uniform(1e-4, 1e-1) for _ in pt),
        pref_attn_seconds=sorted(rng.uniform(1e-5, 1e-1) for _ in pt))


def test_interp1_matches_oracle(lib):
    rng = random.Random(11)
    for _ in range(3000):
        n = rng.randint(1, 7)
        xs = sorted(rng.sample(range(-1000, 1000), n))
        ys = [rng.uniform(-5, 50) for _ in xs]
        x = rng.uniform(-1500, 1500)
        assert close(sched.interp1(xs, ys, x), O.interp1([float(v) for v in xs], ys, x), 1e-12) or \
            abs(sched.interp1(xs, ys, x) - O.interp1([float(v) for v in xs], ys, x)) < 1e-12


def test_inputs_from_profile_matches_oracle(lib):
    rng = random.Random(12)
    for i in range(2000):
        prof = random_profile(rng)
        gb, gt = rng.uniform(1, 3000), rng.uniform(50, 2e6)
        cb, ct = rng.uniform(1, 600), rng.uniform(10, 2e6)
        pf = rng.choice([0.0, rng.uniform(10, 2e5)])
        try:
            ref = O.inputs_from_profile(prof, gb, gt, cb, ct, prefill_tokens=pf)
        except ZeroDivisionError:
            # a table extended to zero time: the library refuses it
            from paper_2506_03296_amd.cpu import CpuError
            with pytest.raises(CpuError):
                sched.inputs_from_profile(prof, gb, gt, cb, ct, prefill_tokens=pf)
            continue
        if ref["t_gatt"] <= 0 or ref["t_glinear"] <= 0:
            continue
        got = sched.inputs_from_profile(prof, gb, gt, cb, ct, prefill_tokens=pf)
        for k in ("n_g", "n_c", "t_glinear", "t_gatt", "t_glinear_pref", "t_gatt_pref"):
            if k in ref:
                assert close(got[k], ref[k], 1e-12), (k, got[k], ref[k])


def test_profile_validation(lib):
    from paper_2506_03296_amd.cpu import CpuError
    prof = random_profile(random.Random(3))
    bad = dict(prof, gatt_tokens=list(reversed(prof["gatt_tokens"])) if len(prof["gatt_tokens"]) > 1 else [1.0, 0.5],
               gatt_seconds=prof["gatt_seconds"] if len(prof["gatt_tokens"]) > 1 else [1.0, 1.0])
    with pytest.raises(CpuError):
        sched.inputs_from_profile(bad, 8, 1000, 1, 100)
    with pytest.raises(CpuError):
        sched.inputs_from_profile(dict(prof, pref_tokens=[]), 8, 1000, 1, 100, prefill_tokens=10)
    with pytest.raises(CpuError):
        sched.inputs_from_profile(prof, 8, 0, 1, 100)


def test_gpu_token_capacity(lib):
    # Llama-3.1-8B: 32 layers x 8 kv-heads x 128 dims, fp16 K and V = 128 KiB per token
    assert sched.gpu_token_capacity(128 * 1024 * 1000, 32, 8, 128) == 1000
    assert sched.gpu_token_capacity(128 * 1024 * 1000 - 1, 32, 8, 128) == 999
    assert sched.gpu_token_capacity(-1, 32, 8, 128) == 0


# ---------------------------------------------------------------------------
# ABI
# ---------------------------------------------------------------------------

def _struct_fields(name):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct %s \{(.*?)\} %s;" % (name, name), text, re.S).group(1)
    fields = []
    for decl in body.split(";"):
        decl = decl.strip()
        if not decl:
            continue
        names = decl.split(None, 1)[1] if not decl.startswith("const") else decl.split(None, 2)[2]
        for n in names.split(","):
            fields.append(re.sub(r"[\s*]", "", n))
    return fields


def test_structs_match_header(lib):
    assert _struct_fields("apex_sched_inputs") == [f[0] for f in sched.Inputs._fields_]
    assert _struct_fields("apex_sched_result") == [f[0] for f in sched.Result._fields_]
    assert _struct_fields("apex_sched_profile") == [f[0] for f in sched.Profile._fields_]


def test_header_symbols_are_exported(lib):
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    declared = set(re.findall(r"\b(apex_sched_\w+)\s*\(", text))
    assert declared == set(sched.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(lib, name)
