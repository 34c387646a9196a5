"""Pins of the scheduler oracle (oracle/scheduler.py), CPU only.

The pins come from the paper's own algebra and numbers, checked in exact
rational arithmetic where a decision is involved:
- Eq. 5 and its solved form Eq. 6 agree on random rational inputs, and the
  decode-only branch of Alg. 2 agrees with Eq. 6;
- the paper's worked numbers (Sec. 3.2): for T_gatt / T_glinear between 0.5
  and 1.5 the Eq. 6 bound lies between 3 + 2 sqrt 2 ~ 5.83 (its minimum, at
  sqrt 2) and 7.5 (at 0.5), so the CPU rate must reach 1 / 7.5 ~ 13 % of the
  GPU rate;
- strictness at the boundary, limits (no CPU work never pays; a vanishing
  linear time makes the bound unbounded);
- the mixed-workload forms reduce to closed conditions derived by hand, and
  with no prefill time the Eq.-5-shaped reading reduces to Eq. 6;
- Alg. 1's three exits;
- planted mistakes in a copy of the oracle fail at least one pin.
"""
import inspect
import math
import random
import types
from fractions import Fraction as F

import pytest

from oracle import scheduler as S


def rand_pos(rng, lo=1, hi=10 ** 6):
    return F(rng.randint(lo, hi), rng.randint(lo, hi))


def _eq5_eq6_agree(mod, rng, n=3000):
    for _ in range(n):
        ng, nc, tl, ta = (rand_pos(rng) for _ in range(4))
        lhs = mod.pipelining_pays_decode(ng, nc, tl, ta)
        solved = ng / nc < 2 * tl / ta + 3 + ta / tl       # Eq. 6 written out here
        if lhs != solved:
            return False
        if mod.strategy_selection(ng, nc, tl, ta)[0] != (S.ASYM_PIPELINE if solved else S.ASYNC_OVERLAP):
            return False
    return True


def test_eq5_is_equivalent_to_eq6_exactly():
    assert _eq5_eq6_agree(S, random.Random(1))


def test_ratio_bound_matches_the_papers_numbers():
    # T_gatt / T_glinear = r  ->  bound = 2 / r + 3 + r
    assert S.ratio_bound(F(2), F(1)) == F(15, 2)          # r = 0.5 -> 7.5
    assert S.ratio_bound(F(2), F(3)) == F(35, 6)          # r = 1.5 -> 5.833...
    assert S.ratio_bound(F(1), F(1)) == 6
    # minimum 3 + 2 sqrt 2 at r = sqrt 2
    r = math.sqrt(2)
    assert abs(S.ratio_bound(1.0, r) - (3 + 2 * math.sqrt(2))) < 1e-12
    grid = [0.5 + i / 1000 for i in range(1001)]
    vals = [S.ratio_bound(1.0, x) for x in grid]
    assert abs(min(vals) - (3 + 2 * math.sqrt(2))) < 1e-6 and abs(max(vals) - 7.5) < 1e-12
    # the CPU must reach 1 / 7.5 = 13.3 % of the GPU rate at r = 0.5
    assert abs(1 / 7.5 - 0.1333) < 1e-4
    tl, ta, ng = F(2), F(1), F(1000)
    assert not S.pipelining_pays_decode(ng, ng * F(2, 15), tl, ta)        # exactly at 13.33 %
    assert S.pipelining_pays_decode(ng, ng * F(2, 15) + F(1, 10 ** 9), tl, ta)
    assert not S.pipelining_pays_decode(ng, ng * F(13, 100), tl, ta)      # 13 % is not enough
    # "N_C often below 10 % of N_G" never pays over the whole stated range
    for r in (F(1, 2), F(1), F(3, 2)):
        assert not S.pipelining_pays_decode(F(100), F(10), F(1), r)


def test_limits():
    rng = random.Random(2)
    for _ in range(200):
        ng, tl, ta = (rand_pos(rng) for _ in range(3))
        assert not S.pipelining_pays_decode(ng, F(0), tl, ta)              # no CPU work
        assert S.pipelining_pays_decode(ng, ng, tl, ta)                     # CPU as fast as GPU
    assert S.ratio_bound(1e-12, 1.0) > 1e11                                 # linears vanish


def test_decode_branch_throughputs():
    st, pipe, gpu = S.strategy_selection(F(10), F(1), F(3), F(2))
    assert gpu == F(10) * 2 / (3 + 2)
    assert pipe == (F(10) * 2 + 1 * (2 * 3 + 2)) / (2 * 3 + 2)
    assert st == (S.ASYM_PIPELINE if pipe > gpu else S.ASYNC_OVERLAP)


def test_mixed_paper_form_reduces_to_cpu_tokens_above_gpu_linear_tokens():
    # (N_G T_gatt + N_C T_ov) / (T_gl + T_gatt) > N_G  <=>  N_C T_ov > N_G T_gl
    rng = random.Random(3)
    for _ in range(3000):
        ng, nc, tl, ta, tlp, tap = (rand_pos(rng) for _ in range(6))
        t_ov = tlp + tap + tl + ta
        st = S.strategy_selection(ng, nc, tl, ta, prefill=True, t_glinear_pref=tlp, t_gatt_pref=tap)[0]
        assert (st == S.ASYM_PIPELINE) == (nc * t_ov > ng * tl)


def test_mixed_eq5_form_closed_condition_and_decode_limit():
    # (N_G T_gatt + N_C T_ov) / T_ov > N_G T_gatt / (T_gl + T_gatt)
    #   <=>  N_G / N_C < (T_gl + T_gatt) T_ov / (T_gatt (T_glp + T_gap))
    rng = random.Random(4)
    for _ in range(3000):
        ng, nc, tl, ta, tlp, tap = (rand_pos(rng) for _ in range(6))
        t_ov = tlp + tap + tl + ta
        st = S.strategy_selection(ng, nc, tl, ta, prefill=True, t_glinear_pref=tlp,
                                  t_gatt_pref=tap, mixed_form="eq5")[0]
        assert (st == S.ASYM_PIPELINE) == (ng / nc < (tl + ta) * t_ov / (ta * (tlp + tap)))
        # a "prefill" that costs one more decode linear is the decode-only case
        st2 = S.strategy_selection(ng, nc, tl, ta, prefill=True, t_glinear_pref=tl, t_gatt_pref=F(0),
                                   mixed_form="eq5")[0]
        assert st2 == S.strategy_selection(ng, nc, tl, ta)[0]


def test_eq7_and_eq1_to_eq4():
    assert S.t_overlap_mixed(1, 2, 3, 4) == 10
    assert S.t_gpuonly(3, 4) == 7
    assert S.t_overlap_decode(3, 4) == 10
    assert S.n_gtotal(5, 4) == 20 and S.n_ctotal(2, 10) == 20


def test_alg1_exits():
    calls = []

    def asym(p, dg, dc):
        calls.append(1)
        return p, dg, dc[:1] if len(dc) > 1 else []

    def inputs(p, dg, dc):
        return dict(n_g=F(10), n_c=F(9), t_glinear=F(1), t_gatt=F(1))

    assert S.main_scheduler([], [1, 2], [], asym, inputs) == S.GPU_ONLY
    assert not calls                                   # no CPU queue: nothing else is consulted
    assert S.main_scheduler([], [1], [7], asym, inputs) == S.ASYNC_OVERLAP
    assert S.main_scheduler([], [1], [7, 8], asym, inputs) == S.ASYM_PIPELINE   # 10/9 < 6
    slow = lambda p, dg, dc: dict(n_g=F(100), n_c=F(1), t_glinear=F(1), t_gatt=F(1))
    assert S.main_scheduler([], [1], [7, 8], asym, slow) == S.ASYNC_OVERLAP
    # mixed branch is taken when the pipelining sub-batch holds prefill requests
    mixed = lambda p, dg, dc: dict(n_g=F(100), n_c=F(1), t_glinear=F(1), t_gatt=F(1),
                                   t_glinear_pref=F(200), t_gatt_pref=F(0))
    assert S.main_scheduler([3], [1], [7, 8], asym, mixed) == S.ASYM_PIPELINE   # 1*202 > 100*1


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

MUTANTS = {
    "eq2_single_linear": ("t_ov = 2 * t_glinear + t_gatt", "t_ov = t_glinear + t_gatt"),
    "gpu_denominator": ("throughput_gpu = n_g * t_gatt / (t_glinear + t_gatt)\n        throughput_pipe",
                        "throughput_gpu = n_g * t_gatt / (2 * t_glinear + t_gatt)\n        throughput_pipe"),
    "strict_becomes_loose": ("ASYM_PIPELINE if throughput_pipe > throughput_gpu", "ASYM_PIPELINE if throughput_pipe >= throughput_gpu"),
    "rates_swapped": ("throughput_pipe = (n_g * t_gatt + n_c * t_ov) / (2 * t_glinear + t_gatt)",
                      "throughput_pipe = (n_c * t_gatt + n_g * t_ov) / (2 * t_glinear + t_gatt)"),
    "bound_term_dropped": ("return 2 * t_glinear / t_gatt + 3 + t_gatt / t_glinear", "return 2 * t_glinear / t_gatt + 3"),
    "mixed_prefill_dropped": ("t_ov = t_glinear_pref + t_gatt_pref + t_glinear + t_gatt\n        if",
                              "t_ov = t_glinear + t_gatt\n        if"),
    "eq5_cycle_time": ("pipe = (n_gtotal(n_g, t_gatt) + n_ctotal(n_c, t_ov)) / t_ov",
                       "pipe = (n_gtotal(n_g, t_gatt) + n_ctotal(n_c, t_ov)) / t_gpuonly(t_glinear, t_gatt)"),
    "alg1_order": ("    if len(d_cpu_in) == 0:\n        return GPU_ONLY", "    if len(d_cpu_in) == 0:\n        return ASYNC_OVERLAP"),
}


def _mutant(name):
    src = inspect.getsource(S)
    old, new = MUTANTS[name]
    assert old in src, name
    mod = types.ModuleType(f"sched_{name}")
    exec(compile(src.replace(old, new, 1), f"<{name}>", "exec"), mod.__dict__)
    return mod


def _pins_pass(mod):
    checks = [
        lambda: _eq5_eq6_agree(mod, random.Random(1), n=400),
        lambda: mod.ratio_bound(F(2), F(1)) == F(15, 2),
        lambda: not mod.pipelining_pays_decode(F(1000), F(1000) * F(2, 15), F(2), F(1)),
        # exactly at the Eq. 6 bound the throughputs tie: no pipelining
        lambda: mod.strategy_selection(F(1000), F(1000) * F(2, 15), F(2), F(1))[0] == S.ASYNC_OVERLAP,
        lambda: mod.strategy_selection(F(10), F(1), F(3), F(2))[2] == F(4),
        lambda: mod.strategy_selection(F(10), F(3), F(1), F(1))[0] == S.ASYM_PIPELINE,
        lambda: mod.strategy_selection(F(100), F(1), F(1), F(1), prefill=True, t_glinear_pref=F(200),
                                       t_gatt_pref=F(0))[0] == S.ASYM_PIPELINE,
        lambda: mod.strategy_selection(F(100), F(1), F(1), F(1), prefill=True, t_glinear_pref=F(50),
                                       t_gatt_pref=F(0))[0] == S.ASYNC_OVERLAP,
        lambda: mod.main_scheduler([], [1], [], lambda p, g, c: (p, g, c), None) == S.GPU_ONLY,
    ]
    try:
        return all(c() for c in checks)
    except Exception:
        return False


def test_planted_mistakes_are_caught():
    assert _pins_pass(S)
    for name in MUTANTS:
        assert not _pins_pass(_mutant(name)), f"planted mistake '{name}' passed every pin"


# ---------------------------------------------------------------------------
# profile interpolation
# ---------------------------------------------------------------------------

def test_interp1_hits_samples_is_linear_between_and_extends_the_end_segments():
    xs = [F(1), F(4), F(10)]
    ys = [F(2), F(8), F(11)]
    for x, y in zip(xs, ys):
        assert S.interp1(xs, ys, x) == y
    assert S.interp1(xs, ys, F(2)) == F(4)                  # slope 2 on [1, 4]
    assert S.interp1(xs, ys, F(7)) == F(19, 2)              # slope 1/2 on [4, 10]
    assert S.interp1(xs, ys, F(12)) == F(12)                # extended right
    assert S.interp1(xs, ys, F(0)) == F(0)                  # extended left: 2 - 2 = 0
    assert S.interp1(xs, ys, F(-5)) == 0                    # never below zero
    assert S.interp1([F(3)], [F(5)], F(100)) == 5           # one sample: constant


def test_interp2_is_bilinear_on_the_grid():
    bs, ts = [F(1), F(3)], [F(10), F(20)]
    table = [[F(1), F(3)], [F(5), F(11)]]
    assert S.interp2(bs, ts, table, F(1), F(10)) == 1
    assert S.interp2(bs, ts, table, F(3), F(20)) == 11
    # centre: mean of the four corners for a bilinear patch
    assert S.interp2(bs, ts, table, F(2), F(15)) == F(1 + 3 + 5 + 11, 4)


def test_inputs_from_profile_rates():
    prof = dict(gatt_tokens=[F(1000), F(2000)], gatt_seconds=[F(1, 100), F(2, 100)],
                glin_batch=[F(1), F(100)], glin_seconds=[F(1, 1000), F(100, 1000)],
                cpu_batch=[F(1), F(10)], cpu_tokens=[F(100), F(1000)],
                cpu_seconds=[[F(1), F(10)], [F(2), F(20)]],
                pref_tokens=[F(10), F(20)], pref_linear_seconds=[F(1), F(2)], pref_attn_seconds=[F(3), F(4)])
    kw = S.inputs_from_profile(prof, F(50), F(1500), F(1), F(100), prefill_tokens=F(15))
    assert kw["t_gatt"] == F(15, 1000) and kw["n_g"] == F(1500) / F(15, 1000)
    assert kw["t_glinear"] == F(50, 1000)
    assert kw["n_c"] == F(100)
    assert kw["t_glinear_pref"] == F(3, 2) and kw["t_gatt_pref"] == F(7, 2)
