"""The committed MI355X profile (profiles/sched_profile_mi355x.json, written
by paper_2506_03296_amd.profiler on the GPU machine) drives the library's
scheduler and the oracle to the same decisions.  CPU only: it reads the
stored measurements, it does not re-measure them."""
import json
import os

import pytest

from oracle import scheduler as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILE = os.path.join(ROOT, "profiles", "sched_profile_mi355x.json")

sched = pytest.importorskip("paper_2506_03296_amd.sched")


@pytest.fixture(scope="module")
def profile():
    with open(PROFILE) as f:
        return json.load(f)


def test_tables_are_well_formed(profile):
    for xs in ("gatt_tokens", "glin_batch", "cpu_batch", "cpu_tokens", "pref_tokens"):
        v = profile[xs]
        assert all(b > a for a, b in zip(v, v[1:])), xs
    for ys in ("gatt_seconds", "glin_seconds", "pref_linear_seconds", "pref_attn_seconds"):
        assert all(t > 0 for t in profile[ys]), ys
    assert all(t > 0 for row in profile["cpu_seconds"] for t in row)
    assert len(profile["cpu_seconds"]) == len(profile["cpu_batch"])
    # attention time grows with the tokens read
    assert all(b > a for a, b in zip(profile["gatt_seconds"], profile["gatt_seconds"][1:]))


@pytest.mark.parametrize("prefill_tokens", [0.0, 1024.0, 8192.0])
def test_decisions_agree_with_the_oracle(profile, prefill_tokens):
    for row in profile["decisions"]:
        kw = sched.inputs_from_profile(profile, 32, 411026, row["cpu_batch"], row["cpu_tokens"],
                                       prefill_tokens=prefill_tokens)
        ref = O.inputs_from_profile(profile, 32, 411026, row["cpu_batch"], row["cpu_tokens"],
                                    prefill_tokens=prefill_tokens)
        for k in ref:
            assert abs(kw[k] - ref[k]) <= 1e-12 * abs(ref[k]), k
        got = sched.select(**kw)
        st, pipe, gpu = O.strategy_selection(prefill=prefill_tokens > 0, **ref)
        assert got["strategy"] == st
        if prefill_tokens == 0:
            assert got["strategy"] == row["strategy"]
            assert abs(ref["n_g"] / ref["n_c"] - row["ratio"]) <= 1e-9 * row["ratio"]


def test_measured_regime_is_async_overlap(profile):
    """On this GPU and host the CPU attends at a few percent of the GPU's
    rate, far above the Eq. 6 bound, so pipelining never pays."""
    for row in profile["decisions"]:
        assert row["ratio"] > 2 * row["bound"]
        assert row["strategy"] == O.ASYNC_OVERLAP
