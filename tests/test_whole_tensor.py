"""The chunked whole-tensor oracle used by the full-size GPU tests, on the CPU:
chunking requests changes nothing, and the error statistics find a planted
error where it is."""
import numpy as np
import pytest

import apex_workloads as W
import whole_tensor

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def c1_cpu():
    return W.DeviceWorkload("c1", device="cpu")


def test_chunked_reference_equals_one_call(oracle_mod, c1_cpu):
    wl = c1_cpu
    whole = oracle_mod.decode_attention_f64(wl.q.numpy(), wl.k_cache.numpy(), wl.v_cache.numpy(),
                                            wl.block_table.numpy(), wl.context_lens.numpy(), wl.scale)
    for chunk in (1, 3, 64):
        got = whole_tensor.oracle_reference(oracle_mod, wl, chunk=chunk)
        assert np.array_equal(got, whole), chunk


def test_prepare_hook_sees_each_chunk_once(oracle_mod, c1_cpu):
    seen = []

    def prepare(case, reqs):
        seen.append(list(reqs))
        assert case.q.shape[0] == len(reqs)
        return case

    whole_tensor.oracle_reference(oracle_mod, c1_cpu, chunk=3, prepare=prepare)
    assert seen == [[0, 1, 2], [3]]


def test_error_statistics_find_a_planted_error():
    rng = np.random.default_rng(3)
    ref = rng.standard_normal((5, 4, 8))
    got = ref.copy()
    got[3, 2, 7] += 1.5e-3
    e = whole_tensor.whole_tensor_errors(got, ref)
    assert e["finite"] and e["requests"] == 5
    assert e["worst_request"] == 3
    assert abs(e["max_abs"] - 1.5e-3) < 1e-12
    assert abs(e["rel_l2"] - 1.5e-3 / np.linalg.norm(ref)) < 1e-12
    whole_tensor.assert_whole_tensor(got, ref, "planted 1.5e-3")
    got[1, 0, 0] += 3e-3
    with pytest.raises(AssertionError, match="max-abs"):
        whole_tensor.assert_whole_tensor(got, ref, "planted 3e-3")
    got[1, 0, 0] = np.nan
    with pytest.raises(AssertionError, match="non-finite"):
        whole_tensor.assert_whole_tensor(got, ref, "NaN")
