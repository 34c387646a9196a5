"""Pins of the fp64 oracle against things other than itself (CPU only).

The paper prints no attention inputs or outputs, so the pins come from the
mathematics of softmax attention: an independent brute force on tiny inputs,
a library routine (torch's scaled_dot_product_attention in float64) on a
densified copy, closed forms (one token, identical keys, two tokens, zero
query), invariants (block placement, token order, weights summing to one,
shift/scale of V), the consecutive GQA head grouping, and hand-derived golden
cases under tests/golden/.  test_planted_mistakes checks that a plausible bug
planted in a copy of the oracle fails at least one of them.
"""
import json
import math
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest

import apex_workloads as W
from oracle import brute_force

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def run(oracle_mod, case, **kw):
    return oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale, **kw)


# ---------------------------------------------------------------------------
# fp16 decoding
# ---------------------------------------------------------------------------

def test_f16_decoder_all_patterns(oracle_mod):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle_mod.f16_bits_to_f64(bits)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


# ---------------------------------------------------------------------------
# brute force and library special case
# ---------------------------------------------------------------------------

TINY = [
    # lens, Hq, Hkv, d, block_size
    ([3, 17, 1], 2, 2, 8, 4),
    ([40, 5], 4, 2, 8, 16),
    ([33, 16, 2], 4, 1, 4, 1),
    ([9], 8, 2, 16, 4),
    ([20, 31], 4, 4, 128, 16),
]


@pytest.mark.parametrize("lens,Hq,Hkv,d,bs", TINY)
def test_matches_brute_force(oracle_mod, lens, Hq, Hkv, d, bs):
    case = W.make_host_case(lens, Hq, Hkv, d=d, block_size=bs, seed=sum(lens) + d)
    ours = run(oracle_mod, case)
    ref = brute_force.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                       case.context_lens, case.scale)
    np.testing.assert_allclose(ours, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_matches_torch_sdpa_f64(oracle_mod, G):
    torch = pytest.importorskip("torch")
    Hkv = 2
    Hq = Hkv * G
    lens = [1, 16, 45, 77]
    case = W.make_host_case(lens, Hq, Hkv, d=64, block_size=16, seed=11 * G)
    ours = run(oracle_mod, case)
    q = torch.from_numpy(case.q.astype(np.float64))
    for b, L in enumerate(lens):
        K = torch.from_numpy(brute_force.dense_kv(case.k_cache, case.block_table, b, L))
        V = torch.from_numpy(brute_force.dense_kv(case.v_cache, case.block_table, b, L))
        K = K.repeat_interleave(G, dim=0)  # [Hq][L][d]
        V = V.repeat_interleave(G, dim=0)
        o = torch.nn.functional.scaled_dot_product_attention(
            q[b][:, None, :], K, V, scale=float(case.scale))[:, 0, :]
        np.testing.assert_allclose(ours[b], o.numpy(), rtol=0, atol=1e-12)


def test_lse_matches_logsumexp(oracle_mod):
    from scipy.special import logsumexp
    case = W.make_host_case([5, 30], 4, 2, d=16, block_size=4, seed=3)
    _, lse = run(oracle_mod, case, return_lse=True)
    q = case.q.astype(np.float64)
    for b, L in enumerate(case.context_lens):
        K = brute_force.dense_kv(case.k_cache, case.block_table, b, int(L))
        for h in range(4):
            z = case.scale * (K[h // 2] @ q[b, h])
            assert abs(lse[b, h] - logsumexp(z)) < 1e-12


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------

def test_single_token_returns_v_exactly(oracle_mod):
    case = W.make_host_case([1, 1, 1], 8, 2, seed=5)
    out = run(oracle_mod, case)
    for b in range(3):
        blk = case.block_table[b, 0]
        for h in range(8):
            assert np.array_equal(out[b, h], case.v_cache[blk, h // 4, 0].astype(np.float64))


def _set_all_keys(case, key_by_head):
    for b, L in enumerate(case.context_lens):
        for t in range(int(L)):
            blk = case.block_table[b, t // 16]
            case.k_cache[blk, :, t % 16, :] = key_by_head


def test_identical_keys_give_mean_of_v(oracle_mod):
    case = W.make_host_case([7, 50, 129], 4, 2, seed=6)
    _set_all_keys(case, np.random.default_rng(0).standard_normal((2, 128)).astype(np.float16))
    out = run(oracle_mod, case)
    for b, L in enumerate(case.context_lens):
        V = brute_force.dense_kv(case.v_cache, case.block_table, b, int(L))
        for h in range(4):
            np.testing.assert_allclose(out[b, h], V[h // 2].mean(axis=0), rtol=0, atol=1e-13)


@pytest.mark.parametrize("what", ["q", "scale"])
def test_zero_query_or_scale_gives_mean_of_v(oracle_mod, what):
    case = W.make_host_case([3, 64], 4, 4, seed=7)
    if what == "q":
        case.q[:] = 0
    else:
        case.scale = 0.0
    out = run(oracle_mod, case)
    for b, L in enumerate(case.context_lens):
        V = brute_force.dense_kv(case.v_cache, case.block_table, b, int(L))
        for h in range(4):
            np.testing.assert_allclose(out[b, h], V[h].mean(axis=0), rtol=0, atol=1e-13)


def test_two_tokens_sigmoid_form(oracle_mod):
    case = W.make_host_case([2], 2, 1, d=32, block_size=16, seed=8)
    out = run(oracle_mod, case)
    blk = case.block_table[0, 0]
    k = case.k_cache[blk, 0, :2].astype(np.float64)
    v = case.v_cache[blk, 0, :2].astype(np.float64)
    for h in range(2):
        qh = case.q[0, h].astype(np.float64)
        z1, z2 = (case.scale * float(np.dot(qh, k[i])) for i in range(2))
        s1 = 1.0 / (1.0 + math.exp(z2 - z1))
        s2 = 1.0 / (1.0 + math.exp(z1 - z2))
        np.testing.assert_allclose(out[0, h], s1 * v[0] + s2 * v[1], rtol=0, atol=1e-14)


def test_empty_and_negative_contexts_give_zero_rows(oracle_mod):
    case = W.make_host_case([0, 5, 0], 4, 2, seed=9)
    case.context_lens[2] = -3
    out, lse = run(oracle_mod, case, return_lse=True)
    assert np.all(out[0] == 0) and np.all(out[2] == 0)
    assert np.all(np.isneginf(lse[0])) and np.all(np.isneginf(lse[2]))
    assert np.all(np.isfinite(out[1])) and np.any(out[1] != 0)


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def test_physical_block_permutation_is_bitwise_invariant(oracle_mod):
    case = W.make_host_case([17, 100, 33], 4, 2, seed=10, slack_blocks=3)
    ref = run(oracle_mod, case)
    rng = np.random.default_rng(1)
    nb = case.k_cache.shape[0]
    perm = rng.permutation(nb)                # new position of old block i is perm[i]
    k2 = np.empty_like(case.k_cache)
    v2 = np.empty_like(case.v_cache)
    k2[perm] = case.k_cache
    v2[perm] = case.v_cache
    bt2 = perm[case.block_table].astype(np.int32)
    out = oracle_mod.decode_attention_f64(case.q, k2, v2, bt2, case.context_lens, case.scale)
    assert np.array_equal(out, ref)


def test_logical_token_permutation_invariant(oracle_mod):
    lens = [37, 64]
    case = W.make_host_case(lens, 4, 2, seed=12)
    ref = run(oracle_mod, case)
    rng = np.random.default_rng(2)
    for b, L in enumerate(lens):
        perm = rng.permutation(L)
        K = np.stack([case.k_cache[case.block_table[b, t // 16], :, t % 16] for t in range(L)])
        V = np.stack([case.v_cache[case.block_table[b, t // 16], :, t % 16] for t in range(L)])
        for t in range(L):
            blk = case.block_table[b, t // 16]
            case.k_cache[blk, :, t % 16] = K[perm[t]]
            case.v_cache[blk, :, t % 16] = V[perm[t]]
    out = run(oracle_mod, case)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)


def test_weights_sum_to_one_and_unit_values(oracle_mod):
    case = W.make_host_case([1, 23, 300], 4, 1, seed=13)
    for b in range(3):
        for h in range(4):
            w = oracle_mod.softmax_weights_f64(case.q, case.k_cache, case.v_cache,
                                               case.block_table, case.context_lens,
                                               case.scale, b, h)
            assert len(w) == case.context_lens[b]
            assert np.all(w > 0)
            assert abs(w.sum() - 1.0) < 1e-12
    case.v_cache[:] = 1
    out = run(oracle_mod, case)
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-13)


def test_shift_and_power_of_two_scaling_of_v(oracle_mod):
    case = W.make_host_case([10, 77], 4, 2, seed=14)
    grid = np.random.default_rng(3).integers(-256, 257, size=case.v_cache.shape) / 64.0
    case.v_cache[:] = grid.astype(np.float16)           # exact in fp16, |v| <= 4
    base = run(oracle_mod, case)
    v0 = case.v_cache.copy()
    case.v_cache[:] = (grid + 1.0).astype(np.float16)   # still exact
    np.testing.assert_allclose(run(oracle_mod, case), base + 1.0, rtol=0, atol=1e-13)
    case.v_cache[:] = (v0.astype(np.float64) * 2.0).astype(np.float16)
    np.testing.assert_allclose(run(oracle_mod, case), 2.0 * base, rtol=0, atol=1e-13)


@pytest.mark.parametrize("G", [2, 4])
def test_gqa_equals_mha_with_repeated_kv_heads(oracle_mod, G):
    Hkv = 2
    case = W.make_host_case([19, 64], Hkv * G, Hkv, seed=15 + G)
    gqa = run(oracle_mod, case)
    k_rep = np.repeat(case.k_cache, G, axis=1)
    v_rep = np.repeat(case.v_cache, G, axis=1)
    mha = oracle_mod.decode_attention_f64(case.q, k_rep, v_rep, case.block_table,
                                          case.context_lens, case.scale)
    assert np.array_equal(gqa, mha)


def test_nan_poison_outside_context_is_never_read(oracle_mod):
    clean = W.make_host_case([5, 40, 16], 4, 2, seed=16, slack_blocks=2)
    dirty = W.make_host_case([5, 40, 16], 4, 2, seed=16, slack_blocks=2, poison=True)
    np.testing.assert_array_equal(run(oracle_mod, clean), run(oracle_mod, dirty))


# ---------------------------------------------------------------------------
# hand-derived golden cases
# ---------------------------------------------------------------------------

def _golden_cases():
    with open(os.path.join(GOLDEN, "closed_form_cases.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("gc", _golden_cases(), ids=lambda c: c["name"])
def test_golden_closed_form_cases(oracle_mod, gc):
    q = np.asarray(gc["q"], dtype=np.float16)
    k = np.asarray(gc["k_cache"], dtype=np.float16)
    v = np.asarray(gc["v_cache"], dtype=np.float16)
    bt = np.asarray(gc["block_table"], dtype=np.int32)
    lens = np.asarray(gc["context_lens"], dtype=np.int32)
    out = oracle_mod.decode_attention_f64(q, k, v, bt, lens, gc["scale"])
    np.testing.assert_allclose(out, np.asarray(gc["expected"]), rtol=0, atol=gc["atol"])


# ---------------------------------------------------------------------------
# the pins catch planted mistakes (mutants of a temporary copy of the oracle)
# ---------------------------------------------------------------------------

MUTANTS = {
    "slot_uses_block_index": ("const int slot = t % block_size;", "const int slot = t / block_size % block_size;"),
    "block_uses_slot": ("(size_t)(t / block_size)];", "(size_t)(t % block_size)];"),
    "head_map_modulo": ("const int g = h / group;", "const int g = h % Hkv;"),
    "kv_index_transposed": ("(((size_t)blk * (size_t)Hkv + (size_t)g) * (size_t)block_size + (size_t)slot)",
                            "(((size_t)blk * (size_t)block_size + (size_t)slot) * (size_t)Hkv + (size_t)g)"),
    "sign_flip": ("w[t] = exp(w[t] - zmax);", "w[t] = exp(zmax - w[t]);"),
    "scale_dropped": ("w[t] = scale * dot;", "w[t] = dot;"),
    "last_token_dropped": ("for (int t = 0; t < L; ++t) {\n        w[t] /= Z;", "for (int t = 0; t < L - 1; ++t) {\n        w[t] /= Z;"),
    "no_normalisation": ("w[t] /= Z;", "w[t] /= 1.0;"),
    "max_not_subtracted_overflow": ("w[t] = exp(w[t] - zmax);", "w[t] = exp(w[t]);"),
}


def _build_mutant(src, old, new, tmpdir, name):
    text = open(src).read()
    assert old in text, f"mutation anchor for {name} not found"
    path = os.path.join(tmpdir, f"{name}.c")
    with open(path, "w") as f:
        f.write(text.replace(old, new, 1))
    lib = os.path.join(tmpdir, f"{name}.so")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                           "-ffp-contract=off", path, "-o", lib, "-lm"])
    return lib


def _pins_pass(mod):
    """A quick subset of the pins above, run against module ``mod``."""
    try:
        for lens, Hq, Hkv, d, bs in TINY[:4]:
            case = W.make_host_case(lens, Hq, Hkv, d=d, block_size=bs, seed=sum(lens) + d)
            ours = mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                            case.context_lens, case.scale)
            ref = brute_force.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                               case.context_lens, case.scale)
            if not np.allclose(ours, ref, rtol=0, atol=1e-12):
                return False
        # a large-logit case: overflow without the max subtraction
        case = W.make_host_case([30], 2, 1, d=8, block_size=4, seed=1, scale=1000.0)
        ours = mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                        case.context_lens, case.scale)
        ref = brute_force.decode_attention(case.q, case.k_cache, case.v_cache, case.block_table,
                                           case.context_lens, case.scale)
        return bool(np.allclose(ours, ref, rtol=0, atol=1e-12))
    except Exception:
        return False


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_planted_mistakes(oracle_mod):
    import oracle as pkg
    src = os.path.join(os.path.dirname(pkg.__file__), "ref_decode.c")
    assert _pins_pass(pkg)
    with tempfile.TemporaryDirectory() as tmp:
        for name, (old, new) in MUTANTS.items():
            lib = _build_mutant(src, old, new, tmp, name)
            saved = pkg._LIB
            saved_path = pkg._build.LIB
            try:
                pkg._LIB = None
                pkg._build.LIB = lib
                caught = not _pins_pass(pkg)
            finally:
                pkg._LIB = saved
                pkg._build.LIB = saved_path
            assert caught, f"planted mistake '{name}' passed every pin"


# ---------------------------------------------------------------------------
# the multiset form of attention over a table that repeats blocks
# (tests/multiset_attention.py), which stands in for the oracle on contexts
# too long for its loop
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("G,Hkv", [(1, 1), (4, 1), (2, 3)])
def test_multiset_form_matches_the_oracle_on_repeating_tables(oracle_mod, G, Hkv):
    import multiset_attention as MS
    rng = np.random.default_rng(300 + 10 * G + Hkv)
    pool, bs, d = 5, 16, 128
    k = rng.standard_normal((pool, Hkv, bs, d)).astype(np.float16)
    v = rng.standard_normal((pool, Hkv, bs, d)).astype(np.float16)
    for trial in range(6):
        L = int(rng.integers(1, 40 * bs))
        nb = -(-L // bs)
        table = rng.integers(0, pool, size=(1, nb + 2)).astype(np.int32)
        if trial % 2:
            table[0, :nb - 1] = 0                 # one block repeated, another at the end
            table[0, nb - 1] = 1
        q = rng.standard_normal((1, G * Hkv, d)).astype(np.float16)
        scale = float(np.float32(1.0 / math.sqrt(d)))
        ref = oracle_mod.decode_attention_f64(q, k, v, table, np.array([L], dtype=np.int32), scale)[0]
        got = MS.multiset_attention(q[0], k, v, table[0], L, scale)
        assert np.allclose(got, ref, rtol=0, atol=1e-12), (trial, L)


def test_multiset_form_counts_and_a_planted_miscount(oracle_mod):
    """Token counts of a ragged table written out by hand; one count off is
    visible in the attention."""
    import multiset_attention as MS
    c = MS.token_counts(np.array([2, 0, 2, 1], dtype=np.int32), 3 * 16 + 5, 16, 3)
    assert c[2].tolist() == [2.0] * 16
    assert c[0].tolist() == [1.0] * 16
    assert c[1].tolist() == [1.0] * 5 + [0.0] * 11
    rng = np.random.default_rng(7)
    k = rng.standard_normal((3, 1, 16, 128)).astype(np.float16)
    v = rng.standard_normal((3, 1, 16, 128)).astype(np.float16)
    q = rng.standard_normal((1, 1, 128)).astype(np.float16)
    table = np.array([[2, 0, 2, 1]], dtype=np.int32)
    ref = oracle_mod.decode_attention_f64(q, k, v, table, np.array([53], dtype=np.int32), 0.125)[0]
    assert np.allclose(MS.multiset_attention(q[0], k, v, table[0], 53, 0.125), ref, rtol=0, atol=1e-12)
    # a context one token longer counts slot 5 of block 1 once more
    assert not np.allclose(MS.multiset_attention(q[0], k, v, table[0], 54, 0.125), ref, rtol=0, atol=1e-6)
