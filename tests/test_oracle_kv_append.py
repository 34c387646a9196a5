"""Pins of the KV-append oracle (oracle/kv_cache.py) against things other than
itself, CPU only.

- a brute force that writes every element through its flat offset in the raw
  cache buffer (row-major [NB][Hkv][bs][d] arithmetic written out by hand);
- invariants: only the addressed slots change, every kv-head row of a token
  lands in the same slot, padding and out-of-pool slots change nothing, the
  written values are the new rows bit for bit;
- the decode step the append serves: appending each request's newest token at
  position L_b - 1 and attending with context_lens = L_b equals softmax
  attention over the request's old rows followed by the new one, computed on
  dense arrays (APEX Sec. 2.1: each iteration's new K/V join the cache that
  the next attention reads);
- planted mistakes in a copy of the oracle fail at least one of the above.
"""
import inspect
import math
import types

import numpy as np
import pytest

import apex_workloads as W
from oracle import brute_force, kv_cache


def brute_append(k_cache, v_cache, k_new, v_new, slots):
    """Element-by-element scatter through flat offsets of the raw buffers."""
    nb, hkv, bs, d = k_cache.shape
    kf = k_cache.reshape(-1).copy()
    vf = v_cache.reshape(-1).copy()
    kn = k_new.reshape(-1)
    vn = v_new.reshape(-1)
    for t, s in enumerate(slots):
        s = int(s)
        if not 0 <= s < nb * bs:
            continue
        blk, pos = divmod(s, bs)
        for g in range(hkv):
            for i in range(d):
                dst = ((blk * hkv + g) * bs + pos) * d + i
                src = (t * hkv + g) * d + i
                kf[dst] = kn[src]
                vf[dst] = vn[src]
    return kf.reshape(k_cache.shape), vf.reshape(v_cache.shape)


SMALL = [
    # T, NB, Hkv, d, bs, padding, out_of_range
    (1, 1, 1, 8, 1, 0, 0),
    (5, 2, 2, 8, 4, 1, 1),
    (16, 3, 3, 16, 8, 0, 2),
    (33, 4, 2, 8, 16, 3, 0),
    (7, 9, 1, 32, 2, 0, 0),
]


@pytest.mark.parametrize("T,NB,Hkv,d,bs,pad,oor", SMALL)
def test_matches_flat_offset_brute_force(T, NB, Hkv, d, bs, pad, oor):
    c = W.make_append_case(T, NB, Hkv, d, bs, seed=T * 7 + d, padding=pad, out_of_range=oor)
    ok, ov = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    bk, bv = brute_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    assert np.array_equal(ok.view(np.uint16), bk.view(np.uint16))
    assert np.array_equal(ov.view(np.uint16), bv.view(np.uint16))


def test_only_addressed_slots_change_and_hold_the_new_rows():
    c = W.make_append_case(40, 6, 4, 16, 16, seed=3, padding=5, out_of_range=4)
    kc, vc = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    nb, hkv, bs, d = c.k_cache.shape
    touched = np.zeros((nb, bs), dtype=bool)
    for t, s in enumerate(c.slot_mapping):
        if 0 <= s < nb * bs:
            blk, pos = divmod(int(s), bs)
            touched[blk, pos] = True
            assert np.array_equal(kc[blk, :, pos].view(np.uint16), c.k_new[t].view(np.uint16))
            assert np.array_equal(vc[blk, :, pos].view(np.uint16), c.v_new[t].view(np.uint16))
    assert touched.sum() == 40 - 5 - 4
    mask = np.broadcast_to(~touched[:, None, :, None], c.k_cache.shape)
    assert np.array_equal(kc.view(np.uint16)[mask], c.k_cache.view(np.uint16)[mask])
    assert np.array_equal(vc.view(np.uint16)[mask], c.v_cache.view(np.uint16)[mask])
    # the inputs are not modified
    assert not np.shares_memory(kc, c.k_cache)


def test_padding_and_out_of_pool_slots_change_nothing():
    c = W.make_append_case(6, 2, 2, 8, 4, seed=4, padding=3, out_of_range=3)
    kc, vc = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    assert np.array_equal(kc.view(np.uint16), c.k_cache.view(np.uint16))
    assert np.array_equal(vc.view(np.uint16), c.v_cache.view(np.uint16))


def test_nan_and_signed_zero_rows_are_copied_bit_for_bit():
    c = W.make_append_case(3, 2, 1, 8, 4, seed=5)
    c.k_new[0, 0, :4] = np.float16(np.nan)
    c.v_new[1, 0, :] = np.float16(-0.0)
    kc, vc = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    bk, bv = brute_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    assert np.array_equal(kc.view(np.uint16), bk.view(np.uint16))
    assert np.array_equal(vc.view(np.uint16), bv.view(np.uint16))


def _dense_attention(q, K, V, scale):
    """softmax(scale * q K^T) V for one query row over dense rows (float64)."""
    z = [scale * float(np.dot(q, K[t])) for t in range(K.shape[0])]
    top = max(z)
    e = [math.exp(x - top) for x in z]
    tot = sum(e)
    return sum((e[t] / tot) * V[t] for t in range(K.shape[0]))


@pytest.mark.parametrize("lens,Hq,Hkv", [([1, 16, 17, 40], 4, 2), ([33, 2], 2, 2)])
def test_append_then_attend_equals_attention_over_old_rows_plus_new(oracle_mod, lens, Hq, Hkv):
    # layout for the step: L_b counts the new token, whose slot is still stale
    case = W.make_host_case(lens, Hq, Hkv, d=16, block_size=16, seed=sum(lens))
    slots = W.append_slots(case.layout, 16)
    rng = np.random.default_rng(99)
    B = len(lens)
    kn = rng.standard_normal((B, Hkv, 16)).astype(np.float16)
    vn = rng.standard_normal((B, Hkv, 16)).astype(np.float16)
    kc, vc = kv_cache.kv_append(case.k_cache, case.v_cache, kn, vn, slots)
    out = oracle_mod.decode_attention_f64(case.q, kc, vc, case.block_table, case.context_lens,
                                          case.scale)
    G = Hq // Hkv
    for b, L in enumerate(lens):
        Kold = brute_force.dense_kv(case.k_cache, case.block_table, b, L - 1)
        Vold = brute_force.dense_kv(case.v_cache, case.block_table, b, L - 1)
        for h in range(Hq):
            g = h // G
            K = np.vstack([Kold[g], kn[b, g].astype(np.float64)[None]])
            V = np.vstack([Vold[g], vn[b, g].astype(np.float64)[None]])
            ref = _dense_attention(case.q[b, h].astype(np.float64), K, V, case.scale)
            np.testing.assert_allclose(out[b, h], ref, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

MUTANTS = {
    "block_and_position_swapped": ("block, pos = s // bs, s % bs", "block, pos = s % bs, s // bs"),
    "position_off_by_one": ("kc[block, :, pos, :] = kn[t]", "kc[block, :, (pos + 1) % bs, :] = kn[t]"),
    "v_gets_k": ("vc[block, :, pos, :] = vn[t]", "vc[block, :, pos, :] = kn[t]"),
    "last_slot_dropped": ("s >= nb * bs", "s >= nb * bs - 1"),
    "padding_wraps": ("if s < 0 or s >= nb * bs", "if s >= nb * bs"),
    "token_order_reversed": ("kc[block, :, pos, :] = kn[t]", "kc[block, :, pos, :] = kn[-1 - t]"),
}


def _mutant(name):
    src = inspect.getsource(kv_cache)
    old, new = MUTANTS[name]
    assert old in src, name
    mod = types.ModuleType(f"kv_cache_{name}")
    exec(compile(src.replace(old, new, 1), f"<{name}>", "exec"), mod.__dict__)
    return mod


def _pins_pass(mod):
    try:
        for T, NB, Hkv, d, bs, pad, oor in SMALL:
            c = W.make_append_case(T, NB, Hkv, d, bs, seed=T * 7 + d, padding=pad, out_of_range=oor)
            ok, ov = mod.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
            bk, bv = brute_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
            if not (np.array_equal(ok.view(np.uint16), bk.view(np.uint16))
                    and np.array_equal(ov.view(np.uint16), bv.view(np.uint16))):
                return False
        # the very last slot of the pool and a padding slot
        c = W.make_append_case(2, 1, 1, 8, 4, seed=1)
        c.slot_mapping[:] = [3, -1]
        ok, _ = mod.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
        bk, _ = brute_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
        return bool(np.array_equal(ok.view(np.uint16), bk.view(np.uint16)))
    except Exception:
        return False


def test_planted_mistakes_are_caught():
    assert _pins_pass(kv_cache)
    for name in MUTANTS:
        assert not _pins_pass(_mutant(name)), f"planted mistake '{name}' passed every pin"
