"""Fused append: apex_decode_attention_ex with k_new/v_new attends the current
token (position L - 1) from the new rows and writes them to its cache slot in
the same launch.

Expected, from the oracles only: the KV append of oracle/kv_cache.py followed
by the fp64 attention over the appended caches.  Outputs to the attention bar,
the LSE to 1e-4 (see LSE_ABS), the caches bit for bit.  The current slots hold NaN in the
caches before the call, so reading one instead of the new rows would show.
"""
import numpy as np
import pytest

import apex_workloads as W
import whole_tensor
from oracle import kv_cache

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3
# The LSE is log(sum of the weights) + max, in fp32 with the weights carried to
# 22 significant bits (two fp16 parts): ~1e-6, checked to 1e-4 like the plain
# call's LSE.
LSE_ABS = 1e-4
D, BS = 128, 16


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(scope="module")
def apex():
    import paper_2506_03296_amd as A
    A.load_library()
    return A


def current_slots(case):
    slots = np.full(len(case.context_lens), -1, dtype=np.int64)
    for b, L in enumerate(case.context_lens):
        if L > 0:
            slots[b] = int(case.block_table[b, (L - 1) // BS]) * BS + (L - 1) % BS
    return slots


def fused_case(lens, G, Hkv, seed, stride=None):
    case = W.make_host_case(lens, G * Hkv, Hkv, seed=seed, poison=True, stride=stride)
    rng = np.random.default_rng(seed + 7)
    B = len(lens)
    kn = rng.standard_normal((B, Hkv, D)).astype(np.float16)
    vn = rng.standard_normal((B, Hkv, D)).astype(np.float16)
    slots = current_slots(case)
    kc, vc = case.k_cache.copy(), case.v_cache.copy()
    for s in slots[slots >= 0]:
        kc[s // BS, :, s % BS, :] = np.float16(np.nan)
        vc[s // BS, :, s % BS, :] = np.float16(np.nan)
    exp_k, exp_v = kv_cache.kv_append(kc, vc, kn, vn, slots)
    return case, kc, vc, kn, vn, exp_k, exp_v


def check(got, ref, what):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), what
    err = float(np.abs(got - ref).max())
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    print(f"[fused] {what}: max_abs={err:.3e} rel_l2={rel:.3e}", flush=True)
    assert err <= MAX_ABS and rel <= REL_L2, what


LENS = [1, 2, 15, 16, 17, 33, 0, 500, 1024, 4096, 3]


@pytest.mark.parametrize("G,Hkv", [(1, 8), (4, 8), (8, 2), (2, 4)])
@pytest.mark.parametrize("workers", [0, 1, 3, 200])
def test_fused_append_matches_append_then_attend(torch_cuda, apex, oracle_mod, G, Hkv, workers):
    torch = torch_cuda
    case, kc, vc, kn, vn, exp_k, exp_v = fused_case(LENS, G, Hkv, seed=101 + G * 10 + Hkv)
    ref, lse_ref = oracle_mod.decode_attention_f64(case.q, exp_k, exp_v, case.block_table,
                                                   case.context_lens, case.scale, return_lse=True)
    dev = "cuda"
    q = torch.from_numpy(case.q).to(dev)
    kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
    bt = torch.from_numpy(case.block_table).to(dev)
    cl = torch.from_numpy(case.context_lens).to(dev)
    lse = torch.empty((len(LENS), G * Hkv), dtype=torch.float32, device=dev)
    out = apex.decode_attention_ex(q, kd, vd, bt, cl, case.scale, num_workers=workers, lse_out=lse,
                                   k_new=torch.from_numpy(kn).to(dev), v_new=torch.from_numpy(vn).to(dev))
    torch.cuda.synchronize()
    check(out.cpu().numpy(), ref, f"G={G} Hkv={Hkv} workers={workers}")
    assert np.all(out.cpu().numpy()[np.asarray(LENS) == 0] == 0)
    got_lse = lse.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lse_ref)
    assert np.all(np.isneginf(got_lse[~fin]))
    assert np.max(np.abs(got_lse[fin] - lse_ref[fin])) <= LSE_ABS
    assert np.array_equal(kd.cpu().numpy().view(np.uint16), exp_k.view(np.uint16))
    assert np.array_equal(vd.cpu().numpy().view(np.uint16), exp_v.view(np.uint16))


def test_fused_append_from_a_fused_qkv_buffer_and_wide_table(torch_cuda, apex, oracle_mod):
    """k_new/v_new as views into one [B][Hq + 2 Hkv][d] projection output
    (token stride wider than a row), with an explicit wide table stride."""
    torch = torch_cuda
    lens = [700, 17, 1, 64, 2000]
    G, Hkv = 4, 8
    stride = 140
    case, kc, vc, kn, vn, exp_k, exp_v = fused_case(lens, G, Hkv, seed=131, stride=stride)
    ref = oracle_mod.decode_attention_f64(case.q, exp_k, exp_v, case.block_table, case.context_lens,
                                          case.scale)
    dev = "cuda"
    B, Hq = len(lens), G * Hkv
    qkv = torch.zeros((B, Hq + 2 * Hkv, D), dtype=torch.float16, device=dev)
    qkv[:, :Hq] = torch.from_numpy(case.q).to(dev)
    qkv[:, Hq:Hq + Hkv] = torch.from_numpy(kn).to(dev)
    qkv[:, Hq + Hkv:] = torch.from_numpy(vn).to(dev)
    q = qkv[:, :Hq].contiguous()
    kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
    bt = torch.from_numpy(case.block_table).to(dev)
    cl = torch.from_numpy(case.context_lens).to(dev)
    out = apex.decode_attention_ex(q, kd, vd, bt, cl, case.scale, block_table_stride=stride,
                                   k_new=qkv[:, Hq:Hq + Hkv], v_new=qkv[:, Hq + Hkv:])
    torch.cuda.synchronize()
    check(out.cpu().numpy(), ref, "fused qkv views")
    assert np.array_equal(kd.cpu().numpy().view(np.uint16), exp_k.view(np.uint16))
    assert np.array_equal(vd.cpu().numpy().view(np.uint16), exp_v.view(np.uint16))


def test_fused_append_on_the_checked_path(torch_cuda, apex, oracle_mod):
    torch = torch_cuda
    lens = [40, 1, 300, 16]
    case, kc, vc, kn, vn, exp_k, exp_v = fused_case(lens, 4, 8, seed=141)
    ref = oracle_mod.decode_attention_f64(case.q, exp_k, exp_v, case.block_table, case.context_lens,
                                          case.scale)
    dev = "cuda"
    kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
    out = apex.decode_attention_ex(torch.from_numpy(case.q).to(dev), kd, vd,
                                   torch.from_numpy(case.block_table).to(dev),
                                   torch.from_numpy(case.context_lens).to(dev), case.scale,
                                   check_inputs=True, k_new=torch.from_numpy(kn).to(dev),
                                   v_new=torch.from_numpy(vn).to(dev))
    torch.cuda.synchronize()
    assert apex.check_device_error() == 0
    check(out.cpu().numpy(), ref, "checked path")
    assert np.array_equal(kd.cpu().numpy().view(np.uint16), exp_k.view(np.uint16))


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_fused_append_full_size_whole_tensor(torch_cuda, apex, oracle_mod, name):
    """The fused call at full size, in the benchmark's launch configuration
    (default grid), over every request.  The oracle's inputs are each chunk of
    requests copied before the call (current slots holding NaN) with the
    oracle's own append of the new rows applied on the host; every request's
    slot is then checked bit for bit on the device."""
    torch = torch_cuda
    print(f"[fused full-size] generating {name}", flush=True)
    wl = W.DeviceWorkload(name)
    cfg = wl.cfg
    B, Hkv = cfg.B, cfg.Hkv
    lens = np.asarray(wl.lens, dtype=np.int64)
    blocks = np.asarray([wl.layout.block_table[b, (L - 1) // BS] for b, L in enumerate(lens)], dtype=np.int64)
    pos = (lens - 1) % BS
    dev = "cuda"
    blk_d, pos_d = torch.from_numpy(blocks).to(dev), torch.from_numpy(pos).to(dev)
    for c in (wl.k_cache, wl.v_cache):
        c[blk_d, :, pos_d, :] = float("nan")
    g = torch.Generator(device=dev)
    g.manual_seed(77)
    kn = torch.randn((B, Hkv, D), generator=g, device=dev).half()
    vn = torch.randn((B, Hkv, D), generator=g, device=dev).half()
    kn_h, vn_h = kn.cpu().numpy(), vn.cpu().numpy()

    def append_on_host(case, reqs):
        L = case.context_lens.astype(np.int64)
        rows = np.arange(len(reqs))
        slots = case.block_table[rows, (L - 1) // BS].astype(np.int64) * BS + (L - 1) % BS
        exp_k, exp_v = kv_cache.kv_append(case.k_cache, case.v_cache, kn_h[reqs], vn_h[reqs], slots)
        return W.HostCase(case.q, exp_k, exp_v, case.block_table, case.context_lens, case.scale)

    print(f"[fused full-size] {name}: oracle over {B} requests", flush=True)
    ref = whole_tensor.oracle_reference(oracle_mod, wl, prepare=append_on_host)
    print(f"[fused full-size] {name}: GPU call", flush=True)
    apex.decode_attention_ex(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens, wl.scale,
                             out=wl.out, k_new=kn, v_new=vn)
    torch.cuda.synchronize()
    whole_tensor.assert_whole_tensor(wl.out.cpu().numpy(), ref, f"{name} fused")
    got_k = wl.k_cache[blk_d, :, pos_d, :]
    got_v = wl.v_cache[blk_d, :, pos_d, :]
    assert torch.equal(got_k.view(torch.int16), kn.view(torch.int16))
    assert torch.equal(got_v.view(torch.int16), vn.view(torch.int16))
    del wl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("workers", [0, 1, 3, 40])
def test_fused_append_checked_path_bad_current_block(torch_cuda, apex, oracle_mod, workers):
    """The checked path when the current token's own table entry is outside
    the pool: the error bit is set and nothing is stored; that block's cached
    tokens are skipped like any bad block, and the current token is still
    attended from the new rows.  Forced grids split the pairs, so the emit is
    also the last arriver's (40 work groups: about one unit each)."""
    torch = torch_cuda
    lens = [40, 17]
    G, Hkv = 4, 8
    case = W.make_host_case(lens, G * Hkv, Hkv, seed=151, poison=True)
    NB = case.k_cache.shape[0]
    rng = np.random.default_rng(152)
    kn = rng.standard_normal((2, Hkv, D)).astype(np.float16)
    vn = rng.standard_normal((2, Hkv, D)).astype(np.float16)
    bt = case.block_table.copy()
    bt[0, 2] = NB + 7                                 # request 0's current block (tokens 32..39)
    kc, vc = case.k_cache.copy(), case.v_cache.copy()
    s1 = int(bt[1, 1]) * BS + 0                       # request 1's current slot (position 16)
    kc[s1 // BS, :, s1 % BS, :] = np.float16(np.nan)
    vc[s1 // BS, :, s1 % BS, :] = np.float16(np.nan)
    exp_k, exp_v = kv_cache.kv_append(kc, vc, kn[1:], vn[1:], np.array([s1], dtype=np.int64))

    # expected: request 0 over tokens 0..31 plus the current token, placed in
    # an extra block at position 32; request 1 as usual
    k_ext = np.concatenate([exp_k, np.full((1, Hkv, BS, D), np.nan, dtype=np.float16)])
    v_ext = np.concatenate([exp_v, np.full((1, Hkv, BS, D), np.nan, dtype=np.float16)])
    k_ext[NB, :, 0, :] = kn[0]
    v_ext[NB, :, 0, :] = vn[0]
    bt_ext = case.block_table.copy()
    bt_ext[0, 2] = NB
    ref = oracle_mod.decode_attention_f64(case.q, k_ext, v_ext, bt_ext, np.array([33, 17], dtype=np.int32),
                                          case.scale)

    dev = "cuda"
    kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
    out = apex.decode_attention_ex(torch.from_numpy(case.q).to(dev), kd, vd, torch.from_numpy(bt).to(dev),
                                   torch.from_numpy(case.context_lens).to(dev), case.scale,
                                   check_inputs=True, num_workers=workers, k_new=torch.from_numpy(kn).to(dev),
                                   v_new=torch.from_numpy(vn).to(dev))
    torch.cuda.synchronize()
    assert apex.check_device_error() == apex.DEVICE_ERR_BLOCK_ID
    check(out.cpu().numpy(), ref, f"bad current block, workers={workers}")
    assert np.array_equal(kd.cpu().numpy().view(np.uint16), exp_k.view(np.uint16))
    assert np.array_equal(vd.cpu().numpy().view(np.uint16), exp_v.view(np.uint16))


@pytest.mark.parametrize("workers", [0, 1, 3])
def test_fused_append_checked_path_context_past_its_row(torch_cuda, apex, oracle_mod, workers):
    """The checked path when a context is longer than its explicit table row:
    the context is cut to the row's tokens, all of them cached, and the
    current token, whose position lies past the row, is attended from the new
    rows but not stored -- the row's last slot keeps its cached token."""
    torch = torch_cuda
    G, Hkv, stride = 4, 8, 4                          # rows of 4 blocks = 64 tokens
    lens = [40, 64, 17]
    case = W.make_host_case(lens, G * Hkv, Hkv, seed=161, poison=True, stride=stride)
    NB = case.k_cache.shape[0]
    rng = np.random.default_rng(162)
    B = len(lens)
    kn = rng.standard_normal((B, Hkv, D)).astype(np.float16)
    vn = rng.standard_normal((B, Hkv, D)).astype(np.float16)
    call_lens = np.array([41, 100, 18], dtype=np.int32)   # request 1: 100 > 64, cut to its row
    kc, vc = case.k_cache.copy(), case.v_cache.copy()
    slots = np.array([int(case.block_table[0, 40 // BS]) * BS + 40 % BS, -1,
                      int(case.block_table[2, 17 // BS]) * BS + 17 % BS], dtype=np.int64)
    for s in slots[slots >= 0]:
        kc[s // BS, :, s % BS, :] = np.float16(np.nan)
        vc[s // BS, :, s % BS, :] = np.float16(np.nan)
    exp_k, exp_v = kv_cache.kv_append(kc, vc, kn, vn, slots)   # request 1 stores nothing

    # expected: requests 0 and 2 as usual; request 1 over its 64 cached tokens
    # plus the current token, placed in an extra block at position 64
    k_ext = np.concatenate([exp_k, np.full((1, Hkv, BS, D), np.nan, dtype=np.float16)])
    v_ext = np.concatenate([exp_v, np.full((1, Hkv, BS, D), np.nan, dtype=np.float16)])
    k_ext[NB, :, 0, :] = kn[1]
    v_ext[NB, :, 0, :] = vn[1]
    bt_ext = np.concatenate([case.block_table, np.zeros((B, 1), dtype=np.int32)], axis=1)
    bt_ext[1, 4] = NB
    ref = oracle_mod.decode_attention_f64(case.q, k_ext, v_ext, bt_ext,
                                          np.array([41, 65, 18], dtype=np.int32), case.scale)

    dev = "cuda"
    kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
    assert apex.check_device_error() == 0
    out = apex.decode_attention_ex(torch.from_numpy(case.q).to(dev), kd, vd,
                                   torch.from_numpy(case.block_table).to(dev),
                                   torch.from_numpy(call_lens).to(dev), case.scale,
                                   block_table_stride=stride, num_workers=workers, check_inputs=True,
                                   k_new=torch.from_numpy(kn).to(dev), v_new=torch.from_numpy(vn).to(dev))
    torch.cuda.synchronize()
    assert apex.check_device_error() == apex.DEVICE_ERR_TABLE_ROW
    check(out.cpu().numpy(), ref, f"context past its row, workers={workers}")
    got_k, got_v = kd.cpu().numpy(), vd.cpu().numpy()
    last = int(case.block_table[1, 3])                # the row's last slot (position 63)
    assert np.array_equal(got_k[last, :, 15].view(np.uint16), kc[last, :, 15].view(np.uint16))
    assert np.array_equal(got_k.view(np.uint16), exp_k.view(np.uint16))
    assert np.array_equal(got_v.view(np.uint16), exp_v.view(np.uint16))


def test_fused_append_when_every_context_is_only_its_current_token_or_empty(torch_cuda, apex, oracle_mod):
    """Nothing cached at all: every request's output is its new V row (one
    token) or zeros (empty), and the new rows land in their slots."""
    torch = torch_cuda
    lens = [1, 0, 1, 1, 0]
    case, kc, vc, kn, vn, exp_k, exp_v = fused_case(lens, 4, 8, seed=171)
    dev = "cuda"
    kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
    for workers in (0, 2):
        out = apex.decode_attention_ex(torch.from_numpy(case.q).to(dev), kd, vd,
                                       torch.from_numpy(case.block_table).to(dev),
                                       torch.from_numpy(case.context_lens).to(dev), case.scale,
                                       num_workers=workers, k_new=torch.from_numpy(kn).to(dev),
                                       v_new=torch.from_numpy(vn).to(dev))
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        for b, L in enumerate(lens):
            if L == 1:
                assert np.array_equal(got[b].view(np.uint16), np.repeat(vn[b], 4, axis=0).view(np.uint16))
            else:
                assert np.all(got[b] == 0)
        assert np.array_equal(kd.cpu().numpy().view(np.uint16), exp_k.view(np.uint16))
        assert np.array_equal(vd.cpu().numpy().view(np.uint16), exp_v.view(np.uint16))


def test_fused_append_partition_32_and_64_bit_paths_agree(torch_cuda, apex, oracle_mod):
    """The fused build on both sides of the kernel's 32-bit partition bound
    (V (launched + 1) < 2^32, V = units on a forced grid).  255 requests of
    4109 tokens: the partition covers the 4108 cached ones, 257 blocks each,
    65535 units; 65536 work groups give 2^32 - 1 (32-bit), 65537 the 64-bit
    path, with the same 65535 workers, so the outputs must agree bit for bit.
    The first 256 blocks of every request repeat blocks of a shared pool; the
    last one, which receives the current token, is the request's own."""
    torch = torch_cuda
    B, L, G, Hkv, pool = 255, 257 * 16 - 3, 1, 1, 1024
    rng = np.random.default_rng(173)
    q = rng.standard_normal((B, G * Hkv, D)).astype(np.float16)
    kc = rng.standard_normal((pool + B, Hkv, BS, D)).astype(np.float16)
    vc = rng.standard_normal((pool + B, Hkv, BS, D)).astype(np.float16)
    table = np.empty((B, 257), dtype=np.int32)
    table[:, :256] = rng.integers(0, pool, size=(B, 256))
    table[:, 256] = pool + np.arange(B)
    lens = np.full(B, L, dtype=np.int32)
    kn = rng.standard_normal((B, Hkv, D)).astype(np.float16)
    vn = rng.standard_normal((B, Hkv, D)).astype(np.float16)
    slots = (pool + np.arange(B, dtype=np.int64)) * BS + (L - 1) % BS
    kc[pool:, :, (L - 1) % BS:, :] = np.float16(np.nan)     # the current slots and past them
    vc[pool:, :, (L - 1) % BS:, :] = np.float16(np.nan)
    exp_k, exp_v = kv_cache.kv_append(kc, vc, kn, vn, slots)
    assert (B * 257 * Hkv) * (65536 + 1) == 2**32 - 1
    ref = oracle_mod.decode_attention_f64(q, exp_k, exp_v, table, lens, W.SCALE)
    dev = "cuda"
    outs = {}
    for workers in (65536, 65537):
        kd, vd = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
        out = apex.decode_attention_ex(torch.from_numpy(q).to(dev), kd, vd, torch.from_numpy(table).to(dev),
                                       torch.from_numpy(lens).to(dev), W.SCALE, num_workers=workers,
                                       k_new=torch.from_numpy(kn).to(dev), v_new=torch.from_numpy(vn).to(dev))
        torch.cuda.synchronize()
        outs[workers] = out.cpu().numpy()
        check(outs[workers], ref, f"65535 units on {workers} work groups")
        assert np.array_equal(kd.cpu().numpy().view(np.uint16), exp_k.view(np.uint16))
        assert np.array_equal(vd.cpu().numpy().view(np.uint16), exp_v.view(np.uint16))
    assert np.array_equal(outs[65536].view(np.uint16), outs[65537].view(np.uint16))
