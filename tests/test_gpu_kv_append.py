"""GPU parity of the paged KV append (apex_kv_append) against its oracle.

Integer/byte work, so the bar is bit-exact: after the call both caches equal
the oracle's scatter (oracle/kv_cache.py) in every byte, including every slot
the call must leave alone.  The chained test then attends over the appended
caches and compares with the fp64 attention oracle to the attention bar.
"""
import numpy as np
import pytest

import apex_workloads as W
from oracle import kv_cache

pytestmark = pytest.mark.gpu


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


def run_append(torch, apex, c, stream=None):
    dev = "cuda"
    kc = torch.from_numpy(c.k_cache).to(dev)
    vc = torch.from_numpy(c.v_cache).to(dev)
    apex.kv_append(torch.from_numpy(c.k_new).to(dev), torch.from_numpy(c.v_new).to(dev), kc, vc,
                   torch.from_numpy(c.slot_mapping).to(dev), stream=stream)
    torch.cuda.synchronize()
    return kc.cpu().numpy(), vc.cpu().numpy()


def assert_bitwise(got, ref, what):
    g, r = got.view(np.uint16), ref.view(np.uint16)
    bad = int(np.count_nonzero(g != r))
    print(f"[append] {what}: {bad} differing elements of {g.size}", flush=True)
    assert bad == 0, what


CASES = [
    # T, NB, Hkv, d, bs, padding, out_of_range
    (1, 1, 1, 8, 1, 0, 0),
    (5, 2, 2, 8, 4, 1, 1),
    (33, 4, 2, 16, 16, 3, 2),
    (32, 64, 8, 128, 16, 0, 0),
    (64, 40, 32, 128, 16, 5, 5),
    (300, 50, 8, 128, 16, 17, 0),
    (257, 30, 3, 24, 16, 0, 7),      # d / 8 does not divide 256
    (1000, 70, 1, 2048, 16, 10, 10),  # widest row
    (77, 9, 8, 64, 32, 0, 0),
]


@pytest.mark.parametrize("T,NB,Hkv,d,bs,pad,oor", CASES)
def test_small_cases_bitwise(torch_cuda, apex, T, NB, Hkv, d, bs, pad, oor):
    c = W.make_append_case(T, NB, Hkv, d, bs, seed=T + 31 * d, padding=pad, out_of_range=oor)
    print(f"[append] T={T} NB={NB} Hkv={Hkv} d={d} bs={bs}", flush=True)
    gk, gv = run_append(torch_cuda, apex, c)
    rk, rv = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    assert_bitwise(gk, rk, "k")
    assert_bitwise(gv, rv, "v")


def test_fused_projection_views_and_side_stream(torch_cuda, apex):
    torch = torch_cuda
    T, Hq, Hkv, d, NB = 48, 32, 8, 128, 12
    c = W.make_append_case(T, NB, Hkv, d, 16, seed=5, padding=2)
    rng = np.random.default_rng(6)
    fused = rng.standard_normal((T, Hq + 2 * Hkv, d)).astype(np.float16)
    fused[:, Hq:Hq + Hkv] = c.k_new
    fused[:, Hq + Hkv:] = c.v_new
    dev = "cuda"
    f = torch.from_numpy(fused).to(dev)
    kc = torch.from_numpy(c.k_cache).to(dev)
    vc = torch.from_numpy(c.v_cache).to(dev)
    slots = torch.from_numpy(c.slot_mapping).to(dev)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        apex.kv_append(f[:, Hq:Hq + Hkv], f[:, Hq + Hkv:], kc, vc, slots, stream=s)
    s.synchronize()
    rk, rv = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    assert_bitwise(kc.cpu().numpy(), rk, "k (fused view)")
    assert_bitwise(vc.cpu().numpy(), rv, "v (fused view)")


def test_empty_call_changes_nothing(torch_cuda, apex):
    torch = torch_cuda
    c = W.make_append_case(4, 3, 2, 128, 16, seed=8)
    kc = torch.from_numpy(c.k_cache).cuda()
    vc = torch.from_numpy(c.v_cache).cuda()
    e = torch.empty((0, 2, 128), dtype=torch.float16, device="cuda")
    apex.kv_append(e, e, kc, vc, torch.empty(0, dtype=torch.int64, device="cuda"))
    torch.cuda.synchronize()
    assert_bitwise(kc.cpu().numpy(), c.k_cache, "k")
    assert_bitwise(vc.cpu().numpy(), c.v_cache, "v")


@pytest.mark.parametrize("lens,Hq,Hkv", [([1, 16, 17, 200, 511, 0], 32, 8), ([33, 64, 2], 32, 32)])
def test_append_then_attend_matches_the_oracles(torch_cuda, apex, oracle_mod, lens, Hq, Hkv):
    torch = torch_cuda
    case = W.make_host_case(lens, Hq, Hkv, seed=sum(lens), poison=True)
    slots = W.append_slots(case.layout)
    rng = np.random.default_rng(12)
    B = len(lens)
    kn = rng.standard_normal((B, Hkv, 128)).astype(np.float16)
    vn = rng.standard_normal((B, Hkv, 128)).astype(np.float16)
    dev = "cuda"
    kc = torch.from_numpy(case.k_cache).to(dev)
    vc = torch.from_numpy(case.v_cache).to(dev)
    apex.kv_append(torch.from_numpy(kn).to(dev), torch.from_numpy(vn).to(dev), kc, vc,
                   torch.from_numpy(slots).to(dev))
    out = apex.decode_attention(torch.from_numpy(case.q).to(dev), kc, vc,
                                torch.from_numpy(case.block_table).to(dev),
                                torch.from_numpy(case.context_lens).to(dev), case.scale)
    torch.cuda.synchronize()
    rk, rv = kv_cache.kv_append(case.k_cache, case.v_cache, kn, vn, slots)
    assert_bitwise(kc.cpu().numpy(), rk, "k")
    assert_bitwise(vc.cpu().numpy(), rv, "v")
    ref = oracle_mod.decode_attention_f64(case.q, rk, rv, case.block_table, case.context_lens,
                                          case.scale)
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    err = float(np.abs(got - ref).max())
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    print(f"[append+attend] max_abs={err:.3e} rel_l2={rel:.3e}", flush=True)
    assert err <= 2e-3 and rel <= 1e-3


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_full_size_decode_step_append(torch_cuda, apex, name):
    """Append each request's newest token at position L_b - 1 into the
    workload's full cache, in the configuration the benchmark times."""
    torch = torch_cuda
    wl = W.DeviceWorkload(name)
    cfg = wl.cfg
    slots = W.append_slots(wl.layout)
    rng = np.random.default_rng(21)
    kn = rng.standard_normal((cfg.B, cfg.Hkv, cfg.d)).astype(np.float16)
    vn = rng.standard_normal((cfg.B, cfg.Hkv, cfg.d)).astype(np.float16)
    # only the blocks holding the new tokens can change: check those bitwise,
    # and a checksum of the whole pool for everything else
    blocks = np.unique(slots[slots >= 0] // cfg.block_size)
    idx = torch.from_numpy(blocks).cuda()
    before_k = wl.k_cache.index_select(0, idx).cpu().numpy()
    before_v = wl.v_cache.index_select(0, idx).cpu().numpy()
    sum_k = wl.k_cache.view(torch.int16).to(torch.int64).sum()
    sum_v = wl.v_cache.view(torch.int16).to(torch.int64).sum()
    apex.kv_append(torch.from_numpy(kn).cuda(), torch.from_numpy(vn).cuda(), wl.k_cache,
                   wl.v_cache, torch.from_numpy(slots).cuda())
    torch.cuda.synchronize()
    remap = {int(b): i for i, b in enumerate(blocks)}
    local = np.array([remap[int(s) // cfg.block_size] * cfg.block_size + int(s) % cfg.block_size
                      for s in slots], dtype=np.int64)
    rk, rv = kv_cache.kv_append(before_k, before_v, kn, vn, local)
    assert_bitwise(wl.k_cache.index_select(0, idx).cpu().numpy(), rk, f"{name} k blocks")
    assert_bitwise(wl.v_cache.index_select(0, idx).cpu().numpy(), rv, f"{name} v blocks")
    dk = int((wl.k_cache.view(torch.int16).to(torch.int64).sum() - sum_k).item())
    dv = int((wl.v_cache.view(torch.int16).to(torch.int64).sum() - sum_v).item())
    assert dk == int(rk.view(np.int16).astype(np.int64).sum() - before_k.view(np.int16).astype(np.int64).sum())
    assert dv == int(rv.view(np.int16).astype(np.int64).sum() - before_v.view(np.int16).astype(np.int64).sum())


def test_bulk_append_bitwise(torch_cuda, apex):
    """A prompt-sized append (the launch shape the benchmark's bulk line
    times): 65536 tokens x 8 kv-heads into a 5000-block pool."""
    T, NB, Hkv = 65536, 5000, 8
    c = W.make_append_case(T, NB, Hkv, 128, 16, seed=77, padding=100, out_of_range=100)
    gk, gv = run_append(torch_cuda, apex, c)
    rk, rv = kv_cache.kv_append(c.k_cache, c.v_cache, c.k_new, c.v_new, c.slot_mapping)
    assert_bitwise(gk, rk, "bulk k")
    assert_bitwise(gv, rv, "bulk v")
