"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Bar (fp16 outputs, fp32 accumulation): every output finite, max-abs error
<= 2e-3 and relative L2 error <= 1e-3 against the unrounded fp64 oracle.
Small cases are compared element by element; the full-size workloads run in
the launch configuration the benchmark times and are compared over the whole
output tensor (the oracle runs over every request, chunk by chunk).
"""
import numpy as np
import pytest

import apex_workloads as W
import whole_tensor

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3


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


def to_dev(torch, case):
    dev = "cuda"
    return (torch.from_numpy(case.q).to(dev), torch.from_numpy(case.k_cache).to(dev),
            torch.from_numpy(case.v_cache).to(dev), torch.from_numpy(case.block_table).to(dev),
            torch.from_numpy(case.context_lens).to(dev))


def run_gpu(torch, apex, case, **kw):
    q, k, v, bt, lens = to_dev(torch, case)
    if kw:
        out = apex.decode_attention_ex(q, k, v, bt, lens, case.scale, **kw)
    else:
        out = apex.decode_attention(q, k, v, bt, lens, case.scale)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def assert_parity(got, ref, what=""):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite outputs"
    err = np.abs(got - ref)
    max_abs = float(err.max()) if err.size else 0.0
    nrm = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(got - ref)) / nrm if nrm > 0 else float(np.linalg.norm(got))
    print(f"[parity] {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e}", flush=True)
    assert max_abs <= MAX_ABS, f"{what}: max-abs {max_abs:.3e}"
    assert rel <= REL_L2, f"{what}: rel-L2 {rel:.3e}"


# ---------------------------------------------------------------------------
# small cases, element by element
# ---------------------------------------------------------------------------

def test_c1_tiny_mha_full_parity(torch_cuda, apex, oracle_mod):
    torch = torch_cuda
    wl = W.DeviceWorkload("c1", device="cpu").to("cuda")
    out = apex.decode_attention(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                                wl.scale)
    torch.cuda.synchronize()
    ref = oracle_mod.decode_attention_f64(wl.q.cpu().numpy(), wl.k_cache.cpu().numpy(),
                                          wl.v_cache.cpu().numpy(), wl.block_table.cpu().numpy(),
                                          wl.context_lens.cpu().numpy(), wl.scale)
    assert_parity(out.cpu().numpy(), ref, "c1")


SMALL = [
    # name, lens, Hq, Hkv
    ("mha_ragged", [1, 15, 16, 17, 100, 511], 8, 8),
    ("g2_ragged", [33, 0, 250, 64, 7], 8, 4),
    ("g4_ragged", [1, 2, 31, 32, 33, 1000, 3001], 16, 4),
    ("g8_ragged", [5, 129, 700], 16, 2),
    ("g4_long", [9000, 40, 2500], 32, 8),
    ("mha_many", list(range(1, 400, 37)), 4, 4),
]


@pytest.mark.parametrize("name,lens,Hq,Hkv", SMALL, ids=[s[0] for s in SMALL])
@pytest.mark.parametrize("workers", [0, 1, 2, 7, 64, 100000])
def test_small_cases_with_poison(torch_cuda, apex, oracle_mod, name, lens, Hq, Hkv, workers):
    case = W.make_host_case(lens, Hq, Hkv, seed=len(lens) * 31 + Hq, poison=True)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    got = run_gpu(torch_cuda, apex, case, num_workers=workers)
    assert_parity(got, ref, f"{name} workers={workers}")
    for b, L in enumerate(lens):
        if L == 0:
            assert np.all(got[b] == 0)


def test_lse_output(torch_cuda, apex, oracle_mod):
    torch = torch_cuda
    case = W.make_host_case([1, 70, 0, 3000], 16, 4, seed=77)
    _, lse_ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache,
                                                 case.block_table, case.context_lens, case.scale,
                                                 return_lse=True)
    for workers in (0, 1, 5, 3000):
        lse = torch.empty((4, 16), dtype=torch.float32, device="cuda")
        run_gpu(torch, apex, case, num_workers=workers, lse_out=lse)
        got = lse.cpu().numpy().astype(np.float64)
        assert np.all(np.isneginf(got[2]))
        fin = np.isfinite(lse_ref)
        assert np.max(np.abs(got[fin] - lse_ref[fin])) < 1e-4


def test_wide_block_table_stride(torch_cuda, apex, oracle_mod):
    case = W.make_host_case([40, 300, 17], 8, 2, seed=5, stride=64)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    got = run_gpu(torch_cuda, apex, case, block_table_stride=64)
    assert_parity(got, ref, "stride=64")


def test_binding_refuses_tensors_the_library_would_misread(torch_cuda, apex):
    """Checked in the binding before any launch: nothing runs on the GPU."""
    torch = torch_cuda
    case = W.make_host_case([40, 300, 17], 8, 2, seed=5, stride=64)
    q, k, v, bt, lens = to_dev(torch, case)
    s = case.scale
    with pytest.raises(TypeError, match="q must be"):
        apex.decode_attention(q.float(), k, v, bt, lens, s)
    with pytest.raises(TypeError, match="context_lens must be"):
        apex.decode_attention(q, k, v, bt, lens.long(), s)
    with pytest.raises(ValueError, match="block_table must be on"):
        apex.decode_attention(q, k, v, bt.cpu(), lens, s)
    with pytest.raises(ValueError, match="k_cache must be contiguous"):
        apex.decode_attention(q, k.transpose(2, 3).contiguous().transpose(2, 3), v, bt, lens, s)
    with pytest.raises(ValueError, match="v_cache must have shape"):
        apex.decode_attention(q, k, v[:-1], bt, lens, s)
    with pytest.raises(ValueError, match="out must have shape"):
        apex.decode_attention(q, k, v, bt, lens, s, out=torch.empty_like(q)[:2])
    with pytest.raises(ValueError, match="block_table_stride says 32"):
        apex.decode_attention_ex(q, k, v, bt, lens, s, block_table_stride=32)
    with pytest.raises(TypeError, match="lse_out must be"):
        apex.decode_attention_ex(q, k, v, bt, lens, s, block_table_stride=64,
                                 lse_out=torch.empty((3, 8), dtype=torch.float16, device="cuda"))
    kn = torch.zeros((3, 2, 128), dtype=torch.float16, device="cuda")
    with pytest.raises(TypeError, match="slot_mapping must be"):
        apex.kv_append(kn, kn.clone(), k, v, torch.zeros(3, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()


def test_caller_workspace_and_side_stream(torch_cuda, apex, oracle_mod):
    torch = torch_cuda
    case = W.make_host_case([500, 5, 2000], 32, 8, seed=6)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    q, k, v, bt, lens = to_dev(torch, case)
    nbytes = apex.workspace_bytes(3, 32, 8)
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = apex.decode_attention_ex(q, k, v, bt, lens, case.scale, workspace=ws, stream=s)
    s.synchronize()
    assert_parity(out.cpu().numpy(), ref, "caller workspace, side stream")
    cb = apex.counter_bytes(3, 8)
    assert int(ws[:cb].abs().sum()) == 0          # counters left at zero
    # a forced small grid shares pairs between work groups; counters still return to zero
    ws2 = torch.zeros(apex.workspace_bytes(3, 32, 8, num_workers=40), dtype=torch.uint8, device="cuda")
    for _ in range(3):
        out = apex.decode_attention_ex(q, k, v, bt, lens, case.scale, workspace=ws2, num_workers=40)
        torch.cuda.synchronize()
        assert_parity(out.cpu().numpy(), ref, "caller workspace, 40 workers")
        assert int(ws2[:cb].abs().sum()) == 0
    small = torch.empty(256, dtype=torch.uint8, device="cuda")
    with pytest.raises(apex.ApexError) as e:
        apex.decode_attention_ex(q, k, v, bt, lens, case.scale, workspace=small)
    assert e.value.code == apex.APEX_ERR_OUT_OF_MEMORY


# ---------------------------------------------------------------------------
# invariants on the GPU path
# ---------------------------------------------------------------------------

def test_single_token_returns_v_bitwise(torch_cuda, apex):
    case = W.make_host_case([1, 1, 1, 1], 32, 8, seed=8, poison=True)
    got = run_gpu(torch_cuda, apex, case)
    for b in range(4):
        blk = case.block_table[b, 0]
        exp = np.repeat(case.v_cache[blk, :, 0], 4, axis=0)
        assert np.array_equal(got[b].astype(np.float16), exp)


def test_identical_keys_give_mean_of_v(torch_cuda, apex):
    case = W.make_host_case([3, 77, 1200], 32, 8, seed=9)
    key = np.random.default_rng(1).standard_normal((8, 128)).astype(np.float16)
    case.k_cache[:] = key[None, :, None, :]
    got = run_gpu(torch_cuda, apex, case)
    from oracle import brute_force
    for b, L in enumerate(case.context_lens):
        V = brute_force.dense_kv(case.v_cache, case.block_table, b, int(L))
        mean = np.repeat(V.mean(axis=1), 4, axis=0)
        assert np.max(np.abs(got[b] - mean)) <= MAX_ABS


def test_unit_values_give_unit_output(torch_cuda, apex):
    case = W.make_host_case([1, 50, 5000], 32, 8, seed=10)
    case.v_cache[:] = 1
    for workers in (0, 3, 777):
        got = run_gpu(torch_cuda, apex, case, num_workers=workers)
        assert np.all(got == 1.0)


def test_block_permutation_is_bitwise_invariant(torch_cuda, apex):
    case = W.make_host_case([100, 1, 2048, 333], 32, 8, seed=11, slack_blocks=5)
    base = run_gpu(torch_cuda, apex, case)
    perm = np.random.default_rng(2).permutation(case.k_cache.shape[0])
    k2 = np.empty_like(case.k_cache)
    v2 = np.empty_like(case.v_cache)
    k2[perm] = case.k_cache
    v2[perm] = case.v_cache
    case.k_cache, case.v_cache = k2, v2
    case.block_table = perm[case.block_table].astype(np.int32)
    assert np.array_equal(run_gpu(torch_cuda, apex, case), base)


def test_gqa_matches_mha_with_repeated_kv(torch_cuda, apex):
    case = W.make_host_case([64, 900, 3], 32, 8, seed=12)
    gqa = run_gpu(torch_cuda, apex, case)
    case.k_cache = np.ascontiguousarray(np.repeat(case.k_cache, 4, axis=1))
    case.v_cache = np.ascontiguousarray(np.repeat(case.v_cache, 4, axis=1))
    mha = run_gpu(torch_cuda, apex, case)
    assert np.max(np.abs(gqa.astype(np.float64) - mha)) <= 1e-3


def test_late_peaked_key_dominates(torch_cuda, apex, oracle_mod):
    case = W.make_host_case([4000], 4, 1, seed=13)
    q = case.q[0, 0].astype(np.float64)
    t = 3990
    blk = case.block_table[0, t // 16]
    case.k_cache[blk, 0, t % 16] = (40.0 * q / np.linalg.norm(q)).astype(np.float16)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    for workers in (0, 1, 9, 250):
        assert_parity(run_gpu(torch_cuda, apex, case, num_workers=workers), ref, f"peaked workers={workers}")


def test_repeated_runs_are_bitwise_identical(torch_cuda, apex):
    case = W.make_host_case([3000, 17, 900, 4500], 32, 8, seed=14)
    a = run_gpu(torch_cuda, apex, case)
    b = run_gpu(torch_cuda, apex, case)
    assert np.array_equal(a, b)


# ---------------------------------------------------------------------------
# full-size workloads, every request, in the benchmark's launch configuration
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_size_whole_tensor_parity(torch_cuda, apex, oracle_mod, name):
    """The call the benchmark times (default grid, library workspace) over the
    whole workload, against the fp64 oracle over every request: max-abs and
    relative L2 over the whole [B][Hq][d] output."""
    torch = torch_cuda
    print(f"[full-size] generating {name}", flush=True)
    wl = W.DeviceWorkload(name)
    print(f"[full-size] {name}: oracle over {wl.cfg.B} requests", flush=True)
    ref = whole_tensor.oracle_reference(oracle_mod, wl)
    print(f"[full-size] {name}: GPU call", flush=True)
    apex.decode_attention(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                          wl.scale, out=wl.out)
    torch.cuda.synchronize()
    whole_tensor.assert_whole_tensor(wl.out.cpu().numpy(), ref, name)
    del wl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["g8", "g2"])
def test_full_size_whole_tensor_parity_other_group_sizes(torch_cuda, apex, oracle_mod, name):
    """The two group sizes the five workloads do not use, at full size and in
    the benchmark's launch configuration: G = 8 (Llama-3-70B heads) with the
    long-output lengths, G = 2 with the GQA decode lengths; whole tensor."""
    torch = torch_cuda
    print(f"[full-size] generating {name}", flush=True)
    wl = W.DeviceWorkload(name)
    ref = whole_tensor.oracle_reference(oracle_mod, wl)
    apex.decode_attention(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                          wl.scale, out=wl.out)
    torch.cuda.synchronize()
    whole_tensor.assert_whole_tensor(wl.out.cpu().numpy(), ref, name)
    del wl
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# batches past the lengths the kernel keeps in LDS (2048 requests), and one
# request split over ~100 work groups (combine in several chunks of 8)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("B", [2048, 2049, 5000])
def test_large_batches_read_lengths_from_memory(torch_cuda, apex, oracle_mod, B):
    rng = np.random.default_rng(B)
    lens = rng.integers(0, 48, size=B)
    lens[rng.random(B) < 0.2] = 0
    case = W.make_host_case(lens, 8, 2, seed=B, poison=True)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    for workers in (0, 3):
        got = run_gpu(torch_cuda, apex, case, num_workers=workers)
        assert_parity(got, ref, f"B={B} workers={workers}")
        assert np.all(got[lens == 0] == 0)


def test_one_long_request_split_over_many_work_groups(torch_cuda, apex, oracle_mod):
    torch = torch_cuda
    case = W.make_host_case([65536], 32, 8, seed=65, poison=True)
    ref, lse_ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache,
                                                   case.block_table, case.context_lens, case.scale,
                                                   return_lse=True)
    plan = apex.plan_host(case.context_lens, 8, 768)
    print(f"[parity] contributors per pair: {plan['contributors'].ravel().tolist()}", flush=True)
    assert plan["contributors"].min() > 8          # more than one combine chunk
    lse = torch.empty((1, 32), dtype=torch.float32, device="cuda")
    got = run_gpu(torch, apex, case, num_workers=768, lse_out=lse)
    assert_parity(got, ref, "L=65536")
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) < 1e-4
    # the default grid (equal-cost ranges, one work group per CU here): 32
    # contributors per pair, combined in four chunks
    plan = apex.plan_host(case.context_lens, 8, 512, cus=256)
    assert plan["contributors"].min() > 8
    got = run_gpu(torch, apex, case, lse_out=lse)
    assert_parity(got, ref, "L=65536, default grid")
    assert np.max(np.abs(lse.cpu().numpy() - lse_ref)) < 1e-4


# ---------------------------------------------------------------------------
# the partition's 32-bit and 64-bit arithmetic.  The kernel partitions in 32
# bits when V (launched + 1) < 2^32 (V = units on a forced grid) and in 64
# bits otherwise; forced grids of up to 2^17 work groups put cases on both
# sides of that bound, and past 2^32 in the range-end products.  The table
# entries repeat blocks of a small pool, so a large unit count takes little
# memory.
# ---------------------------------------------------------------------------

def shared_pool_case(B, L, Hq, Hkv, pool, seed):
    rng = np.random.default_rng(seed)
    nb = -(-L // W.BLOCK_SIZE)
    q = rng.standard_normal((B, Hq, W.D_HEAD)).astype(np.float16)
    k = rng.standard_normal((pool, Hkv, W.BLOCK_SIZE, W.D_HEAD)).astype(np.float16)
    v = rng.standard_normal((pool, Hkv, W.BLOCK_SIZE, W.D_HEAD)).astype(np.float16)
    table = rng.integers(0, pool, size=(B, nb), dtype=np.int32)
    return W.HostCase(q, k, v, table, np.full(B, L, dtype=np.int32), W.SCALE)


def test_partition_64_bit_path_with_range_products_past_2_32(torch_cuda, apex, oracle_mod):
    # 8 requests x 8 kv-heads x 2048 blocks = 2^17 units on 2^17 work groups:
    # V (launched + 1) ~ 2^34, and w V reaches ~2^34; 2048 contributors per pair
    case = shared_pool_case(8, 2048 * 16 - 5, 8, 8, 1024, seed=171)
    units = 8 * 8 * 2048
    assert units * (units + 1) > 2**32
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    got = run_gpu(torch_cuda, apex, case, num_workers=units)
    assert_parity(got, ref, "2^17 units on 2^17 work groups (64-bit partition)")


def test_partition_32_and_64_bit_paths_agree_at_the_bound(torch_cuda, apex, oracle_mod):
    # 255 requests x 257 blocks = 65535 units (one kv-head): on 65536 work
    # groups V (launched + 1) = 2^32 - 1, the largest 32-bit case; on 65537 it
    # is 2^32 + 65534 (64-bit).  Both use 65535 workers, so their ranges, and
    # hence their outputs, must be the same bit for bit.
    case = shared_pool_case(255, 257 * 16 - 3, 1, 1, 1024, seed=172)
    units = 255 * 257
    assert units * (65536 + 1) == 2**32 - 1 and units * (65537 + 1) > 2**32 - 1
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    narrow = run_gpu(torch_cuda, apex, case, num_workers=65536)
    wide = run_gpu(torch_cuda, apex, case, num_workers=65537)
    assert_parity(narrow, ref, "65535 units, 32-bit partition")
    assert_parity(wide, ref, "65535 units, 64-bit partition")
    assert np.array_equal(narrow.view(np.uint16), wide.view(np.uint16))
    # the checked build shares the prologue: the same outputs on both paths
    for workers in (65536, 65537):
        got = run_gpu(torch_cuda, apex, case, num_workers=workers, check_inputs=True)
        assert np.array_equal(got.view(np.uint16), narrow.view(np.uint16)), f"checked, {workers}"
        assert apex.check_device_error() == 0


# ---------------------------------------------------------------------------
# the longest context an int32 length allows, 2^31 - 1 tokens (2^27 blocks):
# the table repeats block 0 and ends on block 1, whose slot 15 (past the
# context) holds NaN.  Expected values from the multiset form
# (tests/multiset_attention.py, checked against the oracle on the CPU).
# ---------------------------------------------------------------------------

def test_longest_context_int32(torch_cuda, apex):
    import multiset_attention as MS
    torch = torch_cuda
    L = 2**31 - 1
    nb = -(-L // W.BLOCK_SIZE)
    assert nb == 2**27 and L - W.BLOCK_SIZE * (nb - 1) == 15
    G, Hkv = 4, 1
    rng = np.random.default_rng(2**31 % 1000)
    q = rng.standard_normal((1, G * Hkv, W.D_HEAD)).astype(np.float16)
    k = rng.standard_normal((2, Hkv, W.BLOCK_SIZE, W.D_HEAD)).astype(np.float16)
    v = rng.standard_normal((2, Hkv, W.BLOCK_SIZE, W.D_HEAD)).astype(np.float16)
    k[1, :, 15, :] = np.float16(np.nan)
    v[1, :, 15, :] = np.float16(np.nan)
    table = np.zeros((1, nb), dtype=np.int32)
    table[0, -1] = 1
    ref = MS.multiset_attention(q[0], k, v, table[0], L, W.SCALE)[None]
    dev = "cuda"
    qd, kd, vd = (torch.from_numpy(x).to(dev) for x in (q, k, v))
    bt = torch.from_numpy(table).to(dev)
    cl = torch.tensor([L], dtype=torch.int32, device=dev)
    # Every wave sums its blocks in fp32; with one block repeated, the rounding
    # of those sums does not average out and grows with the blocks per wave:
    # 2^16 on the default grid (512 work groups here), 2^15 on 1024.  (A
    # forced grid of 256 takes 2^17 per wave and leaves the bar: rel-L2
    # about 1.5e-3.)
    for workers in (0, 1024):
        out = apex.decode_attention_ex(qd, kd, vd, bt, cl, W.SCALE, num_workers=workers)
        torch.cuda.synchronize()
        assert_parity(out.cpu().numpy(), ref, f"L = 2^31 - 1, workers={workers}")
    # the fused append: 2^31 - 2 cached tokens and the current one, stored at
    # slot 14 of block 1
    kn = rng.standard_normal((1, Hkv, W.D_HEAD)).astype(np.float16)
    vn = rng.standard_normal((1, Hkv, W.D_HEAD)).astype(np.float16)
    k_exp, v_exp = k.copy(), v.copy()
    k_exp[1, :, 14, :] = kn[0]
    v_exp[1, :, 14, :] = vn[0]
    ref = MS.multiset_attention(q[0], k_exp, v_exp, table[0], L, W.SCALE)[None]
    k_in, v_in = k.copy(), v.copy()
    k_in[1, :, 14, :] = np.float16(np.nan)
    v_in[1, :, 14, :] = np.float16(np.nan)
    kd, vd = torch.from_numpy(k_in).to(dev), torch.from_numpy(v_in).to(dev)
    out = apex.decode_attention_ex(qd, kd, vd, bt, cl, W.SCALE, k_new=torch.from_numpy(kn).to(dev),
                                   v_new=torch.from_numpy(vn).to(dev))
    torch.cuda.synchronize()
    assert_parity(out.cpu().numpy(), ref, "L = 2^31 - 1, fused append")
    assert np.array_equal(kd.cpu().numpy().view(np.uint16), k_exp.view(np.uint16))
    assert np.array_equal(vd.cpu().numpy().view(np.uint16), v_exp.view(np.uint16))


# ---------------------------------------------------------------------------
# input check (APEX_DECODE_FLAG_CHECK_INPUTS)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name,lens,Hq,Hkv", SMALL[:4], ids=[s[0] for s in SMALL[:4]])
def test_checked_path_matches_default_path_bitwise(torch_cuda, apex, name, lens, Hq, Hkv):
    case = W.make_host_case(lens, Hq, Hkv, seed=len(lens) * 17 + Hq, poison=True)
    for workers in (0, 5):
        plain = run_gpu(torch_cuda, apex, case, num_workers=workers)
        checked = run_gpu(torch_cuda, apex, case, num_workers=workers, check_inputs=True)
        assert np.array_equal(plain.view(np.uint16), checked.view(np.uint16)), name
    assert apex.check_device_error() == 0


def test_checked_path_skips_block_ids_outside_the_pool(torch_cuda, apex, oracle_mod):
    case = W.make_host_case([40, 300, 17, 33], 32, 8, seed=90, poison=True)
    nb = case.k_cache.shape[0]
    bt = case.block_table.copy()
    bt[0, 1] = nb + 3            # a middle block: tokens 16..31 of request 0
    bt[1, 18] = -1               # the last block of request 1 (tokens 288..299)
    bt[3, 2] = 2 ** 31 - 1       # the last block of request 3 (token 32)
    bad = W.HostCase(case.q, case.k_cache, case.v_cache, bt, case.context_lens, case.scale)
    assert apex.check_device_error() == 0
    for workers in (0, 7, 1000):
        got = run_gpu(torch_cuda, apex, bad, num_workers=workers, check_inputs=True)
        assert apex.check_device_error() == apex.DEVICE_ERR_BLOCK_ID
        # expected: the same attention with the bad blocks' tokens absent
        exp_bt = case.block_table.copy()
        exp_lens = case.context_lens.copy()
        exp_bt[0, 1] = case.block_table[0, 2]      # tokens 32..39 move up to 16..23
        exp_lens[0] = 24
        exp_lens[1] = 288
        exp_lens[3] = 32
        ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, exp_bt, exp_lens,
                                              case.scale)
        assert_parity(got, ref, f"bad ids skipped, workers={workers}")
    assert apex.check_device_error() == 0            # reading cleared the word


def test_checked_path_cuts_a_context_to_its_table_row(torch_cuda, apex, oracle_mod):
    case = W.make_host_case([40, 64], 16, 4, seed=91, poison=True, stride=4)
    lens = case.context_lens.copy()
    lens[1] = 100                 # longer than the 4-block row
    longer = W.HostCase(case.q, case.k_cache, case.v_cache, case.block_table, lens, case.scale)
    got = run_gpu(torch_cuda, apex, longer, block_table_stride=4, check_inputs=True)
    assert apex.check_device_error() == apex.DEVICE_ERR_TABLE_ROW
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    assert_parity(got, ref, "context cut to the row")


# ---------------------------------------------------------------------------
# the waves' K/V pipelines run on from segment to segment: when a segment and
# the next both span >= 16 blocks, the next one's first two blocks per wave
# (its blocks 0..7) are loaded during the current one's last steps
# ---------------------------------------------------------------------------

CHAIN_LENS = [15 * 16, 16 * 16, 17 * 16, 16 * 16 - 5, 33 * 16, 4 * 16, 64 * 16 + 3, 16 * 16, 1, 0, 31 * 16]


@pytest.mark.parametrize("workers", [1, 2, 3, 5, 0])
def test_segments_around_the_prefetch_length(torch_cuda, apex, oracle_mod, workers):
    """Whole pairs of 15, 16 and 17 blocks back to back on one work group
    (workers = 1: every transition is a prefetch decision), and splits of the
    same batch at arbitrary points (workers = 2, 3, 5) and the default grid."""
    case = W.make_host_case(CHAIN_LENS, 8, 2, seed=95, poison=True)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    got = run_gpu(torch_cuda, apex, case, num_workers=workers)
    assert_parity(got, ref, f"chained segments, workers={workers}")


def drop_blocks(row, L, bad):
    """Table row and length of the same request with the blocks at positions
    `bad` removed (their tokens take no part; later blocks move up)."""
    nb = -(-L // 16)
    keep = [p for p in range(nb) if p not in bad]
    toks = sum(min(16, L - 16 * p) for p in keep)
    out = np.zeros_like(row)
    out[:len(keep)] = row[keep]
    return out, toks


@pytest.mark.parametrize("workers", [1, 3, 0])
def test_checked_path_bad_ids_at_prefetched_blocks(torch_cuda, apex, oracle_mod, workers):
    """Block ids outside the pool at the positions the previous segment
    prefetches (each wave's first two blocks: positions 0..7 of a segment)."""
    lens = [40 * 16, 20 * 16 + 7, 16 * 16, 33 * 16]
    case = W.make_host_case(lens, 8, 2, seed=96, poison=True)
    nb = case.k_cache.shape[0]
    bad = {0: [0, 5], 1: [1, 20], 2: [7], 3: [0, 1, 2, 3]}
    bt = case.block_table.copy()
    for b, ps in bad.items():
        for p in ps:
            bt[b, p] = nb + 11 * (p + 1)
    bad_case = W.HostCase(case.q, case.k_cache, case.v_cache, bt, case.context_lens, case.scale)
    exp_bt = case.block_table.copy()
    exp_lens = case.context_lens.copy()
    for b, ps in bad.items():
        exp_bt[b], exp_lens[b] = drop_blocks(case.block_table[b], int(lens[b]), set(ps))
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, exp_bt, exp_lens,
                                          case.scale)
    got = run_gpu(torch_cuda, apex, bad_case, num_workers=workers, check_inputs=True)
    assert apex.check_device_error() == apex.DEVICE_ERR_BLOCK_ID
    assert_parity(got, ref, f"bad ids at prefetched blocks, workers={workers}")


# ---------------------------------------------------------------------------
# seeded random sweep: group sizes, length mixes (empty, one token, block
# boundaries, long), table strides, worker counts and the checked path
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(12))
def test_random_configurations(torch_cuda, apex, oracle_mod, seed):
    rng = np.random.default_rng(1000 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    B = int(rng.integers(1, 40))
    kinds = rng.choice(["short", "edge", "long", "zero"], size=B, p=[0.4, 0.3, 0.2, 0.1])
    lens = []
    for k in kinds:
        if k == "short":
            lens.append(int(rng.integers(1, 64)))
        elif k == "edge":
            lens.append(int(16 * rng.integers(1, 40) + rng.choice([-1, 0, 1])))
        elif k == "long":
            lens.append(int(rng.integers(1000, 6000)))
        else:
            lens.append(0)
    maxb = max([1] + [-(-L // 16) for L in lens])
    stride = int(maxb + rng.integers(0, 5)) if rng.random() < 0.4 else None
    case = W.make_host_case(lens, G * Hkv, Hkv, seed=seed, poison=True, stride=stride)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    workers = int(rng.choice([0, 0, 1, 13, 300]))
    kw = dict(num_workers=workers)
    if stride is not None:
        kw["block_table_stride"] = stride
    if rng.random() < 0.3:
        kw["check_inputs"] = True
    print(f"[parity] seed={seed} G={G} Hkv={Hkv} B={B} stride={stride} {kw}", flush=True)
    got = run_gpu(torch_cuda, apex, case, **kw)
    assert_parity(got, ref, f"random seed={seed}")
    assert np.all(got[np.asarray(lens) == 0] == 0)
    if kw.get("check_inputs"):
        assert apex.check_device_error() == 0


# ---------------------------------------------------------------------------
# precision: with fp32 scores and accumulation and the softmax weights carried
# as two fp16 MFMA operands (22 significant bits), the GPU's value before the
# final rounding is off by about 1e-6 absolute (fp32 sums of weighted N(0, 1)
# values), far below an fp16 spacing at every output magnitude above ~2^-10,
# so every output is one of the two fp16 neighbours of the exact (fp64) value
# up to that allowance, and nearly always the nearest one: only values within
# it of a rounding midpoint can go the other way (a bias would show as ~50 %)
# ---------------------------------------------------------------------------

FP32_ALLOWANCE = 1e-6


def fp16_ulp(x):
    """Spacing of fp16 values at |x| (the subnormal spacing below 2^-14)."""
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -14)))
    return 2.0 ** (e - 10)


@pytest.mark.parametrize("name,lens,Hq,Hkv", SMALL + [("few_tokens", [1, 2, 3, 2, 5, 2, 17], 32, 8)],
                         ids=[s[0] for s in SMALL] + ["few_tokens"])
@pytest.mark.parametrize("workers", [0, 7])
def test_outputs_are_fp16_neighbours_of_the_exact_result(torch_cuda, apex, oracle_mod, name, lens, Hq, Hkv,
                                                         workers):
    case = W.make_host_case(lens, Hq, Hkv, seed=len(lens) * 13 + Hq, poison=True)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    got = run_gpu(torch_cuda, apex, case, num_workers=workers).astype(np.float64)
    nonzero = np.asarray(lens) > 0
    ref, got = ref[nonzero], got[nonzero]
    excess = np.abs(got - ref) - fp16_ulp(ref)
    worst = int(np.argmax(excess))
    print(f"[precision] {name} workers={workers}: max excess over one fp16 spacing {excess.flat[worst]:.2e} "
          f"at exact value {ref.flat[worst]:.3e}", flush=True)
    assert np.all(excess <= FP32_ALLOWANCE), "an output is not an fp16 neighbour of the exact value"
    nearest = got == ref.astype(np.float16).astype(np.float64)
    print(f"[precision] {name} workers={workers}: {nearest.mean():.6f} of outputs correctly rounded", flush=True)
    assert nearest.mean() >= 0.98


# ---------------------------------------------------------------------------
# degenerate batches: nothing to attend, or one request among many empty ones
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("lens", [[0], [0, 0, -3, 0], [-1] * 300], ids=["one", "four", "300"])
def test_all_empty_batch_gives_zero_rows(torch_cuda, apex, lens):
    torch = torch_cuda
    case = W.make_host_case(lens, 32, 8, seed=41, poison=True)
    q, k, v, bt, cl = to_dev(torch, case)
    B = len(lens)
    for kw in (dict(), dict(num_workers=5), dict(check_inputs=True)):
        lse = torch.zeros((B, 32), dtype=torch.float32, device="cuda")
        out = torch.full((B, 32, 128), 7.0, dtype=torch.float16, device="cuda")
        apex.decode_attention_ex(q, k, v, bt, cl, case.scale, out=out, lse_out=lse, **kw)
        torch.cuda.synchronize()
        assert bool((out == 0).all()), kw
        assert bool(torch.isneginf(lse).all()), kw
    assert apex.check_device_error() == 0
    out = torch.full((B, 32, 128), 7.0, dtype=torch.float16, device="cuda")
    apex.decode_attention_noalloc(q, k, v, bt, cl, case.scale, out)
    torch.cuda.synchronize()
    assert bool((out == 0).all())


def test_one_long_request_among_many_empty_ones(torch_cuda, apex, oracle_mod):
    lens = [0] * 150 + [5000] + [0, 1] * 60 + [0] * 80
    case = W.make_host_case(lens, 32, 8, seed=42, poison=True)
    ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                          case.context_lens, case.scale)
    for workers in (0, 3, 100):
        got = run_gpu(torch_cuda, apex, case, num_workers=workers)
        assert_parity(got, ref, f"one long among empty, workers={workers}")
        assert np.all(got[np.asarray(lens) == 0] == 0)
