"""apex_decode_attention_noalloc, the entry point that allocates nothing (its
arrival counters and partial results live in a static device array of the
library), against apex_decode_attention on the same inputs: bit for bit --
the same kernel and launch -- and within the attention bar of the fp64
oracle.  Calls come in a row, each next one smaller, so that every call after
the first runs on the array the previous one left behind."""
import numpy as np
import pytest

import apex_workloads as W

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


def both_calls(torch, apex, case):
    dev = "cuda"
    q = torch.from_numpy(case.q).to(dev)
    k = torch.from_numpy(case.k_cache).to(dev)
    v = torch.from_numpy(case.v_cache).to(dev)
    bt = torch.from_numpy(case.block_table).to(dev)
    lens = torch.from_numpy(case.context_lens).to(dev)
    base = apex.decode_attention(q, k, v, bt, lens, case.scale)
    out = torch.full_like(base, float("nan"))
    apex.decode_attention_noalloc(q, k, v, bt, lens, case.scale, out)
    torch.cuda.synchronize()
    return base.cpu().numpy(), out.cpu().numpy()


def check_bar(got, ref, what):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), what
    max_abs = float(np.abs(got - ref).max())
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    print(f"[noalloc] {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e}", flush=True)
    assert max_abs <= MAX_ABS and rel <= REL_L2, what


def ragged_lens(rng, B):
    kinds = rng.choice(["short", "edge", "long", "zero"], size=B, p=[0.35, 0.25, 0.3, 0.1])
    lens = []
    for kind in kinds:
        if kind == "short":
            lens.append(int(rng.integers(1, 64)))
        elif kind == "edge":
            lens.append(int(16 * rng.integers(1, 60) + rng.choice([-1, 0, 1])))
        elif kind == "long":
            lens.append(int(rng.integers(2000, 9000)))
        else:
            lens.append(0)
    return lens


def test_noalloc_matches_the_base_call_on_calls_in_a_row(torch_cuda, apex, oracle_mod):
    """A large ragged GQA batch (pairs split over work groups, so the scratch's
    partials and counters are used), then smaller calls of other group sizes,
    a single request split over many work groups, and a one-token call."""
    rng = np.random.default_rng(2027)
    cases = [
        ("G4 B=96", W.make_host_case(ragged_lens(rng, 96), 32, 8, seed=1, poison=True)),
        ("G1 B=24", W.make_host_case(ragged_lens(rng, 24), 32, 32, seed=2, poison=True)),
        ("G8 B=12", W.make_host_case(ragged_lens(rng, 12), 32, 4, seed=3, poison=True)),
        ("G4 one request of 40000", W.make_host_case([40000], 32, 8, seed=4, poison=True)),
        ("G2 B=3", W.make_host_case([700, 0, 33], 16, 8, seed=5, poison=True)),
        ("G4 one token", W.make_host_case([1], 32, 8, seed=6, poison=True)),
    ]
    for what, case in cases:
        ref = oracle_mod.decode_attention_f64(case.q, case.k_cache, case.v_cache, case.block_table,
                                              case.context_lens, case.scale)
        base, got = both_calls(torch_cuda, apex, case)
        assert np.array_equal(got.view(np.uint16), base.view(np.uint16)), what
        check_bar(got, ref, what)


def test_noalloc_full_size_then_smaller(torch_cuda, apex):
    """The long-output workload (32 requests of 4k-32k tokens), then the
    tiny MHA one, each bit for bit against the base call."""
    torch = torch_cuda
    for name in ("c4", "c1"):
        wl = W.DeviceWorkload(name)
        base = apex.decode_attention(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                                     wl.scale)
        out = torch.full_like(base, float("nan"))
        apex.decode_attention_noalloc(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens,
                                      wl.scale, out)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), base.view(torch.int16)), name
        del wl, base, out
        torch.cuda.empty_cache()


def test_noalloc_refuses_more_pairs_than_its_scratch(torch_cuda, apex):
    """B * Hkv above 65536 is refused on the host; nothing is enqueued."""
    torch = torch_cuda
    B, Hq, Hkv = 8193, 8, 8
    q = torch.zeros((B, Hq, 128), dtype=torch.float16, device="cuda")
    k = torch.zeros((1, Hkv, 16, 128), dtype=torch.float16, device="cuda")
    bt = torch.zeros((B, 1), dtype=torch.int32, device="cuda")
    lens = torch.ones(B, dtype=torch.int32, device="cuda")
    out = torch.full_like(q, 7.0)
    with pytest.raises(apex.ApexError) as e:
        apex.decode_attention_noalloc(q, k, k, bt, lens, 0.1, out)
    assert e.value.code == apex.APEX_ERR_UNSUPPORTED
    assert "65536" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


def test_noalloc_captured_in_a_graph_and_replayed(torch_cuda, apex):
    """The no-allocation call captured in a HIP graph (torch.cuda.graph) and
    replayed; between replays, eager work and eager no-allocation calls of
    another batch share the static scratch.  Every replay must equal the base
    call bit for bit, and a replay must see an in-place change of the query."""
    torch = torch_cuda
    dev = "cuda"
    case = W.make_host_case([3000, 17, 900, 4500, 0, 1, 2048], 32, 8, seed=81, poison=True)
    q, k, v = (torch.from_numpy(x).to(dev) for x in (case.q, case.k_cache, case.v_cache))
    bt, cl = torch.from_numpy(case.block_table).to(dev), torch.from_numpy(case.context_lens).to(dev)
    other = W.make_host_case([700, 33, 5000], 16, 4, seed=82, poison=True)
    oq, ok_, ov = (torch.from_numpy(x).to(dev) for x in (other.q, other.k_cache, other.v_cache))
    obt, ocl = torch.from_numpy(other.block_table).to(dev), torch.from_numpy(other.context_lens).to(dev)
    ref = apex.decode_attention(q, k, v, bt, cl, case.scale)
    oref = apex.decode_attention(oq, ok_, ov, obt, ocl, other.scale)
    out = torch.empty_like(q)
    oout = torch.empty_like(oq)

    # warm up on a side stream (the device's first call sets up outside the capture)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        apex.decode_attention_noalloc(q, k, v, bt, cl, case.scale, out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        apex.decode_attention_noalloc(q, k, v, bt, cl, case.scale, out)
    torch.cuda.synchronize()
    for rep in range(4):
        out.fill_(7.0)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        apex.decode_attention_noalloc(oq, ok_, ov, obt, ocl, other.scale, oout)   # another batch
        torch.cuda.synchronize()
        assert torch.equal(oout.view(torch.int16), oref.view(torch.int16)), f"eager call after replay {rep}"

    q.mul_(-0.5)
    ref2 = apex.decode_attention(q, k, v, bt, cl, case.scale)
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref2.view(torch.int16)), "replay after a new query"


@pytest.mark.parametrize("name", ["c4", "c5"])
def test_noalloc_full_size_workload_equals_the_base_call(torch_cuda, apex, name):
    """A full workload in the benchmark's shape (c4: 32 x 8 pairs, c5: 512 x 8)
    through the static array: the default grid fits it (512 work groups of
    G = 4 under its 1024), so the result is the base call's bit for bit."""
    torch = torch_cuda
    wl = W.DeviceWorkload(name)
    base = apex.decode_attention(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens, wl.scale)
    out = torch.full_like(base, float("nan"))
    apex.decode_attention_noalloc(wl.q, wl.k_cache, wl.v_cache, wl.block_table, wl.context_lens, wl.scale, out)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), base.view(torch.int16))
    del wl, base, out
    torch.cuda.empty_cache()
