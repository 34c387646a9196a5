"""One decode layer-step -- paged KV append, then the attention -- captured in
a HIP graph (torch.cuda.graph) and replayed.

Both calls are stream-ordered only: no host synchronisation, no allocation
(the attention gets a caller workspace) and no memset; the attention's arrival
counters return to zero at the end of every launch.  So every replay must equal
the eager calls bit for bit.  Replays are interleaved with eager work on the
same buffers and with in-place changes of the inputs, which the replays must
see (they read the buffers, not values captured at record time).
"""
import numpy as np
import pytest

import apex_workloads as W

pytestmark = pytest.mark.gpu

HQ, HKV, D, BS = 32, 8, 128, 16


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
    """Cache slot of each request's current (last) token; -1 for L <= 0."""
    slots = np.full(len(case.context_lens), -1, dtype=np.int64)
    for b, L in enumerate(case.context_lens):
        if L > 0:
            slots[b] = int(case.block_table[b, (L - 1) // BS]) * BS + (L - 1) % BS
    return slots


def bits(t):
    return t.view(dtype=__import__("torch").int16).cpu().numpy()


def test_layer_step_graph_replays_bitwise(torch_cuda, apex):
    torch = torch_cuda
    lens = [300, 17, 1600, 64, 0, 999, 4096]
    case = W.make_host_case(lens, HQ, HKV, seed=97)
    B = len(lens)
    dev = "cuda"
    rng = np.random.default_rng(98)
    q = torch.from_numpy(case.q).to(dev)
    bt = torch.from_numpy(case.block_table).to(dev)
    cl = torch.from_numpy(case.context_lens).to(dev)
    k_new = torch.from_numpy(rng.standard_normal((B, HKV, D)).astype(np.float16)).to(dev)
    v_new = torch.from_numpy(rng.standard_normal((B, HKV, D)).astype(np.float16)).to(dev)
    slots = torch.from_numpy(current_slots(case)).to(dev)

    def eager(qq):
        """The layer-step on fresh copies of the caches, library workspace."""
        kc = torch.from_numpy(case.k_cache).to(dev)
        vc = torch.from_numpy(case.v_cache).to(dev)
        apex.kv_append(k_new, v_new, kc, vc, slots)
        out = apex.decode_attention(qq, kc, vc, bt, cl, case.scale)
        torch.cuda.synchronize()
        return out

    ref = eager(q)

    kc = torch.from_numpy(case.k_cache).to(dev)
    vc = torch.from_numpy(case.v_cache).to(dev)
    ws = torch.zeros(apex.workspace_bytes(B, HQ, HKV), dtype=torch.uint8, device=dev)
    out = torch.empty_like(q)

    def step():
        apex.kv_append(k_new, v_new, kc, vc, slots)
        apex.decode_attention_ex(q, kc, vc, bt, cl, case.scale, out=out, workspace=ws)

    # warm up on a side stream (lazy set-up happens outside the capture)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out), bits(ref)), "eager call with the caller workspace"

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    for rep in range(4):
        out.fill_(7.0)                      # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(out), bits(ref)), f"replay {rep}"
        step()                              # an eager step on the same buffers
        torch.cuda.synchronize()
        assert np.array_equal(bits(out), bits(ref)), f"eager step after replay {rep}"
    # the counters in the caller workspace are back to zero
    assert int(ws[:apex.counter_bytes(B, HKV)].to(torch.int32).abs().sum()) == 0

    # the replay reads the buffers: a new query is seen
    q.mul_(-0.5)
    ref2 = eager(q)
    graph.replay()
    torch.cuda.synchronize()
    assert np.array_equal(bits(out), bits(ref2)), "replay after changing q in place"
    assert not np.array_equal(bits(ref2), bits(ref))


def test_fused_layer_step_graph_replays_bitwise(torch_cuda, apex):
    """The fused call (attention + append of the current token in one
    launch) with a caller workspace, captured and replayed: every replay
    equals the eager fused call bit for bit, outputs and caches."""
    torch = torch_cuda
    lens = [300, 17, 1600, 64, 0, 999, 4096, 1]
    case = W.make_host_case(lens, HQ, HKV, seed=99)
    B = len(lens)
    dev = "cuda"
    rng = np.random.default_rng(100)
    q = torch.from_numpy(case.q).to(dev)
    bt = torch.from_numpy(case.block_table).to(dev)
    cl = torch.from_numpy(case.context_lens).to(dev)
    k_new = torch.from_numpy(rng.standard_normal((B, HKV, D)).astype(np.float16)).to(dev)
    v_new = torch.from_numpy(rng.standard_normal((B, HKV, D)).astype(np.float16)).to(dev)

    def eager():
        kc = torch.from_numpy(case.k_cache).to(dev)
        vc = torch.from_numpy(case.v_cache).to(dev)
        out = apex.decode_attention_ex(q, kc, vc, bt, cl, case.scale, k_new=k_new, v_new=v_new)
        torch.cuda.synchronize()
        return out, kc, vc

    ref, ref_k, ref_v = eager()
    kc = torch.from_numpy(case.k_cache).to(dev)
    vc = torch.from_numpy(case.v_cache).to(dev)
    ws = torch.zeros(apex.workspace_bytes(B, HQ, HKV), dtype=torch.uint8, device=dev)
    out = torch.empty_like(q)

    def step():
        apex.decode_attention_ex(q, kc, vc, bt, cl, case.scale, out=out, workspace=ws, k_new=k_new, v_new=v_new)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out), bits(ref)), "eager fused call with the caller workspace"

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        out.fill_(7.0)
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(out), bits(ref)), f"replay {rep}"
        assert np.array_equal(bits(kc), bits(ref_k)) and np.array_equal(bits(vc), bits(ref_v)), f"caches, replay {rep}"
    assert int(ws[:apex.counter_bytes(B, HKV)].to(torch.int32).abs().sum()) == 0
