"""The Asynchronous Overlap runtime (libapex_overlap.so) on the GPU and host.

What it must deliver, checked against the oracles: the result a poll/wait
copies back is the attention of the request's new query over its host KV
cache with this token's K/V appended (oracle/kv_cache.py then the fp64
attention oracle, to the attention bar), and the host cache afterwards holds
exactly the appended rows.  Around that: results submitted in one iteration
are collected in the next while the next submits (two slots per layer); the
readiness check never blocks and reports "not ready" while the compute thread
is held from the host; a slot still in use is refused; bad arguments are
rejected; destroying with work pending drains it.
"""
import time

import numpy as np
import pytest

import apex_workloads as W
from oracle import kv_cache

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
def ov():
    from paper_2506_03296_amd import cpu, overlap
    overlap.load_library()
    cpu.set_threads(max(1, min(8, cpu.threads())))
    return overlap


def make_runtime(ov, layers=2, max_requests=8, num_blocks=96, slots_per_layer=0):
    return ov.Overlap(layers=layers, max_requests=max_requests, Hq=32, Hkv=8, d=128, block_size=16,
                      scale=W.SCALE, num_blocks=num_blocks, max_blocks_per_request=32,
                      threads=4, slots_per_layer=slots_per_layer)


class Requests:
    """CPU-attended requests of one layer: their host cache content, block
    table and lengths, and the next token's rows (host copies for the oracle,
    device copies for the runtime)."""

    def __init__(self, torch, lens, num_blocks, seed, packed=False):
        self.rng = np.random.default_rng(seed)
        self.packed = packed
        self.layout = W.make_layout(lens, 16, self.rng, "random", slack_blocks=num_blocks - sum(
            -(-L // 16) for L in lens), stride=32)
        self.lens = self.layout.lens.copy()
        self.free = list(self.layout.slack)
        self.torch = torch

    def fill(self, k, v):
        k[:] = self.rng.standard_normal(k.shape).astype(np.float16)
        v[:] = self.rng.standard_normal(v.shape).astype(np.float16)

    def next_token(self):
        """Rows of the token at position lens (the step's new token); grows lens."""
        B = len(self.lens)
        # a request crossing into a new block gets a free block of the pool
        for b in range(B):
            if int(self.lens[b]) % 16 == 0:
                self.layout.block_table[b, int(self.lens[b]) // 16] = self.free.pop()
        self.lens = self.lens + 1
        self.q = self.rng.standard_normal((B, 32, 128)).astype(np.float16)
        self.kn = self.rng.standard_normal((B, 8, 128)).astype(np.float16)
        self.vn = self.rng.standard_normal((B, 8, 128)).astype(np.float16)
        lay = W.Layout(self.lens, self.layout.block_table, self.layout.num_blocks)
        self.slots = W.append_slots(lay)
        dev = "cuda"
        t = self.torch
        if self.packed:
            # q | k | v back to back in one device buffer (one copy to the host)
            flat = np.concatenate([self.q.ravel(), self.kn.ravel(), self.vn.ravel()])
            d = t.from_numpy(flat).to(dev)
            nq, nk = self.q.size, self.kn.size
            return (d[:nq].view(self.q.shape), d[nq:nq + nk].view(self.kn.shape),
                    d[nq + nk:].view(self.vn.shape))
        return (t.from_numpy(self.q).to(dev), t.from_numpy(self.kn).to(dev),
                t.from_numpy(self.vn).to(dev))

    def expected(self, oracle_mod, k_before, v_before):
        kc, vc = kv_cache.kv_append(k_before, v_before, self.kn, self.vn, self.slots)
        out = oracle_mod.decode_attention_f64(self.q, kc, vc, self.layout.block_table, self.lens, W.SCALE)
        return out, kc, vc


def assert_close(got, ref, what):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), what
    err = float(np.abs(got - ref).max())
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    print(f"[overlap] {what}: max_abs={err:.3e} rel_l2={rel:.3e}", flush=True)
    assert err <= MAX_ABS and rel <= REL_L2, what


@pytest.mark.parametrize("packed", [False, True])
def test_single_submit_matches_oracles(torch_cuda, ov, oracle_mod, packed):
    torch = torch_cuda
    with make_runtime(ov) as rt:
        req = Requests(torch, [17, 64, 200, 1, 100, 15], 96, seed=1, packed=packed)
        k, v = rt.host_cache(0)
        req.fill(k, v)
        kb, vb = k.copy(), v.copy()
        q, kn, vn = req.next_token()
        t = rt.submit(0, q, kn, vn, req.slots, req.layout.block_table, req.lens)
        out = torch.empty_like(q)
        rt.wait(t, out)
        torch.cuda.synchronize()
        ref, kc, vc = req.expected(oracle_mod, kb, vb)
        assert_close(out.cpu().numpy(), ref, "single submit")
        assert np.array_equal(k.view(np.uint16), kc.view(np.uint16))
        assert np.array_equal(v.view(np.uint16), vc.view(np.uint16))


def test_deferred_collection_over_iterations(torch_cuda, ov, oracle_mod):
    """Iteration n submits every layer, then collects iteration n-1's results
    (one iteration late, as the overlap schedule does); three iterations.
    The runtime appends to a layer's host cache while that layer has jobs
    pending, so the expected caches are the test's own (the oracle's append
    applied iteration by iteration); the runtime's caches are compared with
    them once nothing is pending."""
    torch = torch_cuda
    layers = 3
    with make_runtime(ov, layers=layers) as rt:
        reqs = [Requests(torch, [30, 47, 5, 120], 96, seed=10 + l, packed=l % 2 == 1) for l in range(layers)]
        model = []
        for l in range(layers):
            k, v = rt.host_cache(l)
            reqs[l].fill(k, v)
            model.append((k.copy(), v.copy()))
        prev = None
        for it in range(3):
            cur = []
            for l in range(layers):
                q, kn, vn = reqs[l].next_token()
                t = rt.submit(l, q, kn, vn, reqs[l].slots, reqs[l].layout.block_table, reqs[l].lens)
                ref, kc, vc = reqs[l].expected(oracle_mod, *model[l])
                model[l] = (kc, vc)
                cur.append((t, ref, torch.empty_like(q)))
            if prev is not None:
                for l, (t, ref, out) in enumerate(prev):
                    deadline = time.time() + 60
                    while not rt.poll(t, out):
                        assert time.time() < deadline, "result never became ready"
                        time.sleep(0.001)
                    torch.cuda.synchronize()
                    assert_close(out.cpu().numpy(), ref, f"iteration {it - 1} layer {l}")
            prev = cur
        for l, (t, ref, out) in enumerate(prev):
            rt.wait(t, out)
        torch.cuda.synchronize()
        assert rt.pending() == 0
        for l, (t, ref, out) in enumerate(prev):
            assert_close(out.cpu().numpy(), ref, f"last iteration layer {l}")
            k, v = rt.host_cache(l)
            assert np.array_equal(k.view(np.uint16), model[l][0].view(np.uint16)), f"layer {l} K cache"
            assert np.array_equal(v.view(np.uint16), model[l][1].view(np.uint16)), f"layer {l} V cache"


def test_poll_does_not_block_while_held(torch_cuda, ov, oracle_mod):
    torch = torch_cuda
    from paper_2506_03296_amd.overlap import OverlapError
    with make_runtime(ov) as rt:
        req = Requests(torch, [40, 9], 96, seed=3)
        k, v = rt.host_cache(1)
        req.fill(k, v)
        kb, vb = k.copy(), v.copy()
        rt.hold(True)
        q, kn, vn = req.next_token()
        t = rt.submit(1, q, kn, vn, req.slots, req.layout.block_table, req.lens)
        out = torch.zeros_like(q)
        for _ in range(20):
            t0 = time.perf_counter()
            assert rt.poll(t, out) is False
            assert time.perf_counter() - t0 < 0.05
        assert rt.pending() == 1
        with pytest.raises(OverlapError) as e:
            rt.wait(t, out)
        assert e.value.code == -5
        rt.hold(False)
        rt.wait(t, out)
        torch.cuda.synchronize()
        assert rt.pending() == 0
        ref, _, _ = req.expected(oracle_mod, kb, vb)
        assert_close(out.cpu().numpy(), ref, "after release")
        with pytest.raises(OverlapError):
            rt.poll(t, out)               # already collected


def test_busy_slot_is_refused(torch_cuda, ov):
    torch = torch_cuda
    from paper_2506_03296_amd.overlap import OverlapError
    with make_runtime(ov, slots_per_layer=1) as rt:
        req = Requests(torch, [20], 96, seed=4)
        q, kn, vn = req.next_token()
        t = rt.submit(0, q, kn, vn, req.slots, req.layout.block_table, req.lens)
        with pytest.raises(OverlapError) as e:
            rt.submit(0, q, kn, vn, req.slots, req.layout.block_table, req.lens)
        assert e.value.code == -5
        out = torch.empty_like(q)
        rt.wait(t, out)
        torch.cuda.synchronize()
        t2 = rt.submit(0, q, kn, vn, req.slots, req.layout.block_table, req.lens)
        with pytest.raises(OverlapError):
            rt.poll(t, out)               # superseded ticket
        rt.wait(t2, out)


def test_bad_arguments(torch_cuda, ov):
    torch = torch_cuda
    from paper_2506_03296_amd.overlap import OverlapError
    with make_runtime(ov, max_requests=2) as rt:
        req = Requests(torch, [20, 30, 40], 96, seed=5)
        q, kn, vn = req.next_token()
        with pytest.raises(OverlapError):
            rt.submit(0, q, kn, vn, req.slots, req.layout.block_table, req.lens)     # B > max
        with pytest.raises(OverlapError):
            rt.submit(5, q[:2], kn[:2], vn[:2], req.slots[:2], req.layout.block_table[:2], req.lens[:2])
        bad = req.layout.block_table[:2].copy()
        bad[0, 0] = 96
        with pytest.raises(OverlapError):
            rt.submit(0, q[:2], kn[:2], vn[:2], req.slots[:2], bad, req.lens[:2])
        with pytest.raises(OverlapError):
            rt.host_cache(2)
        # refused in the binding: rows the runtime would copy as raw bytes
        with pytest.raises(ValueError, match="q must be"):
            rt.submit(0, q[:2].float(), kn[:2], vn[:2], req.slots[:2], req.layout.block_table[:2],
                      req.lens[:2])
        with pytest.raises(ValueError, match="context_lens must hold"):
            rt.submit(0, q[:2], kn[:2], vn[:2], req.slots[:2], req.layout.block_table[:2], req.lens[:1])
        t = rt.submit(0, q[:2], kn[:2], vn[:2], req.slots[:2], req.layout.block_table[:2], req.lens[:2])
        with pytest.raises(ValueError, match="out holds 1 rows"):
            rt.wait(t, torch.empty((1, 32, 128), dtype=torch.float16, device="cuda"))
        rt.wait(t, torch.empty((2, 32, 128), dtype=torch.float16, device="cuda"))


def test_destroy_with_pending_work_drains(torch_cuda, ov):
    torch = torch_cuda
    rt = make_runtime(ov)
    req = Requests(torch, [300, 100], 96, seed=6)
    rt.hold(True)
    q, kn, vn = req.next_token()
    rt.submit(0, q, kn, vn, req.slots, req.layout.block_table, req.lens)
    rt.submit(1, q, kn, vn, req.slots, req.layout.block_table, req.lens)
    assert rt.pending() == 2
    rt.close()
