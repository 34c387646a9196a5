"""Offline profiler: the measured tables APEX's scheduler reads (Sec. 3.1
"Offline Profiler and Performance Model", Sec. 3.2 "Parameter Estimation
via Offline Profiling").

    python -m paper_2506_03296_amd.profiler --out profile.json

Per transformer layer of Llama-3.1-8B (hidden 4096, 32 q-heads over 8
kv-heads of 128, MLP 14336), on the GPU it is run on and its host:

  gatt   GPU decode attention (this library's kernel) vs total context
         tokens of the batch (32 requests of equal length, plus wider
         batches at 4096 tokens)
  glin   GPU decode linears vs batch size: QKV, O, gate+up and down
         projections as bf16 GEMMs (torch.matmul on random weights -- a
         profiled input, not part of this library)
  cpu    host attention (this library's CPU backend) on a batch x total
         tokens grid
  pref   prefill linears (the same GEMMs at M = prompt tokens) and prefill
         attention (torch's scaled_dot_product_attention, causal, fp16) vs
         prompt tokens

Times are seconds per layer: GPU ones from events around each call with the
calls queued back to back (median of the repetitions), CPU ones wall clock
(best of the repetitions).  The
output keys are those of apex_sched_profile.
"""
import argparse
import json
import os
import sys
import time

HIDDEN, HQ, HKV, D, MLP = 4096, 32, 8, 128, 14336


def _median(xs):
    xs = sorted(xs)
    return xs[len(xs) // 2]


def gpu_time(torch, fn, reps=20, warmup=3):
    """Median seconds of fn's GPU work.  The stream is held by a spin kernel
    while all repetitions are enqueued, so they run back to back as in an
    engine's queued iteration and each event pair brackets the GPU work, not
    the host's launch latency."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(reps)]
    torch.cuda._sleep(20_000_000)
    for a, b in pairs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return _median([a.elapsed_time(b) * 1e-3 for a, b in pairs])


def decode_batch(torch, B, L, seed):
    """A GQA decode batch of B requests of L tokens on the GPU (random
    placement of 16-token blocks)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    nb_req = -(-L // 16)
    nb = B * nb_req
    k = torch.randn((nb, HKV, 16, D), generator=g, device="cuda").half()
    v = torch.randn((nb, HKV, 16, D), generator=g, device="cuda").half()
    q = torch.randn((B, HQ, D), generator=g, device="cuda").half()
    perm = torch.randperm(nb, generator=g, device="cuda").to(torch.int32)
    bt = perm.reshape(B, nb_req).contiguous()
    lens = torch.full((B,), L, dtype=torch.int32, device="cuda")
    return q, k, v, bt, lens


def profile_gatt(torch, A, log):
    pts = [(32, L) for L in (512, 1024, 2048, 4096, 8192, 16384, 32768)]
    pts += [(B, 4096) for B in (64, 128, 256, 512)]
    rows = []
    for B, L in pts:
        q, k, v, bt, lens = decode_batch(torch, B, L, seed=B * 100003 + L)
        out = torch.empty_like(q)
        t = gpu_time(torch, lambda: A.decode_attention(q, k, v, bt, lens, D ** -0.5, out=out))
        rows.append((B * L, t, B, L))
        log(f"gatt B={B} L={L}: {t * 1e6:.1f} us")
        del q, k, v, bt, lens, out
    rows.sort()
    toks, secs = [], []
    for tok, t, _, _ in rows:
        if toks and tok == toks[-1]:
            secs[-1] = min(secs[-1], t)
            continue
        toks.append(float(tok))
        secs.append(t)
    return toks, secs, [dict(batch=B, length=L, seconds=t) for _, t, B, L in rows]


def layer_linears(torch, M, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    bf = torch.bfloat16

    def w(i, o):
        return (torch.randn((i, o), generator=g, device="cuda") * 0.02).to(bf)

    x = torch.randn((M, HIDDEN), generator=g, device="cuda").to(bf)
    wqkv, wo = w(HIDDEN, (HQ + 2 * HKV) * D), w(HQ * D, HIDDEN)
    wgu, wd = w(HIDDEN, 2 * MLP), w(MLP, HIDDEN)

    def run():
        qkv = torch.matmul(x, wqkv)
        o = torch.matmul(qkv[:, :HQ * D], wo)
        gu = torch.matmul(o, wgu)
        h = torch.nn.functional.silu(gu[:, :MLP]) * gu[:, MLP:]
        return torch.matmul(h, wd)

    return run


def profile_glin(torch, log):
    batches = [1, 8, 32, 128, 512, 2048]
    secs = []
    for B in batches:
        t = gpu_time(torch, layer_linears(torch, B, seed=B))
        secs.append(t)
        log(f"glin B={B}: {t * 1e6:.1f} us")
    return [float(b) for b in batches], secs


def profile_prefill(torch, log):
    toks = [512, 2048, 8192]
    lin, att = [], []
    for S in toks:
        lin.append(gpu_time(torch, layer_linears(torch, S, seed=S), reps=10))
        g = torch.Generator(device="cuda")
        g.manual_seed(S)
        q = torch.randn((1, HQ, S, D), generator=g, device="cuda").half()
        k = torch.randn((1, HKV, S, D), generator=g, device="cuda").half()
        v = torch.randn((1, HKV, S, D), generator=g, device="cuda").half()
        kr = k.repeat_interleave(HQ // HKV, dim=1).contiguous()
        vr = v.repeat_interleave(HQ // HKV, dim=1).contiguous()
        sdpa = torch.nn.functional.scaled_dot_product_attention
        try:
            att.append(gpu_time(torch, lambda: sdpa(q, kr, vr, is_causal=True), reps=10))
        except RuntimeError as e:   # no fused prefill attention on this build
            log(f"prefill attention unavailable: {e}")
            return [], [], []
        log(f"prefill S={S}: linears {lin[-1] * 1e6:.1f} us, attention {att[-1] * 1e6:.1f} us")
        del q, k, v, kr, vr
    return [float(s) for s in toks], lin, att


def profile_cpu(torch, threads, log, reps=3):
    from . import cpu
    cpu.set_threads(threads)
    batches = [1, 4, 16, 64]
    tokens = [8192, 32768, 131072, 524288]
    grid = []
    for B in batches:
        row = []
        for T in tokens:
            L = T // B
            q, k, v, bt, lens = decode_batch(torch, B, L, seed=7 * B + T)
            qh, kh, vh = q.cpu().numpy(), k.cpu().numpy(), v.cpu().numpy()
            bth, lh = bt.cpu().numpy(), lens.cpu().numpy()
            del q, k, v, bt, lens
            out = cpu.decode_attention(qh, kh, vh, bth, lh, D ** -0.5)
            best = float("inf")
            for _ in range(reps):
                t0 = time.perf_counter()
                cpu.decode_attention(qh, kh, vh, bth, lh, D ** -0.5, out=out)
                best = min(best, time.perf_counter() - t0)
            row.append(best)
            log(f"cpu B={B} tokens={T}: {best * 1e3:.2f} ms ({T * HKV * D * 4 / best / 1e9:.1f} GB/s)")
            del qh, kh, vh
        grid.append(row)
    return [float(b) for b in batches], [float(t) for t in tokens], grid


def run_profile(threads=16, log=print):
    import torch

    import paper_2506_03296_amd as A
    if not torch.cuda.is_available():
        raise RuntimeError("the profiler needs a GPU")
    A.load_library()
    gt, gs, gpts = profile_gatt(torch, A, log)
    gb, gls = profile_glin(torch, log)
    pt, pl, pa = profile_prefill(torch, log)
    cb, ct, cs = profile_cpu(torch, threads, log)
    from . import cpu
    props = torch.cuda.get_device_properties(0)
    return {
        "device": props.name, "host_threads": threads,
        "host_isa": {2: "avx512", 1: "avx2"}.get(cpu.isa(), "none"),
        "model": "Llama-3.1-8B layer (hidden 4096, 32/8 heads of 128, MLP 14336)",
        "gatt_tokens": gt, "gatt_seconds": gs, "gatt_points": gpts,
        "glin_batch": gb, "glin_seconds": gls,
        "cpu_batch": cb, "cpu_tokens": ct, "cpu_seconds": cs,
        "pref_tokens": pt, "pref_linear_seconds": pl, "pref_attn_seconds": pa,
    }


def decisions(profile, gpu_batch=32, gpu_tokens=411026,
              cpu_cases=((8, 32768), (32, 131072), (128, 524288), (256, 1048576))):
    """Alg. 2 (decode only) for a GPU batch against several CPU batches,
    through the library's scheduler."""
    from . import sched
    rows = []
    for cb, ct in cpu_cases:
        kw = sched.inputs_from_profile(profile, gpu_batch, gpu_tokens, cb, ct)
        r = sched.select(**kw)
        rows.append(dict(cpu_batch=cb, cpu_tokens=ct, n_g=kw["n_g"], n_c=kw["n_c"],
                         ratio=kw["n_g"] / kw["n_c"], bound=r["ratio_bound"],
                         t_glinear=kw["t_glinear"], t_gatt=kw["t_gatt"], strategy=r["strategy"],
                         cpu_to_gpu_requests=cb / gpu_batch))
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--threads", type=int, default=0, help="host threads (0 = min(16, cores))")
    args = ap.parse_args()
    threads = args.threads or max(1, min(16, len(os.sched_getaffinity(0))))
    prof = run_profile(threads, log=lambda m: print(f"[profiler] {m}", flush=True))
    prof["decisions"] = decisions(prof)
    with open(args.out, "w") as f:
        json.dump(prof, f, indent=1)
    for r in prof["decisions"]:
        print(f"[profiler] CPU batch {r['cpu_batch']} ({r['cpu_tokens']} tokens): N_G/N_C = {r['ratio']:.1f}, "
              f"Eq. 6 bound {r['bound']:.2f} -> {r['strategy']}", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
