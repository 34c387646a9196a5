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


def warm_up(torch, A, seconds=0.3):
    """Continuous attention calls until the GPU runs at its steady clocks (the
    first calls after idle run a few percent slower)."""
    import time
    q, k, v, bt, lens = decode_batch(torch, 32, 4096, seed=1)
    out = torch.empty_like(q)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(50):
            A.decode_attention(q, k, v, bt, lens, D ** -0.5, out=out)
        torch.cuda.synchronize()
    del q, k, v, bt, lens, out


def run_profile(threads=16, log=print):
    import torch

    import paper_2506_03296_amd as A
    if not torch.cuda.is_available():
        raise RuntimeError("the profiler needs a GPU")
    A.load_library()
    warm_up(torch, A)
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


def markdown(prof, command):
    """The profile and its decisions as a markdown summary."""
    L = ["# Strategy-selection profile — MI355X + its host (Llama-3.1-8B layer)", "",
         "Command (repository root, on the GPU box):", "", "```", command, "```", "",
         f"Device: {prof['device']}; host backend: {prof['host_isa']}, {prof['host_threads']} threads. "
         "Raw tables: `profiles/sched_profile_mi355x.json` (the keys of `apex_sched_profile`). GPU times: "
         "events around each call with the calls queued back to back behind a spin kernel (median of 20), "
         "after about 0.3 s of continuous calls (steady clocks); host times: wall clock, best of 3.", "",
         "## GPU decode attention T_gatt (this library's kernel, per layer)", "",
         "| batch × length | context tokens | µs | KV GB/s |", "|---|---|---|---|"]
    for p in prof["gatt_points"]:
        tok = p["batch"] * p["length"]
        L.append(f"| {p['batch']} × {p['length']} | {tok} | {p['seconds'] * 1e6:.1f} | "
                 f"{tok * HKV * D * 4 / p['seconds'] / 1e9:.0f} |")
    L += ["", "## GPU decode linears T_glinear (bf16 GEMMs of one layer, torch.matmul)", "",
          "| batch | µs |", "|---|---|"]
    for b, t in zip(prof["glin_batch"], prof["glin_seconds"]):
        L.append(f"| {int(b)} | {t * 1e6:.1f} |")
    if prof.get("pref_tokens"):
        L += ["", "## Prefill (per layer)", "",
              "| prompt tokens | linears µs | attention µs (torch SDPA, causal) |", "|---|---|---|"]
        for s, a, b in zip(prof["pref_tokens"], prof["pref_linear_seconds"], prof["pref_attn_seconds"]):
            L.append(f"| {int(s)} | {a * 1e6:.1f} | {b * 1e6:.1f} |")
    L += ["", "## Host attention (this library's CPU backend, per layer), ms", "",
          "| batch \\ context tokens | " + " | ".join(str(int(t)) for t in prof["cpu_tokens"]) + " |",
          "|---|" + "---|" * len(prof["cpu_tokens"])]
    for b, row in zip(prof["cpu_batch"], prof["cpu_seconds"]):
        L.append(f"| {int(b)} | " + " | ".join(f"{t * 1e3:.2f}" for t in row) + " |")
    big = prof["cpu_tokens"][-1]
    rates = [big * HKV * D * 4 / row[-1] / 1e9 for row in prof["cpu_seconds"]]
    L += ["", f"KV bytes per context token per layer: {HKV} kv-heads × {D} × 2 B × 2 (K, V) = 4 KiB; the "
          f"{int(big)}-token column moves {big * HKV * D * 4 / 1e9:.1f} GB at ≈ {min(rates):.0f}–{max(rates):.0f} GB/s.",
          "", "## Decisions (Alg. 2, decode only) for the long-output GPU batch (32 requests, 411 026 tokens)", "",
          "| CPU batch | CPU tokens | N_G (tok/s) | N_C (tok/s) | N_G/N_C | Eq. 6 bound | T_gatt/T_glinear | strategy |",
          "|---|---|---|---|---|---|---|---|"]
    for r in prof["decisions"]:
        L.append(f"| {r['cpu_batch']} | {r['cpu_tokens']} | {r['n_g']:.3g} | {r['n_c']:.3g} | {r['ratio']:.1f} | "
                 f"{r['bound']:.2f} | {r['t_gatt'] / r['t_glinear']:.2f} | {r['strategy']} |")
    ratios = [r["ratio"] for r in prof["decisions"]]
    bound = prof["decisions"][0]["bound"]
    if min(ratios) > bound:
        L += ["", f"On this pairing the host's attention rate is ≈ {100 / max(ratios):.1f}–{100 / min(ratios):.1f} % of "
              f"the GPU's (N_G/N_C ≈ {min(ratios):.0f}–{max(ratios):.0f}), above the Eq. 6 bound (≈ {bound:.1f}), so "
              "Asymmetric Pipelining does not pay and the scheduler picks Asynchronous Overlap -- the regime the "
              "paper describes for N_C below 10 % of N_G."]
    return "\n".join(L) + "\n"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--md", default="", help="also write the markdown summary here")
    ap.add_argument("--threads", type=int, default=0, help="host threads (0 = min(16, cores))")
    args = ap.parse_args()
    threads = args.threads or max(1, min(16, len(os.sched_getaffinity(0))))
    prof = run_profile(threads, log=lambda m: print(f"[profiler] {m}", flush=True))
    prof["decisions"] = decisions(prof)
    with open(args.out, "w") as f:
        json.dump(prof, f, indent=1)
    if args.md:
        cmd = "python -m paper_2506_03296_amd.profiler --out " + args.out + " --md " + args.md
        with open(args.md, "w") as f:
            f.write(markdown(prof, cmd))
    for r in prof["decisions"]:
        print(f"[profiler] CPU batch {r['cpu_batch']} ({r['cpu_tokens']} tokens): N_G/N_C = {r['ratio']:.1f}, "
              f"Eq. 6 bound {r['bound']:.2f} -> {r['strategy']}", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
