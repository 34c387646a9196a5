"""Independent brute-force restatement of decode attention (pins the C oracle).

TEST INFRASTRUCTURE.  Written separately from ``ref_decode.c``: it densifies
each request's KV with explicit Python loops over tokens, decodes fp16 with
numpy's own binary16 conversion, and applies softmax attention in float64.
Only for tiny inputs.
"""
import math

import numpy as np


def dense_kv(cache, block_table, b, L):
    """Gather request b's first L token rows -> [Hkv][L][d] (float64)."""
    c = np.asarray(cache)
    if c.dtype == np.uint16:
        c = c.view(np.float16)
    nb, hkv, bs, d = c.shape
    rows = np.zeros((hkv, L, d), dtype=np.float64)
    for t in range(L):
        blk = int(block_table[b][t // bs])
        rows[:, t, :] = c[blk, :, t % bs, :].astype(np.float64)
    return rows


def decode_attention(q, k_cache, v_cache, block_table, context_lens, scale):
    qf = np.asarray(q)
    if qf.dtype == np.uint16:
        qf = qf.view(np.float16)
    qf = qf.astype(np.float64)
    B, Hq, d = qf.shape
    hkv = np.asarray(k_cache).shape[1]
    group = Hq // hkv
    s = float(np.float32(scale))
    out = np.zeros((B, Hq, d))
    for b in range(B):
        L = int(context_lens[b])
        if L <= 0:
            continue
        K = dense_kv(k_cache, block_table, b, L)
        V = dense_kv(v_cache, block_table, b, L)
        for h in range(Hq):
            kh = K[h // group]
            vh = V[h // group]
            logits = [s * sum(qf[b, h, i] * kh[t, i] for i in range(d)) for t in range(L)]
            top = max(logits)
            e = [math.exp(z - top) for z in logits]
            tot = sum(e)
            for t in range(L):
                out[b, h, :] += (e[t] / tot) * vh[t]
    return out
