"""Decode attention of one request whose block table repeats physical blocks,
computed from the multiset of its tokens (test infrastructure, numpy fp64).

Softmax attention weighs every token position on its own, so a cached token
that the table reaches c times enters the sums c times:

    out[h] = sum_t c_t exp(s_t - M) V_t / sum_t c_t exp(s_t - M),
    s_t = scale * q[h] . K_t,   M = max over the tokens present,

summed over the distinct (block, slot) tokens.  Its cost follows the pool,
not the context length, so it stands in for the oracle on contexts far too
long for the oracle's loop (a table of 2^27 entries); tests/test_oracle.py
checks it against the oracle on small tables first.
"""
import numpy as np


def token_counts(table_row, L, block_size, num_blocks):
    """Times each (physical block, slot) holds one of the request's L tokens:
    float64 [num_blocks][block_size]."""
    nb = -(-int(L) // block_size)
    row = np.asarray(table_row[:nb], dtype=np.int64)
    counts = np.zeros((num_blocks, block_size), dtype=np.float64)
    if nb == 0:
        return counts
    full = np.bincount(row[:nb - 1], minlength=num_blocks).astype(np.float64)
    counts += full[:, None]
    counts[row[nb - 1], :int(L) - block_size * (nb - 1)] += 1.0
    return counts


def multiset_attention(q, k_cache, v_cache, table_row, L, scale):
    """q fp16 [Hq][d]; caches fp16 [NB][Hkv][bs][d]; one request of L tokens
    whose blocks are table_row[0 .. ceil(L / bs) - 1].  Returns float64
    [Hq][d] (zeros when L <= 0)."""
    Hq, d = q.shape
    NB, Hkv, bs, _ = k_cache.shape
    out = np.zeros((Hq, d), dtype=np.float64)
    if L <= 0:
        return out
    counts = token_counts(table_row, L, bs, NB)
    present = counts > 0
    c = counts[present]                                    # [n]
    sc = float(np.float32(scale))
    G = Hq // Hkv
    for h in range(Hq):
        g = h // G
        K = k_cache[:, g].astype(np.float64)[present]      # [n][d]
        V = v_cache[:, g].astype(np.float64)[present]
        s = (K @ q[h].astype(np.float64)) * sc
        w = c * np.exp(s - s.max())
        out[h] = (w @ V) / w.sum()
    return out
