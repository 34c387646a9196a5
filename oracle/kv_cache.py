"""Paged KV-cache append, as plain numpy -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline
may import this.  It shares no code with the HIP library.

What it computes.  In the decode phase every request produces one new token
per iteration and its Key and Value vectors are cached at each layer so later
iterations need not recompute them (APEX, Sec. 2.1); the cache is paged
(Sec. 4.1), and the GPU keeps in its memory the KV pairs of the requests it
attends (Sec. 3.1).  Appending is therefore a scatter: token t's K and V rows
(one per kv-head) are stored at the cache slot the engine assigned it.

Readings where the paper is silent (the same layout the attention reads):
  - caches are [num_blocks][Hkv][block_size][d]; slot s names physical block
    s // block_size and position s % block_size inside it;
  - a slot outside [0, num_blocks * block_size) is skipped (negative slots
    are the usual padding marker of a batch); nothing else changes;
  - slots of one call are distinct (with duplicates the result would depend
    on write order, so no order is defined).
"""
import numpy as np


def kv_append(k_cache, v_cache, k_new, v_new, slot_mapping):
    """Return (k_cache', v_cache'): copies with token t's rows k_new[t][g][:]
    and v_new[t][g][:] written at slot slot_mapping[t] for every kv-head g.

    k_cache, v_cache: [NB][Hkv][bs][d]; k_new, v_new: [T][Hkv][d] (any dtype,
    copied bit for bit); slot_mapping: integer [T]."""
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    nb, hkv, bs, d = kc.shape
    kn = np.asarray(k_new)
    vn = np.asarray(v_new)
    slots = np.asarray(slot_mapping).astype(np.int64)
    if kn.shape != (slots.shape[0], hkv, d) or vn.shape != kn.shape:
        raise ValueError("k_new/v_new must be [T][Hkv][d] with T = len(slot_mapping)")
    for t in range(slots.shape[0]):
        s = int(slots[t])
        if s < 0 or s >= nb * bs:
            continue
        block, pos = s // bs, s % bs
        kc[block, :, pos, :] = kn[t]
        vc[block, :, pos, :] = vn[t]
    return kc, vc
