"""Seeded input generators: shapes, byte accounting and determinism (CPU)."""
import numpy as np
import pytest

import apex_workloads as W


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_config_lengths_and_table(name):
    cfg = W.CONFIGS[name]
    lay, mu = W.config_layout(cfg)
    lens = lay.lens
    assert lens.shape == (cfg.B,) and lens.dtype == np.int32
    if cfg.lens == "fixed":
        assert list(lens) == list(cfg.fixed)
    elif cfg.lens == "uniform":
        assert lens.min() >= cfg.lo and lens.max() <= cfg.hi
    elif cfg.lens == "lognormal":
        assert lens.min() >= 4096 and lens.max() <= 32768
        assert 8000 < np.median(lens) < 18000
    elif cfg.lens == "bimodal":
        short = lens[lens <= 1024]
        long_ = lens[lens >= 4096]
        assert len(short) == cfg.B // 2 and len(long_) == cfg.B - cfg.B // 2
    nblk = -(-lens.astype(np.int64) // 16)
    assert lay.num_blocks == int(nblk.sum())
    assert lay.block_table.shape == (cfg.B, int(nblk.max()))
    used = np.concatenate([lay.block_table[b, :n] for b, n in enumerate(nblk)])
    assert np.array_equal(np.sort(used), np.arange(lay.num_blocks))
    if cfg.placement == "contiguous":
        assert np.array_equal(used, np.arange(lay.num_blocks))
    assert (mu is not None) == (cfg.key_offset_std > 0)
    lay2, _ = W.config_layout(cfg)
    assert np.array_equal(lay.block_table, lay2.block_table)


def test_algorithmic_bytes_formula():
    # c1: 792 tokens x 32 kv-heads x 128 x 2 (K,V) x 2 B + Q + O
    assert W.algorithmic_bytes([17, 64, 200, 511], 4, 32, 32, 128) == 792 * 32 * 128 * 4 + 2 * 4 * 32 * 128 * 2
    # GQA: 4096 B per token
    assert W.algorithmic_bytes([1], 1, 32, 8, 128) - 2 * 32 * 128 * 2 == 4096


def test_host_case_is_seeded_and_poison_only_outside_context():
    a = W.make_host_case([5, 33], 4, 2, seed=3)
    b = W.make_host_case([5, 33], 4, 2, seed=3)
    assert W.fp16_digest(a.q, a.k_cache, a.v_cache) == W.fp16_digest(b.q, b.k_cache, b.v_cache)
    p = W.make_host_case([5, 33], 4, 2, seed=3, poison=True)
    for bi, L in enumerate(p.context_lens):
        for t in range(int(L)):
            blk = p.block_table[bi, t // 16]
            assert np.all(np.isfinite(p.k_cache[blk, :, t % 16].astype(np.float32)))
    assert np.isnan(p.k_cache[p.layout.slack[0]].astype(np.float32)).all()
