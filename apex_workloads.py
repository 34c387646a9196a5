"""Seeded synthetic decode-attention workloads (inputs only).

This module draws inputs and nothing else: request lengths, a paged block
placement, and fp16 Q/K/V tensors.  It contains none of the attention
arithmetic, so both the HIP path and the oracle can be fed from it.

The five named workloads are Llama-shaped single-layer decode batches
(d = 128, block_size = 16, fp16 values drawn from N(0, 1) and rounded to
nearest even):

  c1  tiny MHA (Llama-2-7B heads 32/32): B=4, lengths exactly 17, 64, 200,
      511, contiguous block placement
  c2  Llama-2-7B MHA: B=64, lengths uniform in [512, 2048]
  c3  Llama-3.1-8B GQA (32 q-heads over 8 kv-heads): B=128, lengths uniform
      in [1024, 4096]
  c4  long-output chain-of-thought GQA: B=32, lengths round(exp(N(ln 12000,
      0.5^2))) clipped to [4096, 32768]
  c5  memory-pressure mixed GQA batch: B=512, half the lengths uniform in
      [256, 1024] and half in [4096, 16384], shuffled; keys get a per
      kv-head offset vector drawn from N(0, 0.5^2)

Generation order for a seed: lengths -> physical block permutation -> key
offsets (c5) -> Q, K, V from a torch generator with the same seed.  Integer
bounds are inclusive.  Rows of the block table past a request's last block
hold block 0 unless ``poison`` asks for a NaN-filled slack block instead.
"""
from dataclasses import dataclass, field
import hashlib
import math

import numpy as np

D_HEAD = 128
BLOCK_SIZE = 16
SCALE = float(np.float32(1.0 / math.sqrt(D_HEAD)))


@dataclass(frozen=True)
class Config:
    name: str
    title: str
    seed: int
    B: int
    Hq: int
    Hkv: int
    d: int = D_HEAD
    block_size: int = BLOCK_SIZE
    lens: str = "uniform"          # "fixed" | "uniform" | "lognormal" | "bimodal"
    lo: int = 0
    hi: int = 0
    fixed: tuple = ()
    placement: str = "random"      # "random" | "contiguous"
    key_offset_std: float = 0.0


CONFIGS = {
    "c1": Config("c1", "tiny MHA decode attention, Llama-2-7B heads, B=4, L={17,64,200,511}",
                 1, 4, 32, 32, lens="fixed", fixed=(17, 64, 200, 511), placement="contiguous"),
    "c2": Config("c2", "Llama-2-7B MHA decode, B=64, L~U[512,2048], paged bs=16",
                 2, 64, 32, 32, lens="uniform", lo=512, hi=2048),
    "c3": Config("c3", "Llama-3.1-8B GQA decode, B=128, L~U[1024,4096], paged bs=16",
                 3, 128, 32, 8, lens="uniform", lo=1024, hi=4096),
    "c4": Config("c4", "Llama-3.1-8B GQA long-output CoT decode, B=32, L~lognormal(med 12k) in [4096,32768], paged bs=16",
                 4, 32, 32, 8, lens="lognormal", lo=4096, hi=32768),
    "c5": Config("c5", "Llama-3.1-8B GQA memory-pressure mixed batch, B=512, L half U[256,1024] half U[4096,16384], paged bs=16",
                 5, 512, 32, 8, lens="bimodal", placement="random", key_offset_std=0.5),
    # parity shapes beyond the five workloads: the other two group sizes at full size
    "g8": Config("g8", "GQA G=8 (Llama-3-70B heads, 64 q over 8 kv), B=32, c4's lengths, paged bs=16",
                 6, 32, 64, 8, lens="lognormal", lo=4096, hi=32768),
    "g2": Config("g2", "GQA G=2 (32 q over 16 kv), B=128, c3's lengths, paged bs=16",
                 7, 128, 32, 16, lens="uniform", lo=1024, hi=4096),
}


def draw_lengths(cfg, rng):
    if cfg.lens == "fixed":
        return np.asarray(cfg.fixed, dtype=np.int64)
    if cfg.lens == "uniform":
        return rng.integers(cfg.lo, cfg.hi, size=cfg.B, endpoint=True)
    if cfg.lens == "lognormal":
        x = np.exp(rng.normal(math.log(12000.0), 0.5, size=cfg.B))
        return np.clip(np.rint(x), cfg.lo, cfg.hi).astype(np.int64)
    if cfg.lens == "bimodal":
        half = cfg.B // 2
        short = rng.integers(256, 1024, size=half, endpoint=True)
        long_ = rng.integers(4096, 16384, size=cfg.B - half, endpoint=True)
        lens = np.concatenate([short, long_])
        rng.shuffle(lens)
        return lens
    raise ValueError(cfg.lens)


@dataclass
class Layout:
    """Paged placement of a batch: lengths, block table, pool size."""
    lens: np.ndarray          # int32 [B]
    block_table: np.ndarray   # int32 [B][maxb]
    num_blocks: int           # physical blocks in the pool (incl. slack)
    slack: list = field(default_factory=list)   # ids of slack (unused) blocks


def make_layout(lens, block_size, rng, placement="random", slack_blocks=0, stride=None):
    """Assign each request's logical blocks to distinct physical blocks.

    With ``stride`` the table rows are that wide (>= the tight width)."""
    lens = np.asarray(lens, dtype=np.int64)
    nblk = [max(0, -(-int(L) // block_size)) for L in lens]
    used = int(sum(nblk))
    total = used + int(slack_blocks)
    maxb = max([1] + nblk)
    width = maxb if stride is None else int(stride)
    if width < maxb:
        raise ValueError("stride narrower than the longest request")
    if placement == "contiguous":
        perm = np.arange(total, dtype=np.int64)
    elif placement == "random":
        perm = rng.permutation(total)
    else:
        raise ValueError(placement)
    table = np.zeros((len(lens), width), dtype=np.int32)
    off = 0
    for b, n in enumerate(nblk):
        table[b, :n] = perm[off:off + n]
        off += n
    slack = [int(x) for x in perm[used:]]
    return Layout(lens.astype(np.int32), table, total, slack)


@dataclass
class HostCase:
    """A small case held in host memory as numpy arrays (fp16 values)."""
    q: np.ndarray             # float16 [B][Hq][d]
    k_cache: np.ndarray       # float16 [NB][Hkv][bs][d]
    v_cache: np.ndarray
    block_table: np.ndarray   # int32 [B][stride]
    context_lens: np.ndarray  # int32 [B]
    scale: float
    layout: Layout = None

    @property
    def shape(self):
        B, Hq, d = self.q.shape
        return B, Hq, self.k_cache.shape[1], d, self.k_cache.shape[2]


def make_host_case(lens, Hq, Hkv, d=D_HEAD, block_size=BLOCK_SIZE, seed=0,
                   placement="random", slack_blocks=0, poison=False, scale=SCALE,
                   stride=None, key_offset_std=0.0):
    """Draw a small case on the host with numpy (bit-reproducible anywhere).

    ``poison`` fills every slot the attention must not read (tails of last
    blocks, slack blocks) with NaN and points unused table entries at a
    NaN-filled slack block (one slack block is added if none was asked for).
    """
    rng = np.random.default_rng(seed)
    if poison and slack_blocks == 0:
        slack_blocks = 1
    lay = make_layout(lens, block_size, rng, placement, slack_blocks, stride)
    B = len(lay.lens)
    mu = None
    if key_offset_std > 0:
        mu = rng.normal(0.0, key_offset_std, size=(Hkv, d))
    q = rng.standard_normal((B, Hq, d)).astype(np.float16)
    kf = rng.standard_normal((lay.num_blocks, Hkv, block_size, d))
    if mu is not None:
        kf = kf + mu[None, :, None, :]
    k = kf.astype(np.float16)
    v = rng.standard_normal((lay.num_blocks, Hkv, block_size, d)).astype(np.float16)
    if poison:
        nan = np.float16(np.nan)
        for blk in lay.slack:
            k[blk] = nan
            v[blk] = nan
        for b in range(B):
            L = int(lay.lens[b])
            n = max(0, -(-L // block_size))
            if n and L % block_size:
                last = lay.block_table[b, n - 1]
                k[last, :, L % block_size:, :] = nan
                v[last, :, L % block_size:, :] = nan
            lay.block_table[b, n:] = lay.slack[0]
    return HostCase(q, k, v, lay.block_table, lay.lens, float(np.float32(scale)), lay)


def config_layout(cfg, seed=None):
    """Lengths and block table of a named workload (host, numpy)."""
    rng = np.random.default_rng(cfg.seed if seed is None else seed)
    lens = draw_lengths(cfg, rng)
    lay = make_layout(lens, cfg.block_size, rng, cfg.placement)
    mu = None
    if cfg.key_offset_std > 0:
        mu = rng.normal(0.0, cfg.key_offset_std, size=(cfg.Hkv, cfg.d))
    return lay, mu


def algorithmic_bytes(lens, B, Hq, Hkv, d):
    """KV + Q + O bytes the method must move (valid tokens only, fp16)."""
    kv = int(np.sum(np.maximum(np.asarray(lens, dtype=np.int64), 0))) * Hkv * d * 2 * 2
    return kv + 2 * B * Hq * d * 2


def flops(lens, Hq, d):
    """QK^T + PV multiply-adds counted as 2 flops each."""
    return int(np.sum(np.maximum(np.asarray(lens, dtype=np.int64), 0))) * Hq * d * 4


class DeviceWorkload:
    """A named workload materialised in device memory with torch.

    Q/K/V are drawn with ``torch.randn`` on ``device`` from a generator seeded
    with the workload's seed, in fp32 chunks rounded to fp16.  The tails of
    each request's last block are zero.
    """

    def __init__(self, name, device="cuda", seed=None, chunk_blocks=8192):
        import torch
        cfg = CONFIGS[name]
        self.cfg = cfg
        self.name = name
        lay, mu = config_layout(cfg, seed)
        self.layout = lay
        self.lens = lay.lens
        seed = cfg.seed if seed is None else seed
        gen = torch.Generator(device=device)
        gen.manual_seed(seed)
        B, Hq, Hkv, d, bs = cfg.B, cfg.Hq, cfg.Hkv, cfg.d, cfg.block_size
        self.q = torch.randn((B, Hq, d), generator=gen, device=device, dtype=torch.float32).half()
        nb = lay.num_blocks
        self.k_cache = torch.empty((nb, Hkv, bs, d), dtype=torch.float16, device=device)
        self.v_cache = torch.empty_like(self.k_cache)
        mu_t = None
        if mu is not None:
            mu_t = torch.from_numpy(mu).to(device=device, dtype=torch.float32)[None, :, None, :]
        for dst, add_mu in ((self.k_cache, True), (self.v_cache, False)):
            for s in range(0, nb, chunk_blocks):
                e = min(nb, s + chunk_blocks)
                x = torch.randn((e - s, Hkv, bs, d), generator=gen, device=device, dtype=torch.float32)
                if add_mu and mu_t is not None:
                    x += mu_t
                dst[s:e] = x.half()
                del x
        # zero the unused tail slots of every request's last block
        for b in range(B):
            L = int(lay.lens[b])
            if L % bs:
                last = int(lay.block_table[b, (L - 1) // bs])
                self.k_cache[last, :, L % bs:, :] = 0
                self.v_cache[last, :, L % bs:, :] = 0
        self.block_table = torch.from_numpy(lay.block_table).to(device)
        self.context_lens = torch.from_numpy(lay.lens).to(device)
        self.out = torch.empty((B, Hq, d), dtype=torch.float16, device=device)
        self.scale = SCALE

    def to(self, device):
        """Move every tensor to ``device`` (e.g. a case drawn on the CPU)."""
        for name in ("q", "k_cache", "v_cache", "block_table", "context_lens", "out"):
            setattr(self, name, getattr(self, name).to(device))
        return self

    @property
    def algorithmic_bytes(self):
        c = self.cfg
        return algorithmic_bytes(self.lens, c.B, c.Hq, c.Hkv, c.d)

    @property
    def flops(self):
        return flops(self.lens, self.cfg.Hq, self.cfg.d)

    def host_request_case(self, requests):
        """Copy the given requests' Q rows and KV blocks to the host as a
        compact HostCase (same values; block table remapped)."""
        import torch
        reqs = [int(r) for r in requests]
        bs = self.cfg.block_size
        ids = []
        rows = []
        for b in reqs:
            n = -(-int(self.lens[b]) // bs)
            rows.append(list(range(len(ids), len(ids) + n)))
            ids.extend(int(x) for x in self.layout.block_table[b, :n])
        idx = torch.tensor(ids if ids else [0], dtype=torch.long, device=self.k_cache.device)
        k = self.k_cache.index_select(0, idx).cpu().numpy()
        v = self.v_cache.index_select(0, idx).cpu().numpy()
        width = max([1] + [len(r) for r in rows])
        table = np.zeros((len(reqs), width), dtype=np.int32)
        for i, r in enumerate(rows):
            table[i, :len(r)] = r
        q = self.q[torch.tensor(reqs, dtype=torch.long, device=self.q.device)].cpu().numpy()
        lens = np.asarray([self.lens[b] for b in reqs], dtype=np.int32)
        return HostCase(q, k, v, table, lens, self.scale)


def fp16_digest(*arrays):
    """SHA-256 over the raw bytes of the given numpy arrays."""
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def append_slots(layout, block_size=BLOCK_SIZE):
    """Cache slot of each request's newest token (position L_b - 1), as an
    engine assigns it before the step: block_table[b][(L-1) // bs] * bs +
    (L-1) % bs; -1 (padding) for L_b <= 0.  int64 [B]."""
    slots = np.full(len(layout.lens), -1, dtype=np.int64)
    for b, L in enumerate(layout.lens):
        L = int(L)
        if L > 0:
            slots[b] = int(layout.block_table[b, (L - 1) // block_size]) * block_size + (L - 1) % block_size
    return slots


@dataclass
class AppendCase:
    """Inputs of one KV append: caches, new rows and their slots (host)."""
    k_cache: np.ndarray       # float16 [NB][Hkv][bs][d]
    v_cache: np.ndarray
    k_new: np.ndarray         # float16 [T][Hkv][d]
    v_new: np.ndarray
    slot_mapping: np.ndarray  # int64 [T]


def make_append_case(T, num_blocks, Hkv, d=D_HEAD, block_size=BLOCK_SIZE, seed=0,
                     padding=0, out_of_range=0):
    """T new tokens with distinct random slots in a pool of ``num_blocks``
    blocks; ``padding`` of them get slot -1 and ``out_of_range`` of them a
    slot at or past the pool's end."""
    rng = np.random.default_rng(seed)
    cap = num_blocks * block_size
    if T - padding - out_of_range > cap:
        raise ValueError("more tokens than slots")
    slots = rng.choice(cap, size=T - padding - out_of_range, replace=False).astype(np.int64)
    extra = np.concatenate([np.full(padding, -1, dtype=np.int64),
                            cap + rng.integers(0, 4 * block_size, size=out_of_range)])
    slots = np.concatenate([slots, extra])
    rng.shuffle(slots)
    k = rng.standard_normal((num_blocks, Hkv, block_size, d)).astype(np.float16)
    v = rng.standard_normal((num_blocks, Hkv, block_size, d)).astype(np.float16)
    kn = rng.standard_normal((T, Hkv, d)).astype(np.float16)
    vn = rng.standard_normal((T, Hkv, d)).astype(np.float16)
    return AppendCase(k, v, kn, vn, slots)
