"""Seeded synthetic workloads for RcLLM's selective prefill of one layer.

This module only draws random numbers and arranges them into the tensors the
path consumes. It holds none of the path's own steps (no gather, no
re-alignment from a table, no scoring, no selection, no attention) and is the
one piece of code that both the GPU path's tests/benchmark and the CPU oracle
read their inputs from.

What a prompt looks like (arXiv 2605.07443, Sec. II-A and Sec. IV-A):
Instruction + History + Items. Instruction tokens are always recomputed
(Sec. III-C.2a): they form a fresh segment whose K/V exist only as freshly
computed rows. The history is one block drawn from a history pool; each item is
one block drawn from an item pool (Sec. III-B stores item KV blocks offline
and reuses them at any position). Item popularity is heavy-tailed (Sec. III-B),
so item ids follow Zipf(a) without replacement within a request and are then
randomly permuted; a gather-bound variant draws them uniformly.

Values. Cached blocks stand in for KV that an offline forward pass computed at
block-local positions 0..L-1; fresh rows stand in for the current request's
projection at absolute positions. For block b with raw (pre-rotation) keys
r_b ~ N(0,1) and values v_b ~ N(0,1):
    pool K  = rope_model(r_b + eps, t)         t = block-local position
    pool V  = v_b + eta                         eps, eta ~ N(0, sigma^2)
    fresh K = rope_model(r_b, dst_start + t)    (the request's own position)
    fresh V = v_b
where rope_model is the model's positional encoding evaluated in fp64 from
angles computed here (rotate-half pairing, angle pos * base^(-2j/D)). It
synthesises the model's outputs; it is not the path's re-alignment step, which
rotates by a position delta using fp32 tables. Fresh-segment K/V and all of Q
are drawn directly as N(0,1). Values are rounded once to the storage dtype.

Pools are generated in chunks of blocks from a counter-based seed
(seed, pool, chunk), so a pool of tens of GB is generated on the device without
a host copy; the fresh rows of each request are written while the chunk that
holds its block is resident.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class Config:
    name: str
    dtype: str              # "f32" or "bf16"
    B: int
    Hq: int
    Hkv: int
    D: int
    rope_base: float
    F: int                  # instruction tokens (fresh)
    hist_len: int
    hist_pool: int
    n_items: int
    item_len: int
    item_pool: int
    item_dist: str = "zipf"  # "zipf" or "uniform"
    zipf_a: float = 1.1
    sigma: float = 0.05
    pct: int = 15
    miss_items: tuple = ()   # item slots served as fresh (cache misses)
    miss_hist: bool = False  # history served as fresh (a cache miss)

    @property
    def N(self) -> int:
        return self.F + self.hist_len + self.n_items * self.item_len

    @property
    def n_fresh(self) -> int:
        return self.F + len(self.miss_items) * self.item_len + (self.hist_len if self.miss_hist else 0)

    @property
    def n_reused(self) -> int:
        return self.N - self.n_fresh

    def k_for(self, pct: int) -> int:
        """Selected cached tokens at recompute ratio pct%: ceil(pct * n_r / 100)."""
        return (self.n_reused * pct + 99) // 100

    @property
    def k(self) -> int:
        return self.k_for(self.pct)

    @property
    def n_hist_reused(self) -> int:
        return 0 if self.miss_hist else self.hist_len

    @property
    def n_item_reused(self) -> int:
        return (self.n_items - len(self.miss_items)) * self.item_len

    def k_split(self, pct_hist: int, pct_item: int | None = None) -> tuple:
        """Separate budgets for the history and item components (recompute
        ratios r_rev and r_item): (ceil(pct_hist * n_hist / 100),
        ceil(pct_item * n_item / 100))."""
        pct_item = pct_hist if pct_item is None else pct_item
        return ((self.n_hist_reused * pct_hist + 99) // 100,
                (self.n_item_reused * pct_item + 99) // 100)

    @property
    def R(self) -> int:
        return self.n_fresh + self.k

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five workloads. Sizes, dtypes and distributions are those of the
# recommendation prompts the paper evaluates (median 2.2K-3.0K tokens, items
# the majority of the prompt, Sec. IV-B); layer shapes are Llama-3-8B-like
# (32 Q heads, 8 KV heads, head_dim 128) except the tiny fp32 case.
WORKLOADS = {
    1: Config("tiny-fp32", "f32", B=1, Hq=8, Hkv=8, D=64, rope_base=10000.0, F=32,
              hist_len=128, hist_pool=4, n_items=4, item_len=64, item_pool=16, sigma=0.05,
              pct=15),
    2: Config("llama3-8b-layer-b8-3008", "bf16", B=8, Hq=32, Hkv=8, D=128,
              rope_base=500000.0, F=64, hist_len=1024, hist_pool=256, n_items=20,
              item_len=96, item_pool=10000, sigma=0.05, pct=15),
    3: Config("llama3-8b-layer-b4-8160-long", "bf16", B=4, Hq=32, Hkv=8, D=128,
              rope_base=500000.0, F=64, hist_len=4096, hist_pool=256, n_items=50,
              item_len=80, item_pool=20000, sigma=0.08, pct=10),
    4: Config("llama3-8b-layer-b8-4096-sweep", "bf16", B=8, Hq=32, Hkv=8, D=128,
              rope_base=500000.0, F=96, hist_len=1024, hist_pool=256, n_items=31,
              item_len=96, item_pool=10000, sigma=0.05, pct=15),
    5: Config("gather-bound-b64-2080-pool200k", "bf16", B=64, Hq=32, Hkv=8, D=128,
              rope_base=500000.0, F=32, hist_len=512, hist_pool=256, n_items=24,
              item_len=64, item_pool=200000, item_dist="uniform", sigma=0.05, pct=15),
}

SWEEP_PCTS = (0, 5, 10, 15, 25, 50, 100)

# Pool 1 holds the item blocks: their cached K/V are lexical matches, so the
# divergence term of the full importance score is dropped for them.
ITEM_POOL_MASK = 1 << 1

# Small shapes for tests: several attention tiles, ragged tails, GQA and MHA.
TEST_WORKLOADS = {
    "tiny-bf16": Config("tiny-bf16", "bf16", B=2, Hq=8, Hkv=2, D=128, rope_base=500000.0,
                        F=16, hist_len=64, hist_pool=4, n_items=3, item_len=48, item_pool=12),
    "ragged-bf16": Config("ragged-bf16", "bf16", B=3, Hq=16, Hkv=4, D=128,
                          rope_base=500000.0, F=7, hist_len=53, hist_pool=3, n_items=5,
                          item_len=37, item_pool=9, pct=20),
    "mha-d64-bf16": Config("mha-d64-bf16", "bf16", B=2, Hq=4, Hkv=4, D=64, rope_base=10000.0,
                           F=5, hist_len=70, hist_pool=2, n_items=4, item_len=33,
                           item_pool=6, pct=30),
    "miss-bf16": Config("miss-bf16", "bf16", B=2, Hq=8, Hkv=2, D=128, rope_base=500000.0,
                        F=16, hist_len=64, hist_pool=4, n_items=4, item_len=40,
                        item_pool=10, miss_items=(1, 3)),
    "tiny-f32-gqa": Config("tiny-f32-gqa", "f32", B=2, Hq=8, Hkv=2, D=64, rope_base=10000.0,
                           F=9, hist_len=40, hist_pool=3, n_items=3, item_len=21,
                           item_pool=7, pct=25),
    # every segment a cache miss: nothing is reused, every position is fresh
    "allfresh-bf16": Config("allfresh-bf16", "bf16", B=2, Hq=8, Hkv=2, D=128,
                            rope_base=500000.0, F=16, hist_len=64, hist_pool=4, n_items=3,
                            item_len=48, item_pool=12, miss_items=(0, 1, 2), miss_hist=True),
}


@dataclass
class Workload:
    cfg: Config
    seed: int
    q: torch.Tensor                  # [B, N, Hq, D]
    k_fresh: torch.Tensor            # [B, N, Hkv, D]
    v_fresh: torch.Tensor            # [B, N, Hkv, D]
    pools: list                      # [(pool_k, pool_v)], each [P, L, Hkv, D]
    segs: torch.Tensor               # [B, S, 4] int32 (host)
    item_ids: torch.Tensor           # [B, n_items] int64 (host)
    hist_ids: torch.Tensor           # [B] int64 (host)
    planted: torch.Tensor = field(default=None)  # [B, m] positions with extra noise

    @property
    def N(self):
        return self.cfg.N


def _mix(*xs: int) -> int:
    """Fold integers into one 63-bit seed (splitmix64 finaliser on each step)."""
    h = 0x9E3779B97F4A7C15
    for x in xs:
        h = (h ^ (int(x) & 0xFFFFFFFFFFFFFFFF)) & 0xFFFFFFFFFFFFFFFF
        h = (h * 0xBF58476D1CE4E5B9) & 0xFFFFFFFFFFFFFFFF
        h ^= h >> 31
        h = (h * 0x94D049BB133111EB) & 0xFFFFFFFFFFFFFFFF
        h ^= h >> 29
    return h & 0x7FFFFFFFFFFFFFFF


def _gen(device, *key) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_mix(*key))
    return g


def _rope_model(x: torch.Tensor, pos: torch.Tensor, base: float) -> torch.Tensor:
    """The model's positional encoding at absolute positions, in fp64.
    x: [..., T, H, D] (fp64), pos: [T] -> rotated x (fp64)."""
    D = x.shape[-1]
    half = D // 2
    j = torch.arange(half, dtype=torch.float64, device=x.device)
    inv = torch.pow(torch.tensor(base, dtype=torch.float64, device=x.device), -2.0 * j / D)
    ang = pos.to(torch.float64)[:, None] * inv[None, :]          # [T, half]
    c = torch.cos(ang)[:, None, :]                                # [T, 1, half]
    s = torch.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return torch.cat([a * c - b * s, a * s + b * c], dim=-1)


def sample_ids(cfg: Config, seed: int):
    """History ids (uniform) and item ids (Zipf(a) or uniform, no repeats
    within a request, randomly permuted). Drawn on the host."""
    g = _gen("cpu", seed, 1)
    hist = torch.randint(0, cfg.hist_pool, (cfg.B,), generator=g)
    if cfg.item_dist == "zipf":
        ranks = torch.arange(1, cfg.item_pool + 1, dtype=torch.float64)
        w = ranks.pow(-cfg.zipf_a)
        rank_to_id = torch.randperm(cfg.item_pool, generator=g)
        items = torch.empty((cfg.B, cfg.n_items), dtype=torch.int64)
        for b in range(cfg.B):
            r = torch.multinomial(w, cfg.n_items, replacement=False, generator=g)
            r = r[torch.randperm(cfg.n_items, generator=g)]
            items[b] = rank_to_id[r]
    elif cfg.item_dist == "uniform":
        items = torch.empty((cfg.B, cfg.n_items), dtype=torch.int64)
        for b in range(cfg.B):
            # without replacement: rejection on the rare duplicate
            while True:
                c = torch.randint(0, cfg.item_pool, (cfg.n_items,), generator=g)
                if c.unique().numel() == cfg.n_items:
                    break
            items[b] = c
    else:
        raise ValueError(cfg.item_dist)
    return hist, items


def segment_table(cfg: Config, hist: torch.Tensor, items: torch.Tensor) -> torch.Tensor:
    """[B, S, 4] int32: (dst_start, len, pool, block); pool -1 = fresh.
    Pool 0 holds history blocks, pool 1 item blocks."""
    S = 2 + cfg.n_items
    segs = torch.empty((cfg.B, S, 4), dtype=torch.int32)
    for b in range(cfg.B):
        segs[b, 0] = torch.tensor([0, cfg.F, -1, 0])
        segs[b, 1] = (torch.tensor([cfg.F, cfg.hist_len, -1, 0]) if cfg.miss_hist
                      else torch.tensor([cfg.F, cfg.hist_len, 0, int(hist[b])]))
        for i in range(cfg.n_items):
            dst = cfg.F + cfg.hist_len + i * cfg.item_len
            if i in cfg.miss_items:
                segs[b, 2 + i] = torch.tensor([dst, cfg.item_len, -1, 0])
            else:
                segs[b, 2 + i] = torch.tensor([dst, cfg.item_len, 1, int(items[b, i])])
    return segs


def make(cfg: Config, seed: int, device="cpu", sigma: float | None = None,
         planted: int = 0, planted_scale: float = 20.0, chunk_elems: int = 1 << 27,
         pool_seed: int | None = None, pools: list | None = None) -> Workload:
    """Generate one batch of the workload `cfg` on `device`.

    Pool contents are drawn from `pool_seed` (default `seed`). Passing `pools`
    made earlier with the same pool_seed and sigma reuses them: only the batch's
    own draws (ids, Q, fresh rows) are new, the block contents are re-derived
    from the same counter-based seeds."""
    sigma = cfg.sigma if sigma is None else float(sigma)
    pool_seed = seed if pool_seed is None else pool_seed
    dt = cfg.torch_dtype
    B, N, Hq, Hkv, D = cfg.B, cfg.N, cfg.Hq, cfg.Hkv, cfg.D
    hist, items = sample_ids(cfg, seed)
    segs = segment_table(cfg, hist, items)

    gq = _gen(device, seed, 2)
    q = torch.randn((B, N, Hq, D), generator=gq, device=device, dtype=torch.float32).to(dt)
    k_fresh = torch.empty((B, N, Hkv, D), device=device, dtype=dt)
    v_fresh = torch.empty((B, N, Hkv, D), device=device, dtype=dt)

    # fresh segments: drawn directly
    gf = _gen(device, seed, 3)
    for b in range(B):
        for s in range(segs.shape[1]):
            dst, ln, p, _ = (int(x) for x in segs[b, s])
            if p < 0 and ln > 0:
                k_fresh[b, dst:dst + ln] = torch.randn((ln, Hkv, D), generator=gf, device=device,
                                                       dtype=torch.float32).to(dt)
                v_fresh[b, dst:dst + ln] = torch.randn((ln, Hkv, D), generator=gf, device=device,
                                                       dtype=torch.float32).to(dt)

    # which (request, segment) uses which block of which pool
    users = {0: {}, 1: {}}
    for b in range(B):
        for s in range(segs.shape[1]):
            dst, ln, p, blk = (int(x) for x in segs[b, s])
            if p >= 0:
                users[p].setdefault(blk, []).append((b, dst, ln))

    reuse = pools is not None
    new_pools = []
    for p, (P, L) in enumerate([(cfg.hist_pool, cfg.hist_len), (cfg.item_pool, cfg.item_len)]):
        if reuse:
            pk, pv = pools[p]
        else:
            pk = torch.empty((P, L, Hkv, D), device=device, dtype=dt)
            pv = torch.empty((P, L, Hkv, D), device=device, dtype=dt)
        local = torch.arange(L, device=device)
        per_chunk = max(1, chunk_elems // (L * Hkv * D))
        for c, c0 in enumerate(range(0, P, per_chunk)):
            c1 = min(P, c0 + per_chunk)
            if reuse and not any(blk in users[p] for blk in range(c0, c1)):
                continue
            g = _gen(device, pool_seed, 4, p, c)
            shp = (c1 - c0, L, Hkv, D)
            raw = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
            val = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
            if not reuse:
                eps = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
                eta = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
                noisy = raw.to(torch.float64) + sigma * eps.to(torch.float64)
                pk[c0:c1] = _rope_model(noisy, local, cfg.rope_base).to(dt)
                pv[c0:c1] = (val.to(torch.float64) + sigma * eta.to(torch.float64)).to(dt)
                del noisy, eps, eta
            for blk in range(c0, c1):
                for (b, dst, ln) in users[p].get(blk, ()):
                    pos = torch.arange(dst, dst + ln, device=device)
                    r = raw[blk - c0, :ln].to(torch.float64)
                    k_fresh[b, dst:dst + ln] = _rope_model(r, pos, cfg.rope_base).to(dt)
                    v_fresh[b, dst:dst + ln] = val[blk - c0, :ln].to(dt)
            del raw, val
        new_pools.append((pk, pv))
    pools = new_pools

    planted_pos = None
    if planted:
        # extra noise of planted_scale * sigma on the fresh K of m cached positions
        gp = _gen("cpu", seed, 5)
        reused = [i for i in range(N)
                  if not any(int(segs[0, s, 2]) < 0 and int(segs[0, s, 0]) <= i <
                             int(segs[0, s, 0]) + int(segs[0, s, 1])
                             for s in range(segs.shape[1]))]
        reused = torch.tensor(reused)
        planted_pos = torch.empty((B, planted), dtype=torch.int64)
        ge = _gen(device, seed, 6)
        for b in range(B):
            pick = reused[torch.randperm(len(reused), generator=gp)[:planted]].sort().values
            planted_pos[b] = pick
            for i in pick.tolist():
                e = torch.randn((Hkv, D), generator=ge, device=device, dtype=torch.float32)
                kf = k_fresh[b, i].to(torch.float32) + planted_scale * max(sigma, 0.05) * e
                k_fresh[b, i] = kf.to(dt)

    return Workload(cfg=cfg, seed=seed, q=q, k_fresh=k_fresh, v_fresh=v_fresh, pools=pools,
                    segs=segs, item_ids=items, hist_ids=hist, planted=planted_pos)


def to_host_bits(t: torch.Tensor):
    """Host numpy view of a tensor's storage: float32 stays float32, bf16 becomes
    its uint16 bit patterns (the CPU oracle's bf16 storage format)."""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError(t.dtype)


def referenced_subpools(w: Workload):
    """Host copies of only the pool blocks the batch references, plus a segment
    table remapped onto them (for the CPU oracle on pools too large to copy)."""
    segs = w.segs.clone()
    subpools = []
    for p, (pk, pv) in enumerate(w.pools):
        mask = segs[..., 2] == p
        ids = segs[..., 3][mask].to(torch.int64)
        uniq, inv = torch.unique(ids, return_inverse=True)
        segs[..., 3][mask] = inv.to(torch.int32)
        idx = uniq.to(pk.device)
        subpools.append((to_host_bits(pk.index_select(0, idx)),
                         to_host_bits(pv.index_select(0, idx))))
    return subpools, segs.numpy()


def scale_for(D: int) -> float:
    return 1.0 / math.sqrt(D)


@dataclass
class TokenWorkload:
    """A batch whose history is token-granular: every history position reuses
    one single-token prototype row (Sec. III-B builds history prototypes per
    token), items stay blocks. pools[0] holds the prototypes ([n_protos, 1,
    Hkv, D]), pools[1] the item blocks."""
    w: Workload
    token_map: torch.Tensor     # [B, N, 4] int32 (host): {pool, row, delta, 0}
    status_segs: torch.Tensor   # [B, S, 4] int32 (host): fresh / cached runs for selection
    proto_ids: torch.Tensor     # [B, hist_len] int64 (host)


def make_prototypes(cfg: Config, seed: int, device="cpu", n_protos: int = 4096,
                    sigma: float | None = None) -> TokenWorkload:
    """Workload `cfg` with a prototype history: each history position draws a
    prototype id uniformly; the prototype row is stored at position 0
    (pool K = raw + eps, pool V = v + eta) and the position's fresh K/V are
    the model's rows of the clean prototype at that position."""
    sigma = cfg.sigma if sigma is None else float(sigma)
    w = make(cfg, seed, device=device, sigma=sigma)
    dt = cfg.torch_dtype
    B, N, Hkv, D = cfg.B, cfg.N, cfg.Hkv, cfg.D
    g = _gen(device, seed, 7)
    shp = (n_protos, 1, Hkv, D)
    raw = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
    val = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
    eps = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
    eta = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
    proto_k = (raw.to(torch.float64) + sigma * eps.to(torch.float64)).to(dt)  # position 0: no rotation
    proto_v = (val.to(torch.float64) + sigma * eta.to(torch.float64)).to(dt)
    gi = _gen("cpu", seed, 8)
    ids = torch.randint(0, n_protos, (B, cfg.hist_len), generator=gi)
    h0, h1 = cfg.F, cfg.F + cfg.hist_len
    pos = torch.arange(h0, h1, device=device)
    for b in range(B):
        idx = ids[b].to(device)
        r = raw[idx, 0].to(torch.float64)                      # [hist_len, Hkv, D]
        w.k_fresh[b, h0:h1] = _rope_model(r, pos, cfg.rope_base).to(dt)
        w.v_fresh[b, h0:h1] = val[idx, 0].to(dt)
    tmap = torch.zeros((B, N, 4), dtype=torch.int32)
    tmap[..., 0] = -1
    segs = w.segs
    for b in range(B):
        for s in range(segs.shape[1]):
            dst, ln, p, blk = (int(x) for x in segs[b, s])
            if p == 0:
                tmap[b, dst:dst + ln, 0] = 0
                tmap[b, dst:dst + ln, 1] = ids[b, :ln].to(torch.int32)
                tmap[b, dst:dst + ln, 2] = torch.arange(dst, dst + ln, dtype=torch.int32)
            elif p > 0:
                tmap[b, dst:dst + ln, 0] = p
                tmap[b, dst:dst + ln, 1] = blk * cfg.item_len + torch.arange(ln, dtype=torch.int32)
                tmap[b, dst:dst + ln, 2] = dst
    status = segs.clone()
    status[..., 3] = torch.where(status[..., 2] == 0, torch.zeros_like(status[..., 3]), status[..., 3])
    w.pools = [(proto_k, proto_v), w.pools[1]]
    w.segs = status
    return TokenWorkload(w=w, token_map=tmap, status_segs=status, proto_ids=ids)


def token_map_from_segments(segs, block_lens) -> torch.Tensor:
    """The per-position map equivalent to a segment table: row = block *
    block_len + offset, delta = dst_start."""
    segs = torch.as_tensor(segs)
    B, S = segs.shape[:2]
    N = int(segs[0, :, 1].sum())
    tmap = torch.zeros((B, N, 4), dtype=torch.int32)
    tmap[..., 0] = -1
    for b in range(B):
        for s in range(S):
            dst, ln, p, blk = (int(x) for x in segs[b, s])
            if p >= 0:
                tmap[b, dst:dst + ln, 0] = p
                tmap[b, dst:dst + ln, 1] = blk * int(block_lens[p]) + torch.arange(ln, dtype=torch.int32)
                tmap[b, dst:dst + ln, 2] = dst
    return tmap


@dataclass
class LayerWeights:
    """One decoder layer (pre-norm attention + SwiGLU MLP), bf16."""
    w_qkv: torch.Tensor   # [(Hq + 2 Hkv) D, H]: q heads, then k heads, then v heads
    w_o: torch.Tensor     # [H, Hq D]
    w_gu: torch.Tensor    # [2 I, H]: gate rows, then up rows
    w_down: torch.Tensor  # [H, I]
    g_attn: torch.Tensor  # [H]
    g_mlp: torch.Tensor   # [H]


def make_layers(n_layers: int, H: int, Hq: int, Hkv: int, D: int, inter: int, seed: int,
                device="cpu"):
    """Random decoder-layer weights, bf16: projections ~ N(0, 1/fan_in) so the
    residual stream keeps unit scale; norm gains ~ 1 + N(0, 0.1^2)."""
    layers = []
    for l in range(n_layers):
        g = _gen(device, seed, 9, l)

        def w(rows, cols):
            return (torch.randn((rows, cols), generator=g, device=device, dtype=torch.float32)
                    / math.sqrt(cols)).to(torch.bfloat16)

        gains = 1.0 + 0.1 * torch.randn((2, H), generator=g, device=device, dtype=torch.float32)
        layers.append(LayerWeights(w_qkv=w((Hq + 2 * Hkv) * D, H), w_o=w(H, Hq * D),
                                   w_gu=w(2 * inter, H), w_down=w(H, inter),
                                   g_attn=gains[0].to(torch.bfloat16), g_mlp=gains[1].to(torch.bfloat16)))
    return layers


def make_stack(cfg: Config, seed: int, n_layers: int, H: int, inter: int, device="cpu"):
    """A batch of `cfg` for a stack of decoder layers: input states x [B, N, H]
    ~ N(0, 1), one pool set per layer (independent contents, the same
    segment table), random layer weights. Returns (x, layers, pools_by_layer,
    segs [B, S, 4])."""
    w0 = make(cfg, seed, device=device)
    pools = [w0.pools]
    for l in range(1, n_layers):
        pools.append(make(cfg, seed, device=device, pool_seed=seed * 131 + l).pools)
    gx = _gen(device, seed, 10)
    x = torch.randn((cfg.B, cfg.N, H), generator=gx, device=device, dtype=torch.float32).to(cfg.torch_dtype)
    layers = make_layers(n_layers, H, cfg.Hq, cfg.Hkv, cfg.D, inter, seed, device)
    segs = w0.segs
    return x, layers, pools, segs
