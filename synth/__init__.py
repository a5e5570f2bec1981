"""Seeded synthetic KV caches shaped like the paper's workloads.

This module only draws inputs: window queries, keys, values, sequence offsets
and per-sequence slot budgets.  It holds none of the compression method's
arithmetic and is shared by the tests, the benchmark and the smoke check as
the one source of inputs for both the GPU path and the CPU oracle.

The paper evaluates caches of Llama-3.1-8B / Llama-3.3-70B class models at
32K-128K context (LongBench-v2, RULER, a 64K packed prototype).  No weights or
datasets are available here, so caches are synthetic with those shapes:

  keys, window queries  ~ N(0, 1)
  retrieval heads       `needles` planted keys per head: k_j += beta*sqrt(d)*
                        qbar/|qbar|^2 (qbar = mean window query of the head's
                        group), which lifts the mean window logit of key j by
                        exactly beta; positions uniform without replacement in
                        [0, n - w)
  diffuse heads         no needles
  values                sigma_h * N(0,1) or sigma_h * Student-t(3) with
                        log sigma_h ~ U[log 0.2, log 5]
  cancelling pairs      (C5) k_j' = k_j + 0.01 z, v_j' = -v_j

Tensors are produced in the layouts of the C ABI: q_win [L][B*w][H*G][d],
k and v [L][T][H][d], T = total tokens of the ragged batch.
"""
import math
from dataclasses import dataclass, field
from typing import List, Optional

import torch


@dataclass
class CacheConfig:
    name: str
    layers: int
    kv_heads: int
    group: int
    head_dim: int
    window: int
    seqlens: List[int]
    keep_fraction: float          # real-token budget fraction f (n_keep = floor(f n) + 1)
    dtype: torch.dtype
    seed: int
    needles: int = 16
    beta: float = 5.0
    head_mix: str = "half"        # "all" | "half" (heads < H/2) | "bernoulli"
    values: str = "gauss"         # "gauss" | "t3"
    sigma_range: tuple = (0.2, 5.0)
    sigma_on_retrieval: bool = False
    cancel_pairs: int = 0
    retain_mass: float = 0.9
    extra: dict = field(default_factory=dict)

    @property
    def batch(self):
        return len(self.seqlens)

    def n_keep(self):
        return [int(math.floor(self.keep_fraction * n)) + 1 for n in self.seqlens]


def config(name: str, seqlens: Optional[List[int]] = None, layers: Optional[int] = None
           ) -> CacheConfig:
    """The five workload shapes (C1..C5); `seqlens`/`layers` shrink a shape
    for quick checks while keeping its distributions."""
    if name == "C1":  # tiny, fp32, 4 KV heads without GQA
        c = CacheConfig("C1", 1, 4, 1, 64, 16, [1024], 128 / 1024, torch.float32, 1,
                        needles=8, beta=6.0, head_mix="all", sigma_range=(1.0, 1.0))
    elif name == "C2":  # Llama-3-8B shape, one layer, 32K
        c = CacheConfig("C2", 1, 8, 4, 128, 64, [32768], 0.10, torch.bfloat16, 2)
    elif name == "C3":  # Llama-3-8B shape, 32 layers, 128K, Student-t values
        c = CacheConfig("C3", 32, 8, 4, 128, 64, [131072], 0.10, torch.bfloat16, 3,
                        head_mix="bernoulli", values="t3", sigma_on_retrieval=True)
    elif name == "C4":  # ragged batch of 8 single-layer caches
        g = torch.Generator().manual_seed(4)
        lens = torch.randint(8192, 65537, (8,), generator=g).tolist()
        c = CacheConfig("C4", 1, 8, 4, 128, 32, lens, 0.05, torch.bfloat16, 4)
    elif name == "C5":  # Llama-3-70B shape, 80 layers, 128K, cancelling pairs
        c = CacheConfig("C5", 80, 8, 8, 128, 64, [131072], 0.05, torch.bfloat16, 5,
                        cancel_pairs=256, sigma_on_retrieval=True)
    else:
        raise KeyError(name)
    if seqlens is not None:
        c.seqlens = list(seqlens)
    if layers is not None:
        c.layers = layers
    return c


def _is_retrieval(cfg: CacheConfig, gen: torch.Generator, layer: int) -> List[bool]:
    H = cfg.kv_heads
    if cfg.head_mix == "all":
        return [True] * H
    if cfg.head_mix == "half":
        return [h < H // 2 for h in range(H)]
    draw = torch.rand(H, generator=gen, device=gen.device)
    return (draw < 0.5).tolist()


def make_cache(cfg: CacheConfig, device="cpu", layers=None):
    """Draw the cache of `cfg` on `device`.

    Returns a dict: q_win, k, v (torch tensors, cfg.dtype), cu_seqlens (list),
    n_keep (list), retrieval [L][B][H] head types, needle positions.
    `layers` restricts generation to a list of layer indices (others are
    skipped but the random stream of each layer is independent, keyed by
    (seed, layer)), so a subset reproduces the same layers as the full cache.
    """
    L, H, G, d, w = cfg.layers, cfg.kv_heads, cfg.group, cfg.head_dim, cfg.window
    B = cfg.batch
    cu = [0]
    for n in cfg.seqlens:
        assert w <= n
        cu.append(cu[-1] + n)
    T = cu[-1]
    lay = list(range(L)) if layers is None else list(layers)
    q_all = torch.empty((len(lay), B * w, H * G, d), dtype=cfg.dtype, device=device)
    k_all = torch.empty((len(lay), T, H, d), dtype=cfg.dtype, device=device)
    v_all = torch.empty((len(lay), T, H, d), dtype=cfg.dtype, device=device)
    retrieval, needles = [], []
    lo, hi = math.log(cfg.sigma_range[0]), math.log(cfg.sigma_range[1])
    for li, l in enumerate(lay):
        gen = torch.Generator(device=device)
        gen.manual_seed(cfg.seed * 1_000_003 + l)
        ret_l, ndl_l = [], []
        for b in range(B):
            n = cfg.seqlens[b]
            t0 = cu[b]
            ret = _is_retrieval(cfg, gen, l)
            q = torch.randn((w, H * G, d), generator=gen, device=device)
            k = torch.randn((n, H, d), generator=gen, device=device)
            if cfg.values == "t3":
                z = torch.randn((n, H, d), generator=gen, device=device)
                chi = torch.randn((n, H, 3), generator=gen, device=device).pow(2).sum(-1)
                v = z / torch.sqrt(chi / 3.0).unsqueeze(-1)
            else:
                v = torch.randn((n, H, d), generator=gen, device=device)
            sig = torch.exp(lo + (hi - lo) * torch.rand(H, generator=gen, device=device))
            ndl_b = []
            for h in range(H):
                if (not ret[h]) or cfg.sigma_on_retrieval:
                    v[:, h] *= sig[h]
                pos = torch.randperm(n - w, generator=gen, device=device)
                used = 0
                if ret[h] and cfg.needles > 0:
                    p = pos[:cfg.needles]
                    used = cfg.needles
                    qbar = q[:, h * G:(h + 1) * G].reshape(-1, d).mean(0)
                    k[p, h] += cfg.beta * math.sqrt(d) * qbar / qbar.dot(qbar)
                    ndl_b.append(sorted(p.tolist()))
                else:
                    ndl_b.append([])
                if cfg.cancel_pairs > 0:
                    pc = pos[used:used + 2 * cfg.cancel_pairs]
                    a, bb = pc[:cfg.cancel_pairs], pc[cfg.cancel_pairs:]
                    k[bb, h] = k[a, h] + 0.01 * torch.randn((cfg.cancel_pairs, d), generator=gen,
                                                            device=device)
                    v[bb, h] = -v[a, h]
            q_all[li, b * w:(b + 1) * w] = q.to(cfg.dtype)
            k_all[li, t0:t0 + n] = k.to(cfg.dtype)
            v_all[li, t0:t0 + n] = v.to(cfg.dtype)
            ret_l.append(ret)
            ndl_l.append(ndl_b)
            del q, k, v
        retrieval.append(ret_l)
        needles.append(ndl_l)
    return dict(q_win=q_all, k=k_all, v=v_all, cu_seqlens=cu, n_keep=cfg.n_keep(),
                retrieval=retrieval, needles=needles, layers=lay, cfg=cfg)


def make_queries(cfg: CacheConfig, tq: int, device="cpu", layers=None, seed_offset=7919):
    """`tq` new (future) queries per sequence, [L][B*tq][Hq][d] in cfg.dtype:
    standard normal like the window queries, from a stream of their own keyed
    by (seed, layer)."""
    L, H, G, d = cfg.layers, cfg.kv_heads, cfg.group, cfg.head_dim
    lay = list(range(L)) if layers is None else list(layers)
    out = torch.empty((len(lay), cfg.batch * tq, H * G, d), dtype=cfg.dtype, device=device)
    for li, l in enumerate(lay):
        gen = torch.Generator(device=device)
        gen.manual_seed((cfg.seed + seed_offset) * 1_000_003 + l)
        out[li] = torch.randn((cfg.batch * tq, H * G, d), generator=gen, device=device).to(cfg.dtype)
    return out
