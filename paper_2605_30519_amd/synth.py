"""Seeded synthetic inputs for the OmniMem attention step.

Shared by the tests, the smoke check and the benchmark; it holds none of the
method's arithmetic (no pooling, scoring, selection or attention), only random
draws and the paged data layout.

Shapes follow Wan2.1 at 480p: a latent frame is 30 x 52 = 1560 tokens and a chunk
is 3 latent frames (S = Lq = 4680), 12 heads of dimension 128 for the 1.3B model,
40 heads for the 14B model.  Values:
  Q, K, V ~ N(0, 1) i.i.d. (drawn in fp32, then rounded to the storage dtype);
  per-block key offset: every token of block b of head h gets + 0.5 * u[b, h],
    u ~ N(0, I_d), so block means are separable;
  planted relevance (large workloads): per (head, query group) a unit direction
    a[h, r]; queries of group r get + a[h, r] (alpha = 1); a relevant set
    Rel[h, r] = the first K ids of a random permutation of all block ids up to the
    workload's longest history, and every token of a block in Rel[h, r] gets
    + 0.5 * sqrt(d) * a[h, r] on its key.  Heads therefore select different sets.
Every draw comes from its own torch.Generator seeded from (workload, layer,
stream, index), so a chunk can be generated on its own and caches can grow.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Iterable, Optional

import torch

from .omnimem import PagedKVCache


@dataclass(frozen=True)
class Workload:
    name: str
    heads: int
    head_dim: int
    chunk_tokens: int
    query_tokens: int
    block_size: int
    history_chunks: int
    max_history_chunks: int
    top_k: int
    group_size: int
    window_chunks: int
    awe_min_outside_chunks: int
    dtype: torch.dtype
    planted: bool
    layers: int = 1
    seed_id: int = 0

    @property
    def blocks_per_chunk(self) -> int:
        return -(-self.chunk_tokens // self.block_size)

    @property
    def groups(self) -> int:
        return -(-self.query_tokens // self.group_size)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def with_history(self, n: int) -> "Workload":
        return replace(self, history_chunks=n)


# The benchmarked workloads (one attention layer unless `layers` says otherwise).
WORKLOADS = {
    # tiny fp32 correctness case: 2 heads x 64, chunks of 256 tokens, 8 chunks of history
    "tiny_fp32": Workload("tiny_fp32", 2, 64, 256, 256, 64, 8, 8, 4, 256, 1, 3, torch.float32, False, 1, 1),
    # Wan2.1-1.3B layer: 12 x 128, 4680-token chunks, 20 chunks (93,600 keys), K = 64
    "wan1.3b_n20": Workload("wan1.3b_n20", 12, 128, 4680, 4680, 64, 20, 20, 64, 4680, 1, 3, torch.bfloat16, True,
                            1, 2),
    # long rollout: same layer with up to 120 chunks (561,600 keys); swept over 10/30/60/120
    "wan1.3b_long": Workload("wan1.3b_long", 12, 128, 4680, 4680, 64, 120, 120, 64, 4680, 1, 3, torch.bfloat16,
                             True, 1, 3),
    # full chunk step: 30 layers, history ramping 1 -> 60 chunks
    "wan1.3b_30layer": Workload("wan1.3b_30layer", 12, 128, 4680, 4680, 64, 60, 60, 64, 4680, 1, 3, torch.bfloat16,
                                True, 30, 4),
    # Wan2.1-14B-shaped stress layer: 40 x 128, B = 128, K = 32, one group per latent frame
    "wan14b_stress": Workload("wan14b_stress", 40, 128, 4680, 4680, 128, 60, 60, 32, 1560, 1, 3, torch.bfloat16, True,
                              1, 5),
}


def _seed(w: Workload, layer: int, stream: int, index: int) -> int:
    return ((((w.seed_id * 1_000_003) + layer) * 11 + stream) * 1_000_003 + index) % (2**63 - 1)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


@dataclass
class Relevance:
    directions: torch.Tensor  # [H, R, d] unit vectors (fp32)
    relevant: torch.Tensor    # [H, R, max_blocks] bool


def relevance(w: Workload, layer: int, device) -> Optional[Relevance]:
    if not w.planted:
        return None
    H, R, d = w.heads, w.groups, w.head_dim
    nbmax = w.max_history_chunks * w.blocks_per_chunk
    g = _gen(_seed(w, layer, 0, 0), device)
    a = torch.randn((H, R, d), generator=g, device=device)
    a = a / a.norm(dim=-1, keepdim=True)
    rel = torch.zeros((H, R, nbmax), dtype=torch.bool, device=device)
    for h in range(H):
        for r in range(R):
            rel[h, r, torch.randperm(nbmax, generator=g, device=device)[: w.top_k]] = True
    return Relevance(a, rel)


def key_chunk(w: Workload, layer: int, c: int, rel: Optional[Relevance], device) -> torch.Tensor:
    """Keys of history chunk c, [S, H, d] in the workload dtype."""
    S, H, d, B, Bpc = w.chunk_tokens, w.heads, w.head_dim, w.block_size, w.blocks_per_chunk
    g = _gen(_seed(w, layer, 1, c), device)
    k = torch.randn((S, H, d), generator=g, device=device)
    u = torch.randn((Bpc, H, d), generator=g, device=device)
    tok_block = torch.arange(S, device=device) // B
    k += 0.5 * u[tok_block]
    if rel is not None:
        blocks = c * Bpc + torch.arange(Bpc, device=device)
        hit = rel.relevant[:, :, blocks].to(torch.float32)               # [H, R, Bpc]
        add = 0.5 * math.sqrt(d) * torch.einsum("hrb,hrd->bhd", hit, rel.directions)
        k += add[tok_block]
    return k.to(w.dtype)


def value_chunk(w: Workload, layer: int, c: int, device) -> torch.Tensor:
    g = _gen(_seed(w, layer, 2, c), device)
    return torch.randn((w.chunk_tokens, w.heads, w.head_dim), generator=g, device=device).to(w.dtype)


def queries(w: Workload, layer: int, step: int, rel: Optional[Relevance], device) -> torch.Tensor:
    """Queries of the chunk being generated at AR step `step`, [Lq, H, d]."""
    g = _gen(_seed(w, layer, 3, step), device)
    q = torch.randn((w.query_tokens, w.heads, w.head_dim), generator=g, device=device)
    if rel is not None:
        group = torch.arange(w.query_tokens, device=device) // w.group_size
        q += rel.directions.permute(1, 0, 2)[group]
    return q.to(w.dtype)


@dataclass
class LayerInputs:
    q: torch.Tensor   # [Lq, H, d]
    k: torch.Tensor   # [n, S, H, d]   logical history, chunk by chunk
    v: torch.Tensor
    rel: Optional[Relevance]


def make_layer(w: Workload, layer: int = 0, n_chunks: Optional[int] = None, device="cpu", step=None) -> LayerInputs:
    n = w.history_chunks if n_chunks is None else n_chunks
    rel = relevance(w, layer, device)
    k = torch.empty((n, w.chunk_tokens, w.heads, w.head_dim), dtype=w.dtype, device=device)
    v = torch.empty_like(k)
    for c in range(n):
        k[c] = key_chunk(w, layer, c, rel, device)
        v[c] = value_chunk(w, layer, c, device)
    q = queries(w, layer, n if step is None else step, rel, device)
    return LayerInputs(q, k, v, rel)


def page_layer(k: torch.Tensor, v: torch.Tensor, block_size: int, seed: int = 0, pad_value: float = 0.0,
               nonresident: Iterable[int] = (), extra_pages: int = 0) -> PagedKVCache:
    """Lay a logical history [n, S, H, d] out as a paged cache: block b of the
    history goes to a page chosen by a seeded permutation of the pool (so physical
    order differs from logical order); unused slots of each chunk's last page hold
    `pad_value`; blocks listed in `nonresident` get page id -1."""
    n, S, H, d = (int(s) for s in k.shape)
    B = block_size
    Bpc = -(-S // B)
    nblocks = n * Bpc
    num_pages = nblocks + extra_pages
    perm = torch.randperm(max(num_pages, 1), generator=_gen(seed, "cpu"))[:nblocks].to(torch.int32)
    dev = k.device
    k_pages = torch.full((num_pages, H, B, d), pad_value, dtype=k.dtype, device=dev)
    v_pages = torch.full((num_pages, H, B, d), pad_value, dtype=v.dtype, device=dev)
    if nblocks:
        pad = Bpc * B - S
        pidx = perm.to(device=dev, dtype=torch.long)
        for src, dst in ((k, k_pages), (v, v_pages)):
            x = src
            if pad:
                x = torch.cat([x, torch.full((n, pad, H, d), pad_value, dtype=x.dtype, device=dev)], dim=1)
            dst[pidx] = x.reshape(nblocks, B, H, d).permute(0, 2, 1, 3)
    table = perm.clone()
    for b in nonresident:
        table[int(b)] = -1
    table = table.reshape(n, Bpc).to(dev).contiguous()
    return PagedKVCache(k_pages, v_pages, table, S)


def page_layer_per_head(k: torch.Tensor, v: torch.Tensor, block_size: int, seed: int = 0, pad_value: float = 0.0,
                        nonresident: Optional[dict] = None, extra_pages: int = 0) -> PagedKVCache:
    """Like page_layer, with one page table per head ([H, n, Bpc]): head h's block b
    goes to the (page, h) slab of its own seeded permutation, so one page holds
    blocks of different chunks for different heads.  nonresident: {head: block ids}
    marked -1 in that head's table only."""
    n, S, H, d = (int(s) for s in k.shape)
    B = block_size
    Bpc = -(-S // B)
    nblocks = n * Bpc
    num_pages = nblocks + extra_pages
    dev = k.device
    k_pages = torch.full((num_pages, H, B, d), pad_value, dtype=k.dtype, device=dev)
    v_pages = torch.full((num_pages, H, B, d), pad_value, dtype=v.dtype, device=dev)
    tables = []
    pad = Bpc * B - S
    for h in range(H):
        perm = torch.randperm(max(num_pages, 1), generator=_gen(seed * 1009 + h, "cpu"))[:nblocks].to(torch.int32)
        if nblocks:
            pidx = perm.to(device=dev, dtype=torch.long)
            for src, dst in ((k, k_pages), (v, v_pages)):
                x = src[:, :, h]
                if pad:
                    x = torch.cat([x, torch.full((n, pad, d), pad_value, dtype=x.dtype, device=dev)], dim=1)
                dst[pidx, h] = x.reshape(nblocks, B, d)
        t = perm.clone()
        for b in (nonresident or {}).get(h, ()):
            t[int(b)] = -1
        tables.append(t.reshape(n, Bpc))
    return PagedKVCache(k_pages, v_pages, torch.stack(tables).to(dev).contiguous(), S)


def resident_mask(cache: PagedKVCache, n_chunks: Optional[int] = None) -> torch.Tensor:
    """[n*Bpc] bool (shared table) or [H, n*Bpc] (per-head tables), True where the
    page table holds a page (host tensor)."""
    t = cache.page_table.cpu()
    if t.dim() == 3:
        if n_chunks is not None:
            t = t[:, :n_chunks]
        t = t.reshape(t.shape[0], -1)
        return (t >= 0) & (t < cache.k_pages.shape[0])
    if n_chunks is not None:
        t = t[:n_chunks]
    return (t.reshape(-1) >= 0) & (t.reshape(-1) < cache.k_pages.shape[0])
