"""Parity of the probability-averaged compression score with the fp64 oracle, through
the C ABI: omnimem_select_compressed with score_mode = SCORE_PROB against
oracle.select_prob.  A block's score for a query group is the mean over the group's
rows of each row's softmax probability of the block over every pooled key of the
history (Sec. 3.1, Eq. 3, App. C).

The oracle takes the pooled keys in fp64 from the same stored K (non-resident blocks
pool to zero, as the compressed history stores them).  Id sets must match except at
an oracle near-tie; the scores of the selected blocks must match to 1e-4 relative
(the kernel's logits carry about 2^-16 relative error from its two-piece bf16
split of the pooled keys, fp32 accumulation and the hardware exp2/log2).

Shapes cover both kernel modes: 128-row slices that hold whole groups (G <= 64:
G = 1, 7, 15, 32, 33, 40, 64) and slices that are parts of one group (G >= 65:
one, two, three and 37 parts), several 64-key tiles with a ragged last tile,
d = 64 and 128, B = 64 and 128, bf16 and fp32 queries, ragged last groups and
non-resident blocks.  For bf16 caches the two key pieces come from the compressed
cache's pooled-key and residual pages; the same selection with the pieces split per
call (no residual pages) must be identical bit for bit.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2605_30519_amd import (SCORE_PROB, CompressedCache, omnimem_compress_chunk, omnimem_select,
                                  omnimem_select_compressed, synth)
from parity import check_selection, say
from test_gpu_compressed import oracle_pooled
from test_gpu_parity import host

pytestmark = pytest.mark.gpu
NAN = float("nan")
SCORE_RTOL = 1e-4


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def oracle_prob(x, w, n, resident=None, heads=None, G=None, K=None):
    kbar, _, _ = oracle_pooled(x, w, n, resident)
    return oracle.select_prob(host(x.q), kbar, n, w.blocks_per_chunk, K or w.top_k, G or w.group_size,
                              w.window_chunks, w.awe_min_outside_chunks, w.scale,
                              resident=None if resident is None else resident[: n * w.blocks_per_chunk],
                              heads=heads, want_all_scores=True)


def check_prob(sel, ref, heads=None):
    idx, cnt = host(sel.idx).numpy(), host(sel.cnt).numpy()
    ties = check_selection(idx, cnt, ref, heads=heads)
    score = host(sel.score).numpy().astype(np.float64)
    worst = 0.0
    for h in (range(idx.shape[0]) if heads is None else heads):
        for r in range(idx.shape[1]):
            c = int(cnt[h, r])
            assert np.isneginf(score[h, r, c:]).all()
            if c == 0:
                continue
            want = ref["all_scores"][h, r, idx[h, r, :c]]
            rel = np.abs(score[h, r, :c] - want) / want
            worst = max(worst, float(rel.max()))
    say(f"  scores: max relative error {worst:.2e} ({ties} near-tie rows)")
    assert worst <= SCORE_RTOL, worst
    return worst


PROB_SMALL = [
    # H, d, S, Lq, B, n, K, G, E, T, dtype
    (3, 128, 600, 300, 64, 14, 7, 130, 1, 2, torch.bfloat16),   # two parts per group; last group 40 rows
    (2, 64, 600, 333, 64, 9, 5, 333, 1, 3, torch.bfloat16),     # d = 64, one group in 3 parts
    (2, 128, 600, 257, 128, 9, 3, 100, 1, 2, torch.bfloat16),   # B = 128, 88-token tail block, one part
    (2, 128, 600, 300, 64, 14, 4, 15, 1, 3, torch.bfloat16),    # the paper's G = 15: 8 groups per slice
    (2, 128, 600, 200, 64, 8, 4, 1, 0, 0, torch.bfloat16),      # one row per group: 128 groups per slice
    (2, 128, 600, 97, 64, 8, 4, 32, 0, 0, torch.bfloat16),      # G = 32, last group 1 row
    (2, 128, 600, 100, 64, 8, 4, 33, 1, 2, torch.bfloat16),     # G = 33: 3 groups per slice
    (2, 128, 600, 300, 64, 8, 4, 64, 1, 2, torch.bfloat16),     # G = 64: the largest whole-group mode
    (2, 128, 600, 300, 64, 8, 4, 65, 1, 2, torch.bfloat16),     # G = 65: one part per group
    (2, 128, 600, 100, 128, 9, 3, 40, 0, 0, torch.float32),     # fp32 queries
    (2, 64, 600, 50, 64, 7, 3, 7, 1, 0, torch.float32),         # fp32, d = 64, 18 groups per slice
    (2, 128, 600, 300, 64, 9, 3, 150, 1, 2, torch.float32),     # fp32, two parts per group
    (1, 64, 64, 1, 64, 3, 2, 1, 2, 0, torch.float32),           # one query row, one tile
]


@pytest.mark.parametrize("H,d,S,Lq,B,n,K,G,E,T,dtype", PROB_SMALL)
def test_prob_small(dev, H, d, S, Lq, B, n, K, G, E, T, dtype):
    say(f"prob small H={H} d={d} S={S} Lq={Lq} B={B} n={n} K={K} G={G} {dtype}")
    w = synth.Workload("small", H, d, S, Lq, B, n, n, K, G, E, T, dtype, dtype == torch.bfloat16, 1, 7)
    x = synth.make_layer(w, 0, device=dev)
    Bpc = w.blocks_per_chunk
    nonres = [1, n * Bpc - 2] if n * Bpc > 4 else []
    cache = synth.page_layer(x.k, x.v, B, seed=3, pad_value=NAN, nonresident=nonres, extra_pages=5)
    resident = synth.resident_mask(cache).numpy()
    cc = CompressedCache.allocate(cache, n)
    done = 0
    for c in sorted({1, (n + 1) // 2, n}):
        while done < c:
            omnimem_compress_chunk(cache, done, cc, num_chunks=done + 1)
            done += 1
        say(f"  history n={c} ({c * Bpc} pooled keys)")
        sel = omnimem_select_compressed(cache, cc, x.q, K, G, E, T, w.scale, num_chunks=c, score_mode=SCORE_PROB)
        torch.cuda.synchronize()
        ref = oracle_prob(x, w, c, resident=resident)
        assert sel.awe_active == int(ref["awe"])
        assert not np.isin(host(sel.idx).numpy(), nonres).any()
        check_prob(sel, ref)
        if cc.k_lo is not None:
            check_residual(cc, c * Bpc)
            say("  the same selection with the pooled keys split per call (no residual pages)")
            split = omnimem_select_compressed(cache, dataclasses.replace(cc, k_lo=None), x.q, K, G, E, T, w.scale,
                                              num_chunks=c, score_mode=SCORE_PROB)
            torch.cuda.synchronize()
            assert torch.equal(split.idx, sel.idx) and torch.equal(split.cnt, sel.cnt)
            assert torch.equal(split.score, sel.score)


def check_residual(cc, nb):
    """The residual pages hold bf16(k_mean - bf16(k_mean)) of every pooled token, in
    the pooled-key pages' layout, next to k_pages = bf16(k_mean) (torch rounds fp32
    to bf16 to nearest even, as the kernels do)."""
    H, d = int(cc.k_pages.shape[1]), int(cc.k_pages.shape[3])
    km = cc.k_mean[:, :nb]
    hi = km.to(torch.bfloat16)
    lo = (km - hi.float()).to(torch.bfloat16)
    tokens = lambda t: t.permute(1, 0, 2, 3).reshape(H, -1, d)[:, :nb]
    assert torch.equal(tokens(cc.k_pages), hi)
    assert torch.equal(tokens(cc.k_lo), lo)


def test_prob_edge_cases(dev):
    w = synth.Workload("edge", 2, 128, 200, 150, 64, 4, 4, 5, 50, 1, 1, torch.bfloat16, False, 1, 8)
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, 64, seed=1, pad_value=NAN)
    cc = CompressedCache.allocate(cache, 4)
    say("prob edge: empty history selects nothing")
    sel = omnimem_select_compressed(cache, cc, x.q, 5, 50, 1, 1, w.scale, num_chunks=0, score_mode=SCORE_PROB)
    torch.cuda.synchronize()
    assert (host(sel.cnt) == 0).all() and (host(sel.idx) == -1).all()
    say("prob edge: the full-K path and unknown modes are refused")
    with pytest.raises(Exception):
        omnimem_select_compressed(cache, cc, x.q, 5, 50, 1, 1, w.scale, score_mode=2)
    from paper_2605_30519_amd import omnimem as om
    params = om.select_params(5, 50, 1, 1, w.scale, SCORE_PROB)
    assert om.omnimem_select_workspace_bytes(cache, 150, params) > 0
    with pytest.raises(Exception):
        import ctypes
        desc = cache.descriptor(None)
        ws = om.workspace_tensor(om.omnimem_select_workspace_bytes(cache, 150, params), x.q.device)
        idx = torch.empty((2, 3, 5), dtype=torch.int32, device=dev)
        cnt = torch.empty((2, 3), dtype=torch.int32, device=dev)
        om._check(om.lib().omnimem_select(ctypes.byref(desc), om._ptr(x.q), 150, ctypes.byref(params), om._ptr(idx),
                                          om._ptr(cnt), None, None, om._ptr(ws), ws.numel(), None), "omnimem_select")
    say("prob edge: K covering the history takes every candidate")
    for c in range(4):
        omnimem_compress_chunk(cache, c, cc)
    a = omnimem_select_compressed(cache, cc, x.q, 100, 50, 1, 1, w.scale, score_mode=SCORE_PROB)
    b = omnimem_select(cache, x.q, 100, 50, 1, 1, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(a.idx, b.idx) and torch.equal(a.cnt, b.cnt) and (host(a.cnt) == 16).all()
    say("prob edge: with one row per group the ranking is the logit ranking")
    a = omnimem_select_compressed(cache, cc, x.q, 5, 1, 0, 0, w.scale, score_mode=SCORE_PROB)
    b = omnimem_select_compressed(cache, cc, x.q, 5, 1, 0, 0, w.scale)
    torch.cuda.synchronize()
    same = (a.idx == b.idx).all(dim=-1).float().mean().item()
    say(f"  rows with identical id lists: {same:.4f}")
    assert same > 0.99


@pytest.mark.parametrize("G", [None, 15])
def test_prob_wan13b_n20(dev, G):
    """The 1.3B layer at 20 cached chunks: the workload's one group per head (37
    slices of at most 128 rows) and the paper's G = 15 (312 groups, 8 per slice);
    the oracle checks heads 0 and 1."""
    w = synth.WORKLOADS["wan1.3b_n20"]
    n = w.history_chunks
    group = G or w.group_size
    K = w.top_k if G is None else 4
    say(f"prob wan1.3b_n20 G={group} K={K}")
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=12, pad_value=NAN)
    cc = CompressedCache.allocate(cache, n)
    for c in range(n):
        omnimem_compress_chunk(cache, c, cc, num_chunks=c + 1)
    sel = omnimem_select_compressed(cache, cc, x.q, K, group, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                                    score_mode=SCORE_PROB)
    torch.cuda.synchronize()
    say("  oracle, heads 0-1")
    ref = oracle_prob(x, w, n, heads=(0, 2), G=group, K=K)
    assert sel.awe_active == 1
    check_prob(sel, ref, heads=range(2))
