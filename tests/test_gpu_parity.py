"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Small shapes are compared element by element on every output; the full-size
workloads are compared on the complete selection (every head and group; four of
the thirty layers of the ramp) and on sampled attention rows the oracle computes
one by one.
Inputs are the seeded synthetic workloads; the oracle always receives host copies
of exactly the values the GPU consumed (logical, unpaged layout), while the GPU
reads a paged cache whose pages are shuffled, whose tail slots hold NaN and which
may contain non-resident blocks.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_30519_amd import (omnimem_dense_attn, omnimem_select, omnimem_sparse_attn,
                                  omnimem_union_gather_attn, synth)
from parity import (check_bf16, check_f32, check_lse, check_selection, say)

pytestmark = pytest.mark.gpu
NAN = float("nan")


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def host(x):
    return x.detach().cpu()


def sample_rows(H, Lq, m, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, H, m).astype(np.int32), rng.integers(0, Lq, m).astype(np.int32)


def run_select(cache, x, w, n=None):
    sel = omnimem_select(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                         num_chunks=n)
    torch.cuda.synchronize()
    return sel


def oracle_select(x, w, n, resident=None, heads=None):
    return oracle.select(host(x.q), host(x.k[:n]), w.block_size, w.top_k, w.group_size, w.window_chunks,
                         w.awe_min_outside_chunks, w.scale, resident=resident, heads=heads, want_all_scores=True)


def attn_check(got_out, got_lse, ref_out, ref_lse, hs, qs, dtype, what):
    o = host(got_out).float().numpy()[qs, hs]
    lse = host(got_lse).numpy()[hs, qs]
    if dtype == torch.float32:
        check_f32(o, ref_out, what)
        check_lse(lse, ref_lse, what + " lse", 1e-5)
    else:
        check_bf16(o, ref_out, what)
        check_lse(lse, ref_lse, what + " lse", 5e-3)


# ----------------------------------------------------------------- tiny fp32

def test_tiny_fp32_every_history_length(dev):
    w = synth.WORKLOADS["tiny_fp32"]
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=11, pad_value=NAN)
    for n in range(0, w.history_chunks + 1):
        say(f"tiny_fp32 n={n}: select / sparse / dense")
        sel = run_select(cache, x, w, n)
        ref = oracle_select(x, w, n)
        assert sel.awe_active == int(ref["awe"]) == int(n >= 4)
        check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
        if ref["awe"]:  # selected blocks avoid the window exactly when exclusion is on
            assert (host(sel.idx).numpy() < (n - w.window_chunks) * w.blocks_per_chunk).all()
        out, lse = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale, num_chunks=n)
        o_ref, l_ref, hs, qs = oracle.sparse_attn(host(x.q), host(x.k[:n]), host(x.v[:n]), w.block_size, ref["idx"],
                                                  ref["cnt"], w.group_size, w.scale)
        attn_check(out, lse, o_ref, l_ref, hs, qs, w.dtype, f"sparse n={n}")
        for c0 in {0, max(n - w.window_chunks, 0)}:
            dout, dlse = omnimem_dense_attn(cache, x.q, c0, n, w.scale, num_chunks=n)
            d_ref, dl_ref, hs, qs = oracle.dense_attn(host(x.q), host(x.k[:n]), host(x.v[:n]), w.block_size, c0, n,
                                                      w.scale)
            attn_check(dout, dlse, d_ref, dl_ref, hs, qs, w.dtype, f"dense [{c0},{n})")


# ------------------------------------------------- small shapes, every output

SMALL = [
    # H, d, S, Lq, B, n, K, G, E, T, dtype
    (3, 128, 300, 300, 64, 6, 7, 130, 1, 2, torch.bfloat16),   # ragged tail block, 3 groups, ragged tiles
    (2, 64, 200, 333, 64, 5, 5, 333, 1, 3, torch.bfloat16),    # d = 64, one group spanning 3 row tiles
    (2, 128, 300, 257, 128, 4, 3, 100, 1, 2, torch.bfloat16),  # B = 128 (two 64-key halves, 44-token tail)
    (2, 128, 130, 70, 64, 3, 2, 1, 1, 1, torch.bfloat16),      # per-query selection (G = 1, R = 70)
    (2, 128, 300, 300, 64, 5, 4, 15, 1, 3, torch.bfloat16),    # the paper's G = 15 (R = 20)
    (2, 128, 300, 1000, 64, 14, 4, 15, 1, 3, torch.bfloat16),  # G = 15, R = 67: tiled scoring, ragged tiles
    (2, 128, 300, 100, 128, 4, 3, 40, 0, 0, torch.float32),    # fp32, d = 128, B = 128, no window
    (1, 64, 64, 1, 64, 3, 2, 1, 2, 0, torch.float32),          # one query row, exact-block chunks
    (2, 64, 200, 100, 64, 5, 4, 15, 1, 3, torch.bfloat16),     # bf16, d = 64, groups of at most 32 rows (one wave per group)
    (3, 64, 200, 30, 64, 5, 4, 30, 1, 2, torch.bfloat16),      # bf16, d = 64, Lq <= 32: dense, one wave per group
    (2, 128, 130, 20, 64, 4, 3, 7, 1, 1, torch.bfloat16),      # bf16, d = 128, Lq <= 32: dense, one wave per group
    (2, 64, 300, 130, 128, 4, 3, 65, 1, 2, torch.bfloat16),    # bf16, d = 64, B = 128, groups of 65 rows
]


@pytest.mark.parametrize("H,d,S,Lq,B,n,K,G,E,T,dtype", SMALL)
def test_small_shapes_every_output(dev, H, d, S, Lq, B, n, K, G, E, T, dtype):
    say(f"small H={H} d={d} S={S} Lq={Lq} B={B} n={n} K={K} G={G} E={E} T={T} {dtype}")
    w = synth.Workload("small", H, d, S, Lq, B, n, n, K, G, E, T, dtype, dtype == torch.bfloat16, 1, 7)
    x = synth.make_layer(w, 0, device=dev)
    Bpc = w.blocks_per_chunk
    nonres = [1, n * Bpc - 2] if n * Bpc > 4 else []
    cache = synth.page_layer(x.k, x.v, B, seed=3, pad_value=NAN, nonresident=nonres, extra_pages=5)
    resident = synth.resident_mask(cache).numpy()
    sel = run_select(cache, x, w)
    ref = oracle_select(x, w, n, resident=resident)
    assert sel.awe_active == int(ref["awe"])
    check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
    assert not np.isin(host(sel.idx).numpy(), nonres).any()
    got_score = host(sel.score).numpy()
    want = np.where(ref["idx"] >= 0, ref["score"], -np.inf)
    fin = np.isfinite(want)
    assert np.allclose(got_score[fin], want[fin], rtol=1e-4, atol=1e-5) and np.isneginf(got_score[~fin]).all()

    out, lse = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, G, w.scale)
    o_ref, l_ref, hs, qs = oracle.sparse_attn(host(x.q), host(x.k), host(x.v), B, ref["idx"], ref["cnt"], G, w.scale,
                                              resident=resident)
    attn_check(out, lse, o_ref, l_ref, hs, qs, dtype, "sparse")
    for c0, c1 in [(0, n), (n - 1, n), (1, n - 1)]:
        dout, dlse = omnimem_dense_attn(cache, x.q, c0, c1, w.scale)
        d_ref, dl_ref, hs, qs = oracle.dense_attn(host(x.q), host(x.k), host(x.v), B, c0, c1, w.scale,
                                                  resident=resident)
        attn_check(dout, dlse, d_ref, dl_ref, hs, qs, dtype, f"dense [{c0},{c1})")
    # the union-gather comparator reproduces sparse attention bit for bit
    uout, ulse, ub = omnimem_union_gather_attn(cache, x.q, sel.idx, sel.cnt, G, w.scale)
    torch.cuda.synchronize()
    per, tot = oracle.union(host(sel.idx).numpy(), host(sel.cnt).numpy(), n * Bpc)
    assert int(ub.item()) == tot
    assert torch.equal(uout.view(torch.int16) if dtype == torch.bfloat16 else uout.view(torch.int32),
                       out.view(torch.int16) if dtype == torch.bfloat16 else out.view(torch.int32))
    assert torch.equal(ulse, lse)


# ------------------------------------------------------------- edge cases

def test_edge_cases(dev):
    w = synth.Workload("edge", 2, 128, 200, 150, 64, 4, 4, 5, 50, 1, 1, torch.bfloat16, False, 1, 8)
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, 64, seed=1, pad_value=NAN)
    say("edge: empty history")
    sel = run_select(cache, x, w, 0)
    assert (host(sel.cnt) == 0).all() and (host(sel.idx) == -1).all() and sel.awe_active == 0
    out, lse = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale, num_chunks=0)
    dout, dlse = omnimem_dense_attn(cache, x.q, 0, 0, w.scale, num_chunks=0)
    torch.cuda.synchronize()
    for o, l in ((out, lse), (dout, dlse)):
        assert (host(o).float() == 0).all() and torch.isneginf(host(l)).all()

    say("edge: K larger than the history")
    big = synth.Workload("edge", 2, 128, 200, 150, 64, 4, 4, 100, 50, 1, 1, torch.bfloat16, False, 1, 8)
    sel = run_select(cache, x, big)
    ref = oracle_select(x, big, 4)
    assert not ref["awe"] and (host(sel.cnt) == 16).all()
    check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
    out, lse = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, big.group_size, big.scale)
    dout, dlse = omnimem_dense_attn(cache, x.q, 0, 4, big.scale)
    torch.cuda.synchronize()
    # all blocks selected in ascending order: same tiles in the same order as dense
    assert torch.equal(out.view(torch.int16), dout.view(torch.int16)) and torch.equal(lse, dlse)

    say("edge: caller lists with duplicates, padding inside, out-of-range ids")
    R = -(-150 // 50)
    idx = torch.tensor([[[3, 3, -1, 9, 99, 2]] * R] * 2, dtype=torch.int32, device=dev)
    cnt = torch.full((2, R), 6, dtype=torch.int32, device=dev)
    out, lse = omnimem_sparse_attn(cache, x.q, idx, cnt, 50, w.scale)
    ref_idx = np.array([[[3, 3, 9, 2]] * R] * 2, dtype=np.int32)
    o_ref, l_ref, hs, qs = oracle.sparse_attn(host(x.q), host(x.k), host(x.v), 64, ref_idx, np.full((2, R), 4),
                                              50, w.scale)
    attn_check(out, lse, o_ref, l_ref, hs, qs, torch.bfloat16, "caller list")

    say("edge: every block non-resident")
    cold = synth.page_layer(x.k, x.v, 64, seed=1, nonresident=range(16))
    sel = run_select(cold, x, w)
    assert (host(sel.cnt) == 0).all()
    dout, dlse = omnimem_dense_attn(cold, x.q, 0, 4, w.scale)
    torch.cuda.synchronize()
    assert (host(dout).float() == 0).all() and torch.isneginf(host(dlse)).all()

    say("edge: determinism")
    a1 = run_select(cache, x, w)
    a2 = run_select(cache, x, w)
    assert torch.equal(a1.idx, a2.idx) and torch.equal(a1.score, a2.score)
    o1, l1 = omnimem_sparse_attn(cache, x.q, a1.idx, a1.cnt, w.group_size, w.scale)
    o2, l2 = omnimem_sparse_attn(cache, x.q, a1.idx, a1.cnt, w.group_size, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)


# ------------------------------------------------------- running-max jumps

def test_running_max_jumps(dev):
    """Blocks whose scores jump far above and below the running max, in both list
    orders: the bf16 kernel's speculative exponentials must settle every jump
    (finite overshoot: rescale; overflow: recompute from the keys still in LDS)."""
    H, d, S, Lq, B, n = 2, 128, 256, 300, 64, 4
    g = torch.Generator().manual_seed(11)
    u = torch.randn(H, d, generator=g)
    u = u / u.norm(dim=-1, keepdim=True)
    q = (3.0 * u[None] + 0.3 * torch.randn(Lq, H, d, generator=g)).to(torch.bfloat16)
    nb = n * (S // B)
    # per-block key scale: scaled scores about 0.8 m, so m = 40 overshoots the running
    # max by ~46 in log2 units and m = 400 by ~460 (an overflow without settling)
    m = torch.tensor([1.0, 40.0, 1.0, 0.5, 400.0, 2.0, 0.25, 60.0, 1.0, 3.0, 400.0, 1.0, 0.1, 8.0, 1.0, 50.0])[:nb]
    k = (u[None, None] * 3.0 + 0.3 * torch.randn(n, S, H, d, generator=g))
    k = k * m.repeat_interleave(B).view(n, S, 1, 1)
    k = k.to(torch.bfloat16)
    v = torch.randn(n, S, H, d, generator=g).to(torch.bfloat16)
    scale = d ** -0.5
    cache = synth.page_layer(k.to(dev), v.to(dev), B, seed=5, pad_value=NAN)
    qd = q.to(dev)
    say("jumps: dense over all blocks (ascending order)")
    dout, dlse = omnimem_dense_attn(cache, qd, 0, n, scale)
    d_ref, dl_ref, hs, qs = oracle.dense_attn(q, k, v, B, 0, n, scale)
    attn_check(dout, dlse, d_ref, dl_ref, hs, qs, torch.bfloat16, "jumps dense")
    for name, order in (("descending scale", torch.argsort(m, descending=True)),
                        ("ascending scale", torch.argsort(m)),
                        ("shuffled", torch.randperm(nb, generator=g))):
        say(f"jumps: sparse, blocks in {name} order")
        ids = order.to(torch.int32)
        idx = ids.view(1, 1, nb).expand(H, 1, nb).contiguous().to(dev)
        cnt = torch.full((H, 1), nb, dtype=torch.int32, device=dev)
        out, lse = omnimem_sparse_attn(cache, qd, idx, cnt, Lq, scale)
        o_ref, l_ref, hs, qs = oracle.sparse_attn(q, k, v, B, idx.cpu().numpy(), cnt.cpu().numpy(), Lq, scale)
        attn_check(out, lse, o_ref, l_ref, hs, qs, torch.bfloat16, f"jumps sparse {name}")


def test_partial_first_tile(dev):
    """The 64-row kernel takes its running max from the first tile's own scores: a
    list that starts with a chunk's ragged tail block (8 valid tokens, NaN padding
    after them) must set that max from the valid keys only, and the later tiles,
    below it and then far above it, must still match the oracle."""
    H, d, S, Lq, B, n = 2, 128, 200, 300, 64, 3   # 4 blocks per chunk, the last with 8 tokens
    g = torch.Generator().manual_seed(21)
    q = (0.5 * torch.randn(Lq, H, d, generator=g)).to(torch.bfloat16)
    k = torch.randn(n, S, H, d, generator=g)
    k[0, 192:] *= 4.0     # chunk 0's tail block: the first tile's scores, above the next blocks'
    k[2, :64] *= 16.0     # chunk 2's first block: a jump far above them
    k = k.to(torch.bfloat16)
    v = torch.randn(n, S, H, d, generator=g).to(torch.bfloat16)
    scale = d ** -0.5
    cache = synth.page_layer(k.to(dev), v.to(dev), B, seed=9, pad_value=NAN)
    qd = q.to(dev)
    for ids in ([3, 0, 5, 8, 1, 11, 6], [3], [7, 3, 11]):
        say(f"partial first tile: list {ids}")
        idx = torch.tensor(ids, dtype=torch.int32).view(1, 1, -1).expand(H, 1, len(ids)).contiguous().to(dev)
        cnt = torch.full((H, 1), len(ids), dtype=torch.int32, device=dev)
        out, lse = omnimem_sparse_attn(cache, qd, idx, cnt, Lq, scale)
        o_ref, l_ref, hs, qs = oracle.sparse_attn(q, k, v, B, idx.cpu().numpy(), cnt.cpu().numpy(), Lq, scale)
        attn_check(out, lse, o_ref, l_ref, hs, qs, torch.bfloat16, f"partial first tile {ids}")



def test_long_sparse_lists(dev):
    """Lists longer than one decoded stretch of the 64-row kernel (256 entries):
    the first stretch's entries are read before the list's count, later ones after
    it.  Padding, non-resident blocks and duplicates sit on both
    sides of entry 256; the heads' counts end the list in the second stretch at two
    places, exactly at its start (256), and one head's list is all padding."""
    H, d, S, Lq, B, n = 4, 128, 640, 100, 64, 40   # 10 full blocks per chunk, 400 blocks
    nb = n * (S // B)
    g = torch.Generator().manual_seed(33)
    q = (0.5 * torch.randn(Lq, H, d, generator=g)).to(torch.bfloat16)
    k = torch.randn(n, S, H, d, generator=g).to(torch.bfloat16)
    v = torch.randn(n, S, H, d, generator=g).to(torch.bfloat16)
    scale = d ** -0.5
    nonres = [7, 250, 333]
    cache = synth.page_layer(k.to(dev), v.to(dev), B, seed=4, nonresident=nonres)
    resident = synth.resident_mask(cache).numpy()
    rng = np.random.default_rng(5)
    top_k = 300
    idx = np.full((H, 1, top_k), -1, np.int32)
    for h in range(H):
        ids = rng.permutation(nb)[:top_k].astype(np.int32)
        ids[[3, 255, 256, 290]] = -1          # padding on both sides of entry 256
        ids[[100, 258]] = nonres[h % 3]       # non-resident
        ids[[200, 259]] = ids[50]             # duplicates of a valid id
        idx[h, 0] = ids if h < 3 else -1     # head 3: nothing but padding
    cnt = np.array([[300], [270], [256], [300]], np.int32)
    idx_d, cnt_d = torch.from_numpy(idx).to(dev), torch.from_numpy(cnt).to(dev)
    out, lse = omnimem_sparse_attn(cache, q.to(dev), idx_d, cnt_d, Lq, scale)
    o_ref, l_ref, hs, qs = oracle.sparse_attn(q, k, v, B, idx, cnt, Lq, scale, resident=resident)
    attn_check(out, lse, o_ref, l_ref, hs, qs, torch.bfloat16, "long sparse lists")


# ------------------------------------------------------------- long block lists

@pytest.mark.parametrize("n,zero_q,K", [(5000, True, 64), (5000, False, 64), (20000, False, 64), (20000, True, 64),
                                        (33000, False, 64), (33000, True, 64), (20000, False, 16), (33000, True, 16),
                                        (33000, False, 3)])
def test_long_lists_and_ties(dev, n, zero_q, K):
    """Top-K over long block lists: 5000 blocks spread over several key partitions of
    the register-resident search (512 threads), 20000 blocks need the 1024-thread
    register search, 33000 blocks take the streaming search; with K <= 16 the
    one-wave-per-row kernel walks all of them.  Zero queries make every score
    exactly 0, so the lowest candidate ids must be chosen."""
    say(f"long list n={n} zero_q={zero_q} K={K}")
    w = synth.Workload("long", 1, 64, 64, 8, 64, n, n, K, 8, 1, 1, torch.bfloat16, False, 1, 9)
    g = torch.Generator(device=dev).manual_seed(17 + n)
    k = torch.randn((n, 64, 1, 64), generator=g, device=dev).to(torch.bfloat16)
    q = torch.randn((8, 1, 64), generator=g, device=dev).to(torch.bfloat16)
    if zero_q:
        q.zero_()
    nonres = [0, 5, 2047, 2048, n - 3]
    cache = synth.page_layer(k, k, 64, seed=2, nonresident=nonres)
    resident = synth.resident_mask(cache).numpy()
    x = synth.LayerInputs(q=q, k=k, v=k, rel=None)
    sel = run_select(cache, x, w)
    ref = oracle_select(x, w, n, resident=resident)
    got = host(sel.idx).numpy()
    check_selection(got, host(sel.cnt).numpy(), ref)
    if zero_q:
        assert (got == ref["idx"]).all()
        omega = [b for b in range(n - 1) if resident[b]]  # the last chunk is the excluded window
        assert got[0, 0].tolist() == omega[:K]


@pytest.mark.parametrize("d,K,per_head,zero_q", [(64, 10, True, False), (128, 4, False, False), (64, 16, False, True),
                                                  (128, 7, True, True), (64, 3, False, False)])
def test_many_groups_small_k(dev, d, K, per_head, zero_q):
    """Many query groups (R = 75) and K <= 16: scores and top-K in one kernel, with 240
    candidate blocks split over its waves in several 16-block tiles, non-resident
    blocks, per-head tables; zero queries make every score 0, so each group takes its
    K lowest candidate ids."""
    H, S, Lq, B, n, G = 2, 200, 600, 64, 60, 8
    say(f"many groups d={d} K={K} per_head={per_head} zero_q={zero_q}")
    w = synth.Workload("groups", H, d, S, Lq, B, n, n, K, G, 1, 2, torch.bfloat16, True, 1, 13)
    x = synth.make_layer(w, 0, device=dev)
    if zero_q:
        x.q.zero_()
    nb = n * w.blocks_per_chunk
    if per_head:
        cache = synth.page_layer_per_head(x.k, x.v, B, seed=8, nonresident={0: [2, 40, nb - 9], 1: [0, 1]})
    else:
        cache = synth.page_layer(x.k, x.v, B, seed=8, nonresident=[3, 77, 150])
    mask = synth.resident_mask(cache).numpy()
    sel = run_select(cache, x, w)
    got = host(sel.idx).numpy()
    for h in range(H):
        res = mask[h] if mask.ndim == 2 else mask
        ref = oracle.select(host(x.q), host(x.k), B, K, G, 1, 2, w.scale, resident=res, heads=(h, h + 1),
                            want_all_scores=True)
        check_selection(got, host(sel.cnt).numpy(), ref, heads=[h])
        if zero_q:
            omega = [b for b in range(nb - w.blocks_per_chunk) if res[b]]  # the last chunk is the window
            assert (got[h] == np.array(omega[:K], np.int32)).all()


# ------------------------------------------------------------ full-size workloads

def planted_recall(sel, x, w, n):
    """Planted relevance must be found: Rel[h,r] & Omega is selected whenever it fits in K."""
    rel = x.rel.relevant[:, :, : n * w.blocks_per_chunk].cpu().numpy()
    idx = host(sel.idx).numpy()
    Bpc = w.blocks_per_chunk
    missed = 0
    for h in range(w.heads):
        for r in range(w.groups):
            want = set(np.nonzero(rel[h, r])[0].tolist())
            if sel.awe_active:
                want = {b for b in want if b < (n - w.window_chunks) * Bpc}
            if len(want) <= w.top_k:
                missed += len(want - set(idx[h, r].tolist()))
    return missed


def test_wan13b_n20(dev):
    w = synth.WORKLOADS["wan1.3b_n20"]
    say("wan1.3b_n20: generate")
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=21, pad_value=NAN)
    sel = run_select(cache, x, w)
    say("wan1.3b_n20: oracle select (all heads)")
    ref = oracle_select(x, w, w.history_chunks)
    assert sel.awe_active == 1
    ties = check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
    say(f"  selection matches ({ties} near-tie rows)")
    assert planted_recall(sel, x, w, w.history_chunks) == 0
    out, lse = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale)
    hs, qs = sample_rows(w.heads, w.query_tokens, 384, 1)
    o_ref, l_ref, _, _ = oracle.sparse_attn(host(x.q), host(x.k), host(x.v), w.block_size, ref["idx"], ref["cnt"],
                                            w.group_size, w.scale, hs=hs, qs=qs)
    attn_check(out, lse, o_ref, l_ref, hs, qs, w.dtype, "sparse (384 sampled rows)")
    dout, dlse = omnimem_dense_attn(cache, x.q, 0, w.history_chunks, w.scale)
    hs, qs = sample_rows(w.heads, w.query_tokens, 32, 2)
    d_ref, dl_ref, _, _ = oracle.dense_attn(host(x.q), host(x.k), host(x.v), w.block_size, 0, w.history_chunks,
                                            w.scale, hs=hs, qs=qs)
    attn_check(dout, dlse, d_ref, dl_ref, hs, qs, w.dtype, "dense (32 sampled rows)")


def test_wan13b_long_sweep(dev):
    w = synth.WORKLOADS["wan1.3b_long"]
    say("wan1.3b_long: generate 120 chunks")
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=31, pad_value=NAN)
    kh, vh = host(x.k), host(x.v)
    for n in (10, 30, 60, 120):
        say(f"wan1.3b_long n={n}: select, oracle over all heads")
        xn = synth.LayerInputs(synth.queries(w, 0, n, x.rel, dev), x.k, x.v, x.rel)
        sel = run_select(cache, xn, w, n)
        ref = oracle.select(host(xn.q), kh[:n], w.block_size, w.top_k, w.group_size, w.window_chunks,
                            w.awe_min_outside_chunks, w.scale, want_all_scores=True)
        ties = check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
        say(f"  selection matches ({ties} near-tie rows)")
        assert sel.awe_active == 1 and planted_recall(sel, xn, w, n) == 0
        out, lse = omnimem_sparse_attn(cache, xn.q, sel.idx, sel.cnt, w.group_size, w.scale, num_chunks=n)
        hs, qs = sample_rows(w.heads, w.query_tokens, 96, n)
        o_ref, l_ref, _, _ = oracle.sparse_attn(host(xn.q), kh[:n], vh[:n], w.block_size, ref["idx"], ref["cnt"],
                                                w.group_size, w.scale, hs=hs, qs=qs)
        attn_check(out, lse, o_ref, l_ref, hs, qs, w.dtype, f"sparse n={n}")
        if n in (10, 120):
            dout, dlse = omnimem_dense_attn(cache, xn.q, 0, n, w.scale, num_chunks=n)
            hs, qs = sample_rows(w.heads, w.query_tokens, 8, n + 1)
            d_ref, dl_ref, _, _ = oracle.dense_attn(host(xn.q), kh[:n], vh[:n], w.block_size, 0, n, w.scale, hs=hs,
                                                    qs=qs)
            attn_check(dout, dlse, d_ref, dl_ref, hs, qs, w.dtype, f"dense n={n}")


@pytest.mark.parametrize("layer", [0, 9, 19, 29])
def test_wan13b_30layer_ramp_sampled(dev, layer):
    """Four of the thirty layers (independent seeds), every head, at the history
    lengths around the exclusion switch and at the end of the ramp."""
    w = synth.WORKLOADS["wan1.3b_30layer"]
    say(f"wan1.3b_30layer layer={layer}: generate 60 chunks")
    x = synth.make_layer(w, layer, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=100 + layer, pad_value=NAN)
    kh, vh = host(x.k), host(x.v)
    for n in (1, 2, 3, 4, 5, 30, 60):
        say(f"  layer={layer} n={n}")
        xn = synth.LayerInputs(synth.queries(w, layer, n, x.rel, dev), x.k, x.v, x.rel)
        sel = run_select(cache, xn, w, n)
        assert sel.awe_active == int(n >= 4)
        ref = oracle.select(host(xn.q), kh[:n], w.block_size, w.top_k, w.group_size, w.window_chunks,
                            w.awe_min_outside_chunks, w.scale, want_all_scores=True)
        check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
        idx = host(sel.idx).numpy()
        win0 = (n - w.window_chunks) * w.blocks_per_chunk
        if sel.awe_active:
            assert (idx < win0).all()
        assert planted_recall(sel, xn, w, n) == 0
        if n in (4, 60):
            out, lse = omnimem_sparse_attn(cache, xn.q, sel.idx, sel.cnt, w.group_size, w.scale, num_chunks=n)
            hs, qs = sample_rows(w.heads, w.query_tokens, 64, n)
            o_ref, l_ref, _, _ = oracle.sparse_attn(host(xn.q), kh[:n], vh[:n], w.block_size, ref["idx"], ref["cnt"],
                                                    w.group_size, w.scale, hs=hs, qs=qs)
            attn_check(out, lse, o_ref, l_ref, hs, qs, w.dtype, f"sparse layer={layer} n={n}")
    del x, cache
    torch.cuda.empty_cache()


def test_wan14b_stress(dev):
    w = synth.WORKLOADS["wan14b_stress"]
    say("wan14b_stress: generate 60 chunks x 40 heads")
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=51, pad_value=NAN)
    sel = run_select(cache, x, w)
    say("wan14b_stress: oracle select over all 40 heads")
    kh, vh = host(x.k), host(x.v)
    ref = oracle.select(host(x.q), kh, w.block_size, w.top_k, w.group_size, w.window_chunks,
                        w.awe_min_outside_chunks, w.scale, want_all_scores=True)
    ties = check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
    say(f"  selection matches ({ties} near-tie rows)")
    assert planted_recall(sel, x, w, w.history_chunks) == 0
    out, lse = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale)
    hs, qs = sample_rows(w.heads, w.query_tokens, 160, 5)
    o_ref, l_ref, _, _ = oracle.sparse_attn(host(x.q), kh, vh, w.block_size, ref["idx"], ref["cnt"], w.group_size,
                                            w.scale, hs=hs, qs=qs)
    attn_check(out, lse, o_ref, l_ref, hs, qs, w.dtype, "sparse (96 sampled rows)")
    say("wan14b_stress: union gather")
    uout, ulse, ub = omnimem_union_gather_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale)
    torch.cuda.synchronize()
    nb = w.history_chunks * w.blocks_per_chunk
    per, tot = oracle.union(host(sel.idx).numpy(), host(sel.cnt).numpy(), nb)
    omega = nb - w.window_chunks * w.blocks_per_chunk
    say(f"  union {tot} of {omega} candidate blocks ({100.0 * tot / omega:.1f}%), sum_h |U_h| = {int(per.sum())}")
    assert int(ub.item()) == tot and tot > 0.8 * omega
    assert torch.equal(uout.view(torch.int16), out.view(torch.int16)) and torch.equal(ulse, lse)


def test_per_head_page_tables(dev):
    """The same layer paged with one table per head (each head's blocks on pages of
    its own permutation, so a page holds different chunks for different heads):
    selection, sparse, dense and union-free outputs equal the shared-table ones bit
    for bit, and blocks made non-resident for one head only are skipped for that
    head alone, against the oracle head by head."""
    H, d, S, Lq, B, n, K, G = 3, 128, 300, 300, 64, 6, 7, 130
    w = synth.Workload("perhead", H, d, S, Lq, B, n, n, K, G, 1, 2, torch.bfloat16, True, 1, 7)
    x = synth.make_layer(w, 0, device=dev)
    shared = synth.page_layer(x.k, x.v, B, seed=3, pad_value=NAN)
    per = synth.page_layer_per_head(x.k, x.v, B, seed=4, pad_value=NAN)
    say("per-head tables: same data, other pages")
    a = run_select(shared, x, w)
    b = run_select(per, x, w)
    assert torch.equal(a.idx, b.idx) and torch.equal(a.cnt, b.cnt) and torch.equal(a.score, b.score)
    for cache_pair in ((shared, per),):
        o1, l1 = omnimem_sparse_attn(cache_pair[0], x.q, a.idx, a.cnt, G, w.scale)
        o2, l2 = omnimem_sparse_attn(cache_pair[1], x.q, a.idx, a.cnt, G, w.scale)
        d1, m1 = omnimem_dense_attn(cache_pair[0], x.q, 0, n, w.scale)
        d2, m2 = omnimem_dense_attn(cache_pair[1], x.q, 0, n, w.scale)
        torch.cuda.synchronize()
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
        assert torch.equal(d1.view(torch.int16), d2.view(torch.int16)) and torch.equal(m1, m2)
    from paper_2605_30519_amd import CompressedCache, omnimem_compress_chunk
    c1, c2 = CompressedCache.allocate(shared, n), CompressedCache.allocate(per, n)
    for c in range(n):
        omnimem_compress_chunk(shared, c, c1)
        omnimem_compress_chunk(per, c, c2)
    torch.cuda.synchronize()
    assert torch.equal(c1.k_mean, c2.k_mean) and torch.equal(c1.k_pages.view(torch.int16), c2.k_pages.view(torch.int16))
    say("per-head tables: residency differs by head")
    Bpc = w.blocks_per_chunk
    nonres = {0: [1, 7], 2: [3, n * Bpc - 2]}
    per2 = synth.page_layer_per_head(x.k, x.v, B, seed=4, pad_value=NAN, nonresident=nonres)
    mask = synth.resident_mask(per2).numpy()
    sel = run_select(per2, x, w)
    out, lse = omnimem_sparse_attn(per2, x.q, sel.idx, sel.cnt, G, w.scale)
    dout, dlse = omnimem_dense_attn(per2, x.q, 0, n, w.scale)
    for h in range(H):
        ref = oracle.select(host(x.q), host(x.k), B, K, G, 1, 2, w.scale, resident=mask[h], heads=(h, h + 1),
                            want_all_scores=True)
        check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref, heads=[h])
        assert not np.isin(host(sel.idx).numpy()[h], nonres.get(h, [])).any()
        hs = np.full(Lq, h, np.int32)
        qs = np.arange(Lq, dtype=np.int32)
        o_ref, l_ref, _, _ = oracle.sparse_attn(host(x.q), host(x.k), host(x.v), B, host(sel.idx).numpy(),
                                                host(sel.cnt).numpy(), G, w.scale, resident=mask[h], hs=hs, qs=qs)
        attn_check(out, lse, o_ref, l_ref, hs, qs, torch.bfloat16, f"per-head sparse h={h}")
        d_ref, dl_ref, _, _ = oracle.dense_attn(host(x.q), host(x.k), host(x.v), B, 0, n, w.scale, resident=mask[h],
                                                hs=hs, qs=qs)
        attn_check(dout, dlse, d_ref, dl_ref, hs, qs, torch.bfloat16, f"per-head dense h={h}")


# -------------------------------------------------- groups of at most 32 rows

def _walk_lists(H, R, nb, top_k, seed):
    """Caller lists for the one-wave-per-group walk: lengths 0..top_k, padding, ids
    out of range, duplicates, groups whose every entry is invalid, and lists longer
    than one wave's window of 64 entries."""
    rng = np.random.default_rng(seed)
    idx = np.full((H, R, top_k), -1, np.int32)
    cnt = np.zeros((H, R), np.int32)
    for h in range(H):
        for r in range(R):
            kind = (h * R + r) % 7
            if kind == 0:
                c = 0                                   # empty group
            elif kind == 1:
                c = 5
                idx[h, r, :c] = [-1, nb, nb + 7, -3, -1]  # nothing valid
            else:
                c = int(rng.integers(1, top_k + 1)) if kind != 2 else top_k
                ids = rng.integers(0, nb, c).astype(np.int32)
                ids[rng.random(c) < 0.05] = -1
                idx[h, r, :c] = ids
            cnt[h, r] = c
    return idx, cnt


@pytest.mark.parametrize("d,S,B,per_head", [(128, 200, 128, False), (64, 130, 64, True)])
def test_small_group_walk(dev, d, S, B, per_head):
    """Groups of 8 rows over 4 heads (4100 groups: several per wave of the persistent
    one-wave-per-group kernel, so tiles stream across group boundaries), caller lists
    of up to 96 entries, a partial last block per chunk (8 keys in the second 64-key
    sub-tile at B = 128), non-resident blocks, and per-head tables; sampled rows
    against the oracle, empty groups exactly zero with lse = -inf.  Dense calls of at
    most 32 rows over more than 64 blocks take the same kernel."""
    H, Lq, n, G, top_k = 4, 8200, 40, 8, 96
    w = synth.Workload("walk", H, d, S, Lq, B, n, n, 4, G, 1, 1, torch.bfloat16, False, 1, 9)
    x = synth.make_layer(w, 0, device=dev)
    Bpc = w.blocks_per_chunk
    nb = n * Bpc
    if per_head:
        cache = synth.page_layer_per_head(x.k, x.v, B, seed=6, pad_value=NAN, nonresident={1: [3, 17], 3: [0, nb - 1]})
    else:
        cache = synth.page_layer(x.k, x.v, B, seed=6, pad_value=NAN, nonresident=[5, 11, nb - 2])
    mask = synth.resident_mask(cache).numpy()
    R = -(-Lq // G)
    idx, cnt = _walk_lists(H, R, nb, top_k, seed=d)
    say(f"walk d={d} B={B}: {H * R} groups, lists up to {top_k}")
    out, lse = omnimem_sparse_attn(cache, x.q, torch.from_numpy(idx).to(dev), torch.from_numpy(cnt).to(dev), G,
                                   w.scale)
    torch.cuda.synchronize()
    o, l = host(out).float().numpy(), host(lse).numpy()
    # every group whose list holds no resident block: zero output, lse -inf
    for h in range(H):
        m = mask[h] if mask.ndim == 2 else mask
        for r in range(R):
            ids = idx[h, r, :cnt[h, r]]
            if not any(0 <= b < nb and m[b] for b in ids):
                rows = slice(r * G, min(r * G + G, Lq))
                assert (o[rows, h] == 0).all() and np.isneginf(l[h, rows]).all(), (h, r)
    # sampled rows, group kinds mixed, head by head (per-head residency); the oracle
    # takes ids past the history as padding, which is what the kernel does with them
    idx_ref = np.where(idx >= nb, -1, idx)
    rng = np.random.default_rng(d + 1)
    for h in range(H):
        qs = np.unique(np.concatenate([rng.integers(0, Lq, 120), np.arange(Lq - 5, Lq)])).astype(np.int32)
        hs = np.full(qs.shape, h, np.int32)
        res = mask[h] if mask.ndim == 2 else mask
        o_ref, l_ref, _, _ = oracle.sparse_attn(host(x.q), host(x.k), host(x.v), B, idx_ref, cnt, G, w.scale,
                                                resident=res, hs=hs, qs=qs)
        live = np.isfinite(l_ref)
        attn_check(out, lse, o_ref[live], l_ref[live], hs[live], qs[live], torch.bfloat16, f"walk h={h}")
        assert np.isneginf(l[h, qs[~live]]).all()

    say(f"walk d={d} B={B}: dense, 20 query rows over {nb} blocks")
    q20 = x.q[:20].contiguous()
    dout, dlse = omnimem_dense_attn(cache, q20, 0, n, w.scale)
    torch.cuda.synchronize()
    for h in range(H):
        res = mask[h] if mask.ndim == 2 else mask
        hs = np.full(20, h, np.int32)
        qs = np.arange(20, dtype=np.int32)
        d_ref, dl_ref, _, _ = oracle.dense_attn(host(q20), host(x.k), host(x.v), B, 0, n, w.scale, resident=res,
                                                hs=hs, qs=qs)
        attn_check(dout, dlse, d_ref, dl_ref, hs, qs, torch.bfloat16, f"walk dense h={h}")
