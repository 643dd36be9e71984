"""Parity of the compressed-history path (App. C's first cache level) and of Eq. 1's
gated three-branch fusion with the fp64 oracle, through the C ABI: chunks pooled
one by one as they are appended (omnimem_compress_chunk), selection from the
pooled keys (omnimem_select_compressed) at every history length, compression
attention over the pooled sequence (omnimem_cmp_attn, Eq. 1's CMP branch), and
the sigmoid-gated sum of the CMP, SLC and SWA branches (omnimem_gated_combine).

The oracle pools the same logical K/V in fp64 (oracle.cmp_cache) and rounds the
pooled tokens to bf16 for a bf16 cache, as the stored pooled sequence is.  A block
whose page is not resident when its chunk is pooled pools to zero by contract.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_30519_amd import (CompressedCache, omnimem_cmp_attn, omnimem_compress_chunk, omnimem_dense_attn,
                                  omnimem_gated_combine, omnimem_select, omnimem_select_compressed,
                                  omnimem_sparse_attn, synth)
from parity import check_bf16, check_f32, check_selection, say
from test_gpu_parity import attn_check, host, oracle_select, sample_rows

pytestmark = pytest.mark.gpu
NAN = float("nan")


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def oracle_pooled(x, w, n, resident=None):
    """Pooled keys in fp64 and the stored pooled K/V (rounded to the cache dtype),
    [H, n*Bpc, d]; non-resident blocks are zero."""
    k, v = host(x.k[:n]), host(x.v[:n])   # the exact stored values; the oracle widens them exactly
    kbar = oracle.pool_keys(k, w.block_size)
    kc, vc = oracle.cmp_cache(k, v, w.block_size, round_to="bf16" if w.dtype == torch.bfloat16 else None)
    if resident is not None:
        gone = ~resident[: n * w.blocks_per_chunk]
        kbar[:, gone] = 0.0
        kc[:, gone] = 0.0
        vc[:, gone] = 0.0
    return kbar, kc, vc


def stored_pooled(cc, ntok):
    """The pooled sequence as stored: [H, ntok, d] float64 for keys and values."""
    def seq(p):
        H, d = p.shape[1], p.shape[3]
        return host(p).float().numpy().astype(np.float64).transpose(1, 0, 2, 3).reshape(H, -1, d)[:, :ntok]
    return seq(cc.k_pages), seq(cc.v_pages)


def check_pooled(cc, x, w, n, resident=None):
    ntok = n * w.blocks_per_chunk
    kbar, kc, vc = oracle_pooled(x, w, n, resident)
    got_mean = host(cc.k_mean).numpy().astype(np.float64)[:, :ntok]
    assert np.allclose(got_mean, kbar, rtol=2e-6, atol=1e-6), np.abs(got_mean - kbar).max()
    gk, gv = stored_pooled(cc, ntok)
    if w.dtype == torch.bfloat16:
        # the kernel rounds its fp32 mean, the oracle its fp64 mean: at most one bf16 step apart
        for got, want in ((gk, kc), (gv, vc)):
            step = np.ldexp(1.0, np.frexp(np.maximum(np.abs(want), 1e-30))[1] - 8)
            assert (np.abs(got - want) <= step).all(), np.abs(got - want).max()
            assert np.mean(got == want) > 0.99
    else:
        assert np.allclose(gk, kc, rtol=2e-6, atol=1e-6) and np.allclose(gv, vc, rtol=2e-6, atol=1e-6)
    return kc, vc


SMALL = [
    # H, d, S, Lq, B, n, K, G, E, T, dtype
    (3, 128, 300, 300, 64, 6, 7, 130, 1, 2, torch.bfloat16),   # ragged tail block, 3 groups
    (2, 64, 200, 333, 64, 5, 5, 333, 1, 3, torch.bfloat16),    # d = 64
    (2, 128, 300, 257, 128, 4, 3, 100, 1, 2, torch.bfloat16),  # B = 128, 44-token tail
    (2, 128, 300, 300, 64, 5, 4, 15, 1, 3, torch.bfloat16),    # the paper's G = 15
    (2, 128, 300, 1000, 64, 14, 4, 15, 1, 3, torch.bfloat16),  # G = 15, R = 67: tiled scoring
    (2, 128, 300, 100, 128, 4, 3, 40, 0, 0, torch.float32),    # fp32
    (1, 64, 64, 1, 64, 3, 2, 1, 2, 0, torch.float32),          # one query row, exact-block chunks
]


@pytest.mark.parametrize("H,d,S,Lq,B,n,K,G,E,T,dtype", SMALL)
def test_compressed_small_every_history_length(dev, H, d, S, Lq, B, n, K, G, E, T, dtype):
    say(f"compressed small H={H} d={d} S={S} Lq={Lq} B={B} n={n} K={K} G={G} {dtype}")
    w = synth.Workload("small", H, d, S, Lq, B, n, n, K, G, E, T, dtype, dtype == torch.bfloat16, 1, 7)
    x = synth.make_layer(w, 0, device=dev)
    Bpc = w.blocks_per_chunk
    nonres = [1, n * Bpc - 2] if n * Bpc > 4 else []
    cache = synth.page_layer(x.k, x.v, B, seed=3, pad_value=NAN, nonresident=nonres, extra_pages=5)
    resident = synth.resident_mask(cache).numpy()
    cc = CompressedCache.allocate(cache, n + 1)
    for c in range(n + 1):
        if c > 0:
            omnimem_compress_chunk(cache, c - 1, cc, num_chunks=c)   # append chunk c-1
            torch.cuda.synchronize()
            kc, vc = check_pooled(cc, x, w, c, resident)
        sel = omnimem_select_compressed(cache, cc, x.q, K, G, E, T, w.scale, num_chunks=c)
        torch.cuda.synchronize()
        ref = oracle_select(x, w, c, resident=resident[: c * Bpc])
        assert sel.awe_active == int(ref["awe"])
        check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
        if c > 0:
            assert not np.isin(host(sel.idx).numpy(), nonres).any()
            out, lse = omnimem_cmp_attn(cc, c, x.q, w.scale)
            o_ref, l_ref, hs, qs = oracle.cmp_attn(host(x.q), kc, vc, w.scale)
            attn_check(out, lse, o_ref, l_ref, hs, qs, dtype, f"cmp n={c}")
    # pooling a chunk again writes the same bytes
    before = (cc.k_mean.clone(), cc.k_pages.clone(), cc.v_pages.clone())
    omnimem_compress_chunk(cache, n - 1, cc)
    torch.cuda.synchronize()
    assert all(torch.equal(a, b) for a, b in zip(before, (cc.k_mean, cc.k_pages, cc.v_pages)))


def test_compressed_edge_cases(dev):
    w = synth.Workload("edge", 2, 128, 200, 150, 64, 4, 4, 5, 50, 1, 1, torch.bfloat16, False, 1, 8)
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, 64, seed=1, pad_value=NAN)
    cc = CompressedCache.allocate(cache, 4)
    say("compressed edge: empty history")
    out, lse = omnimem_cmp_attn(cc, 0, x.q, w.scale)
    sel = omnimem_select_compressed(cache, cc, x.q, 5, 50, 1, 1, w.scale, num_chunks=0)
    torch.cuda.synchronize()
    assert (host(out).float() == 0).all() and torch.isneginf(host(lse)).all()
    assert (host(sel.cnt) == 0).all() and (host(sel.idx) == -1).all()
    say("compressed edge: a chunk beyond the history or the capacity is refused")
    with pytest.raises(Exception):
        omnimem_compress_chunk(cache, 4, cc)
    small = CompressedCache.allocate(cache, 2)
    with pytest.raises(Exception):
        omnimem_select_compressed(cache, small, x.q, 5, 50, 1, 1, w.scale)
    say("compressed edge: K covering the history selects every block, as the full path does")
    for c in range(4):
        omnimem_compress_chunk(cache, c, cc)
    a = omnimem_select_compressed(cache, cc, x.q, 100, 50, 1, 1, w.scale)
    b = omnimem_select(cache, x.q, 100, 50, 1, 1, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(a.idx, b.idx) and torch.equal(a.cnt, b.cnt) and (host(a.cnt) == 16).all()


def test_compressed_wan13b_n20(dev):
    w = synth.WORKLOADS["wan1.3b_n20"]
    n = w.history_chunks
    say("compressed wan1.3b_n20: generate, append 20 chunks")
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=12, pad_value=NAN)
    cc = CompressedCache.allocate(cache, n)
    for c in range(n):
        omnimem_compress_chunk(cache, c, cc, num_chunks=c + 1)
    torch.cuda.synchronize()
    kc, vc = check_pooled(cc, x, w, n)
    say("  select from the pooled keys")
    sel = omnimem_select_compressed(cache, cc, x.q, w.top_k, w.group_size, w.window_chunks,
                                    w.awe_min_outside_chunks, w.scale)
    full = omnimem_select(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    torch.cuda.synchronize()
    ref = oracle_select(x, w, n)
    assert sel.awe_active == 1
    check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
    check_selection(host(full.idx).numpy(), host(full.cnt).numpy(), ref)
    say("  compression attention, sampled rows")
    out, lse = omnimem_cmp_attn(cc, n, x.q, w.scale)
    hs, qs = sample_rows(w.heads, w.query_tokens, 96, 5)
    o_ref, l_ref, _, _ = oracle.cmp_attn(host(x.q), kc, vc, w.scale, hs=hs, qs=qs)
    attn_check(out, lse, o_ref, l_ref, hs, qs, w.dtype, "cmp wan1.3b_n20")


# ------------------------------------------------ Eq. 1: the three branches fused

@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_gated_combine_kernel(dev, dtype):
    """The fusion kernel alone, on seeded branch outputs and gate logits (saturated,
    zero and random), against the oracle's fusion of the same values."""
    say(f"gated combine kernel {dtype}")
    lq, H, d = 301, 3, 128
    g = torch.Generator(device=dev).manual_seed(81)
    outs = [torch.randn((lq, H, d), generator=g, device=dev).to(dtype) for _ in range(3)]
    logits = 4 * torch.randn((lq, H, 3), generator=g, device=dev)
    logits[:50] = 0.0
    logits[50:60, :, 0] = 1e4
    logits[60:70, :, 1] = -1e4
    host_outs = [host(o).float().numpy().astype(np.float64) for o in outs]
    for drop in (None, 0, 2):
        args = [None if c == drop else outs[c] for c in range(3)]
        got = omnimem_gated_combine(*args, logits)
        torch.cuda.synchronize()
        want = oracle.gated_combine(*[None if c == drop else host_outs[c] for c in range(3)], host(logits).numpy())
        gotf = host(got).float().numpy()
        # fp32 evaluation: a few fp32 ulps of the sum of |terms| (cancellation can
        # leave a tiny sum of O(1) terms), then one rounding to the output dtype
        absum = oracle.gated_combine(*[None if c == drop else np.abs(host_outs[c]) for c in range(3)],
                                     host(logits).numpy())
        fp32_err = 8 * 2.0 ** -24 * absum
        if dtype == torch.float32:
            assert (np.abs(gotf - want) <= fp32_err + 2.0 ** -24 * np.abs(want)).all(), np.abs(gotf - want).max()
        else:  # within one bf16 step of the fp64 value, plus the fp32 evaluation error
            step = np.ldexp(1.0, np.frexp(np.maximum(np.abs(want), 1e-30))[1] - 8)
            assert (np.abs(gotf - want) <= step + fp32_err).all(), np.abs(gotf - want).max()
    # in place: out is one of the branches
    b = outs[1].clone()
    omnimem_gated_combine(outs[0], b, outs[2], logits, out=b)
    ref = omnimem_gated_combine(outs[0], outs[1], outs[2], logits)
    torch.cuda.synchronize()
    assert torch.equal(b, ref)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_three_branch_forward(dev, dtype):
    """Eq. 1 end to end: CMP over the compressed history, SLC over the selected
    blocks, SWA over the window chunks, fused with sigmoid gates; against the oracle's
    three branches and fusion computed from the same inputs."""
    H, d, S, Lq, B, n, K, G, E, T = 2, 128, 300, 257, 64, 6, 5, 100, 1, 2
    say(f"three-branch forward {dtype}")
    w = synth.Workload("three", H, d, S, Lq, B, n, n, K, G, E, T, dtype, dtype == torch.bfloat16, 1, 9)
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, B, seed=4, pad_value=NAN)
    cc = CompressedCache.allocate(cache, n)
    for c in range(n):
        omnimem_compress_chunk(cache, c, cc)
    sel = omnimem_select_compressed(cache, cc, x.q, K, G, E, T, w.scale)
    o_cmp, _ = omnimem_cmp_attn(cc, n, x.q, w.scale)
    o_slc, _ = omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, G, w.scale)
    o_swa, _ = omnimem_dense_attn(cache, x.q, n - E, n, w.scale)
    logits = torch.randn((Lq, H, 3), generator=torch.Generator(device=dev).manual_seed(82), device=dev)
    out = omnimem_gated_combine(o_cmp, o_slc, o_swa, logits)
    torch.cuda.synchronize()
    ref = oracle_select(x, w, n)
    check_selection(host(sel.idx).numpy(), host(sel.cnt).numpy(), ref)
    kbar, kc, vc = oracle_pooled(x, w, n)
    r_cmp, _, hs, qs = oracle.cmp_attn(host(x.q), kc, vc, w.scale)
    r_slc, _, _, _ = oracle.sparse_attn(host(x.q), host(x.k), host(x.v), B, ref["idx"], ref["cnt"], G, w.scale)
    r_swa, _, _, _ = oracle.dense_attn(host(x.q), host(x.k), host(x.v), B, n - E, n, w.scale)
    shape = (H, Lq, d)   # oracle rows come head-major: (h, q) pairs in order
    fused = oracle.gated_combine(*(r.reshape(shape).transpose(1, 0, 2) for r in (r_cmp, r_slc, r_swa)),
                                 host(logits).numpy())
    got = host(out).float().numpy()
    if dtype == torch.float32:
        check_f32(got, fused, "three-branch fused")
    else:
        check_bf16(got, fused, "three-branch fused")
