"""The Python binding's argument checks, on the CPU.  The C ABI receives raw
pointers, so the binding is the only layer that can check tensor shapes, dtypes,
contiguity and devices; each bad argument below must be refused with a ValueError
naming it, before the library is asked to launch anything.  CPU tensors of the
right shape are refused last, for not being on the GPU."""
import pytest
import torch

from paper_2605_30519_amd import omnimem as om

H, D, B, S, N = 2, 64, 64, 100, 3          # Bpc = 2
LQ, G, K = 40, 20, 3                       # R = 2


def cache(dtype=torch.bfloat16):
    pages = torch.zeros((N * 2, H, B, D), dtype=dtype)
    table = torch.arange(N * 2, dtype=torch.int32).view(N, 2)
    return om.PagedKVCache(pages, pages.clone(), table, S)


def q(dtype=torch.bfloat16, lq=LQ, h=H, d=D):
    return torch.zeros((lq, h, d), dtype=dtype)


def lists(R=2, k=K, dtype=torch.int32):
    return torch.zeros((H, R, k), dtype=dtype), torch.zeros((H, R), dtype=dtype)


def refused(match, fn, *args, **kw):
    with pytest.raises(ValueError, match=match):
        fn(*args, **kw)


def test_query_checks():
    c = cache()
    refused(r"q must have shape \(40, 2, 64\)", om.omnimem_sparse_attn, c, q(d=32), *lists(), G)
    refused("q must have shape", om.omnimem_dense_attn, c, q(h=3), 0, N)
    refused("q must be torch.bfloat16", om.omnimem_dense_attn, c, q(torch.float32), 0, N)
    refused("q must be contiguous", om.omnimem_dense_attn, c, q().transpose(0, 1).contiguous().transpose(0, 1), 0, N)
    refused(r"q must be a \[lq, H, d\] tensor", om.omnimem_select, c, q()[0], K, G, 1, 0)
    refused("must live on a GPU", om.omnimem_dense_attn, c, q(), 0, N)


def test_selection_list_checks():
    c = cache()
    idx, cnt = lists(R=3)                              # built for another group size
    refused(r"idx must have shape \(2, 2, 3\)", om.omnimem_sparse_attn, c, q(), idx, cnt, G)
    idx, cnt = lists(dtype=torch.int64)
    refused("idx must be torch.int32", om.omnimem_sparse_attn, c, q(), idx, cnt, G)
    idx, _ = lists()
    refused(r"cnt must have shape \(2, 2\)", om.omnimem_sparse_attn, c, q(), idx, torch.zeros(2, 3, dtype=torch.int32),
            G)
    idx, cnt = lists()
    refused("idx must be contiguous", om.omnimem_sparse_attn, c, q(), idx.transpose(0, 1).contiguous()
            .transpose(0, 1), cnt, G)
    refused("group_size must be >= 1", om.omnimem_sparse_attn, c, q(), idx, cnt, 0)
    refused("idx must have shape", om.omnimem_union_gather_attn, c, q(), *lists(R=1), G)
    refused("must live on a GPU", om.omnimem_sparse_attn, c, q(), idx, cnt, G)


def test_output_checks():
    c = cache()
    idx, cnt = lists()
    refused("out must have shape", om.omnimem_sparse_attn, c, q(), idx, cnt, G, out=q(lq=LQ + 1))
    refused("out must be torch.bfloat16", om.omnimem_dense_attn, c, q(), 0, N, out=q(torch.float32))
    refused(r"lse must have shape \(2, 40\)", om.omnimem_dense_attn, c, q(), 0, N,
            lse=torch.zeros(LQ, H, dtype=torch.float32))
    refused("lse must be torch.float32", om.omnimem_sparse_attn, c, q(), idx, cnt, G,
            lse=torch.zeros(H, LQ, dtype=torch.float64))
    bad = om.Selection(torch.zeros((H, 2, K + 1), dtype=torch.int32), torch.zeros((H, 2), dtype=torch.int32), None, 0)
    refused(r"out.idx must have shape \(2, 2, 3\)", om.omnimem_select, c, q(), K, G, 1, 0, out=bad)


def test_cache_checks():
    c = cache()
    c.page_table = torch.zeros((N, 3), dtype=torch.int32)
    refused("page_table must be", om.omnimem_dense_attn, c, q(), 0, N)
    c = cache()
    c.v_pages = c.v_pages[:, :, :32].contiguous()
    refused("share one", om.omnimem_dense_attn, c, q(), 0, N)
    refused("the cache must live on a GPU", om.omnimem_select, cache(), q(), K, G, 1, 0)


def test_compressed_and_fusion_checks():
    c = cache()
    cc = om.CompressedCache(torch.zeros((H, N * 2, D)), torch.zeros((1, H, 64, D), dtype=torch.bfloat16),
                            torch.zeros((1, H, 64, D), dtype=torch.bfloat16), torch.zeros(1, dtype=torch.int32),
                            B, S, N)
    bad = om.CompressedCache(cc.k_mean[:, :1].contiguous(), cc.k_pages, cc.v_pages, cc.page_table, B, S, N)
    refused("k_mean holds fewer pooled tokens", om.omnimem_select_compressed, c, bad, q(), K, G, 1, 0)
    bad = om.CompressedCache(cc.k_mean, cc.k_pages.float(), cc.v_pages, cc.page_table, B, S, N)
    refused("cmp k_pages must be torch.bfloat16", om.omnimem_select_compressed, c, bad, q(), K, G, 1, 0)
    lo = torch.zeros((1, H, 64, D), dtype=torch.bfloat16)
    bad = om.CompressedCache(cc.k_mean, cc.k_pages, cc.v_pages, cc.page_table, B, S, N, lo.float())
    refused("cmp k_lo must be torch.bfloat16", om.omnimem_select_compressed, c, bad, q(), K, G, 1, 0)
    bad = om.CompressedCache(cc.k_mean, cc.k_pages, cc.v_pages, cc.page_table, B, S, N, lo[:, :, :32].contiguous())
    refused("cmp k_lo must have shape", om.omnimem_compress_chunk, c, 0, bad)
    c32 = cache(torch.float32)
    bad = om.CompressedCache(cc.k_mean, cc.k_pages.float(), cc.v_pages.float(), cc.page_table, B, S, N, lo)
    refused("k_lo exists for bf16 caches only", om.omnimem_compress_chunk, c32, 0, bad)
    refused("q must be", om.omnimem_cmp_attn, cc, N, q(torch.float32))
    o = q()
    refused("gate_logits must be", om.omnimem_gated_combine, o, o, None, torch.zeros((LQ, H, 2)))
    refused("must live on a GPU", om.omnimem_gated_combine, o, o, None, torch.zeros((LQ, H, 3)))
