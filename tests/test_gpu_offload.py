"""The LRU hot cache of full-resolution chunks (App. B "Inference and Offloading",
App. F, Alg. 1's WaitUntilReload) through the C ABI: selection from the compressed
history with every block a candidate, the selected chunks made resident by
omnimem_lru_require (reloaded from pinned host pools into a pool of a few GPU
slots), then selection attention over the hot cache.  The attention output must
equal, bit for bit, the same kernel over the fully resident cache: only the
physical pages differ.  The bookkeeping (hits, misses, evictions, page-table rows)
is checked against an LRU simulated on the host.
"""
import numpy as np
import pytest
import torch

from paper_2605_30519_amd import (CompressedCache, LruOffload, PagedKVCache, omnimem_compress_chunk,
                                  omnimem_select_compressed, omnimem_sparse_attn, selected_chunks, synth)
from parity import say

pytestmark = pytest.mark.gpu
NAN = float("nan")


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def host_pools(x, B, pad_value=NAN):
    """Pinned host pools [n*Bpc, H, B, d]: chunk c's block o in page c*Bpc + o."""
    n, S, H, d = (int(s) for s in x.k.shape)
    Bpc = -(-S // B)
    pools = []
    for t in (x.k, x.v):
        pad = Bpc * B - S
        y = t.cpu()
        if pad:
            y = torch.cat([y, torch.full((n, pad, H, d), pad_value, dtype=y.dtype)], dim=1)
        pinned = torch.empty((n * Bpc, H, B, d), dtype=y.dtype, pin_memory=True)
        pinned.copy_(y.reshape(n * Bpc, B, H, d).permute(0, 2, 1, 3))
        pools.append(pinned)
    return pools


def simulate_lru(requests, slots):
    """Host model of the policy: per request, hits refresh recency; misses fill a free
    slot or evict the least recently used chunk not in the request."""
    resident, clock, hits, misses, evictions = {}, 0, 0, 0, 0
    for req in requests:
        want = list(dict.fromkeys(req))
        for c in want:
            if c in resident:
                clock += 1
                resident[c] = clock
                hits += 1
        for c in want:
            if c in resident:
                continue
            if len(resident) >= slots:
                victim = min((k for k in resident if k not in want), key=lambda k: resident[k])
                del resident[victim]
                evictions += 1
            clock += 1
            resident[c] = clock
            misses += 1
    return set(resident), hits, misses, evictions


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_lru_hot_cache_matches_resident(dev, dtype):
    H, d, S, Lq, B, n, K, G, E, T = 2, 128, 300, 257, 64, 8, 3, 100, 1, 2
    say(f"lru hot cache {dtype}")
    w = synth.Workload("lru", H, d, S, Lq, B, n, n, K, G, E, T, dtype, dtype == torch.bfloat16, 1, 10)
    x = synth.make_layer(w, 0, device=dev)
    full = synth.page_layer(x.k, x.v, B, seed=5, pad_value=NAN)
    Bpc = w.blocks_per_chunk
    cc = CompressedCache.allocate(full, n)
    for c in range(n):
        omnimem_compress_chunk(full, c, cc)
    k_host, v_host = host_pools(x, B)
    slots = 7
    pool = PagedKVCache(torch.zeros((slots * Bpc, H, B, d), dtype=dtype, device=dev),
                        torch.zeros((slots * Bpc, H, B, d), dtype=dtype, device=dev),
                        torch.zeros((n, Bpc), dtype=torch.int32, device=dev), S)
    lru = LruOffload(pool, slots, k_host, v_host)
    torch.cuda.synchronize()
    assert (pool.page_table == -1).all()
    with pytest.raises(Exception):   # more distinct chunks than slots
        lru.require(list(range(n)))
    requests, last = [], []
    for step in range(6):
        if step:
            # other work between steps touches chunks outside the last selection, so that
            # some of the next selection's chunks have been evicted and must be reloaded
            other = [c for c in range(n) if c not in last][: 2 + step % 2]
            requests.append(other)
            lru.require(other)
        # queries of several AR steps: different selections over the same history
        q = synth.queries(w, 0, n + step, x.rel, dev) if step else x.q
        sel = omnimem_select_compressed(pool, cc, q, K, G, E, T, w.scale, all_candidates=True)
        chunks = selected_chunks(sel, Bpc)
        assert len(chunks) <= slots, chunks
        requests.append(chunks)
        got = lru.require(chunks)
        say(f"  step {step}: chunks {chunks}, reloaded {got}")
        out, lse = omnimem_sparse_attn(pool, q, sel.idx, sel.cnt, G, w.scale)
        ref, ref_lse = omnimem_sparse_attn(full, q, sel.idx, sel.cnt, G, w.scale)
        torch.cuda.synchronize()
        view = torch.int16 if dtype == torch.bfloat16 else torch.int32
        assert torch.equal(out.view(view), ref.view(view)) and torch.equal(lse, ref_lse)
        table = pool.page_table.cpu().numpy()
        for c in range(n):
            slot = lru.slot_of(c)
            want_row = np.arange(slot * Bpc, slot * Bpc + Bpc) if slot >= 0 else np.full(Bpc, -1)
            assert np.array_equal(table[c], want_row), (c, table[c], slot)
        last = chunks
    resident, hits, misses, evictions = simulate_lru(requests, slots)
    st = lru.stats()
    assert (st["hits"], st["misses"], st["evictions"]) == (hits, misses, evictions), (st, hits, misses, evictions)
    assert {c for c in range(n) if lru.slot_of(c) >= 0} == resident
    page_bytes = H * B * d * (2 if dtype == torch.bfloat16 else 4)
    assert st["bytes_reloaded"] == 2 * misses * Bpc * page_bytes
    lru.close()


def test_lru_policy_and_errors(dev):
    """Thrash and reuse patterns against the host model; oversized requests and bad
    chunk ids are refused without changing anything."""
    H, d, S, B, n = 1, 64, 64, 64, 6
    w = synth.Workload("lru2", H, d, S, 8, B, n, n, 2, 8, 0, 0, torch.bfloat16, False, 1, 11)
    x = synth.make_layer(w, 0, device=dev)
    k_host, v_host = host_pools(x, B)
    slots = 3
    pool = PagedKVCache(torch.zeros((slots, H, B, d), dtype=torch.bfloat16, device=dev),
                        torch.zeros((slots, H, B, d), dtype=torch.bfloat16, device=dev),
                        torch.zeros((n, 1), dtype=torch.int32, device=dev), S)
    lru = LruOffload(pool, slots, k_host, v_host)
    reqs = [[0, 1], [2], [0, 3], [4, 5], [1, 1, 1], [5, 4], [2, 3, 0]]
    for r in reqs:
        lru.require(r)
    resident, hits, misses, evictions = simulate_lru(reqs, slots)
    st = lru.stats()
    assert (st["hits"], st["misses"], st["evictions"]) == (hits, misses, evictions)
    assert {c for c in range(n) if lru.slot_of(c) >= 0} == resident
    # the reloaded pages hold the host pages
    torch.cuda.synchronize()
    for c in resident:
        s = lru.slot_of(c)
        assert torch.equal(pool.k_pages[s].cpu().view(torch.int16), k_host[c].view(torch.int16))
        assert torch.equal(pool.v_pages[s].cpu().view(torch.int16), v_host[c].view(torch.int16))
    before = lru.stats()
    for bad in ([0, 1, 2, 3], [6], [-1]):
        with pytest.raises(Exception):
            lru.require(bad)
    assert lru.stats() == before
    lru.close()
