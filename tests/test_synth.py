"""The synthetic input generator and the paged layout (CPU)."""
import torch

from paper_2605_30519_amd import synth


def test_generation_is_seeded_and_chunkwise():
    w = synth.Workload("t", 2, 64, 100, 50, 64, 3, 5, 2, 25, 1, 1, torch.bfloat16, True, 1, 3)
    a = synth.make_layer(w, 0)
    b = synth.make_layer(w, 0)
    assert torch.equal(a.k.view(torch.int16), b.k.view(torch.int16)) and torch.equal(a.q.view(torch.int16),
                                                                                      b.q.view(torch.int16))
    # a longer history shares its first chunks with a shorter one
    c = synth.make_layer(w.with_history(5), 0)
    assert torch.equal(c.k[:3].view(torch.int16), a.k.view(torch.int16))
    d = synth.make_layer(w, 1)
    assert not torch.equal(d.k.view(torch.int16), a.k.view(torch.int16))
    # every (head, group) has exactly K planted blocks over the longest history
    assert (a.rel.relevant.sum(-1) == w.top_k).all()


def test_paged_layout_round_trip():
    w = synth.Workload("t", 3, 64, 150, 10, 64, 4, 4, 2, 10, 1, 1, torch.float32, False, 1, 4)
    x = synth.make_layer(w, 0)
    cache = synth.page_layer(x.k, x.v, 64, seed=9, pad_value=float("nan"), nonresident=[5], extra_pages=3)
    Bpc = w.blocks_per_chunk
    assert cache.page_table.shape == (4, Bpc) and cache.k_pages.shape == (4 * Bpc + 3, 3, 64, 64)
    table = cache.page_table.reshape(-1)
    assert table[5] == -1
    live = table[table >= 0]
    assert len(set(live.tolist())) == len(live)            # pages are distinct
    for b in range(4 * Bpc):
        if b == 5:
            continue
        c, o = divmod(b, Bpc)
        toks = range(o * 64, min(o * 64 + 64, 150))
        page = int(table[b])
        for h in range(3):
            got = cache.k_pages[page, h, : len(toks)]
            assert torch.equal(got, x.k[c, list(toks), h])
            assert torch.equal(cache.v_pages[page, h, : len(toks)], x.v[c, list(toks), h])
            if len(toks) < 64:
                assert torch.isnan(cache.k_pages[page, h, len(toks):]).all()
    assert synth.resident_mask(cache).tolist() == [b != 5 for b in range(4 * Bpc)]
