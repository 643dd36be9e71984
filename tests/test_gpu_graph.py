"""The chunk step under HIP graph capture: the library allocates nothing and issues
no memset or copy inside select, sparse attention or the probability-score
selection (all scratch is the caller's workspace), so one captured step replays
as is.  Each replay is checked bit for bit against the eager step, with the
program's own eager work and synchronisations between replays, and the outputs
overwritten before each replay so that a stale result cannot pass."""
import numpy as np
import pytest
import torch

from paper_2605_30519_amd import (SCORE_PROB, CompressedCache, omnimem_compress_chunk, omnimem_select,
                                  omnimem_select_compressed, omnimem_select_workspace_bytes, omnimem_sparse_attn,
                                  select_params, synth)
from paper_2605_30519_amd.omnimem import Selection, workspace_tensor
from parity import say

pytestmark = pytest.mark.gpu
NAN = float("nan")


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def test_graph_replay_matches_eager(dev):
    w = synth.Workload("graph", 3, 128, 600, 600, 64, 8, 8, 7, 130, 1, 2, torch.bfloat16, True, 1, 41)
    n, K, G, E, T = w.history_chunks, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=2, pad_value=NAN, nonresident=[3], extra_pages=4)
    cc = CompressedCache.allocate(cache, n)
    for c in range(n):
        omnimem_compress_chunk(cache, c, cc)
    H, R, lq = w.heads, -(-w.query_tokens // G), w.query_tokens
    ws = workspace_tensor(omnimem_select_workspace_bytes(cache, lq, select_params(K, G, E, T, w.scale)), dev)
    ws_p = workspace_tensor(omnimem_select_workspace_bytes(cache, lq, select_params(4, 15, E, T, w.scale, SCORE_PROB)),
                            dev)
    Rp = -(-lq // 15)

    def selection(r, k):
        return Selection(torch.empty((H, r, k), dtype=torch.int32, device=dev),
                         torch.empty((H, r), dtype=torch.int32, device=dev),
                         torch.empty((H, r, k), dtype=torch.float32, device=dev), 0)

    sel, sel_p = selection(R, K), selection(Rp, 4)
    out = torch.empty_like(x.q)
    lse = torch.empty((H, lq), dtype=torch.float32, device=dev)
    outputs = (sel.idx, sel.cnt, sel.score, out, lse, sel_p.idx, sel_p.cnt, sel_p.score)

    def step():
        omnimem_select(cache, x.q, K, G, E, T, w.scale, workspace=ws, out=sel)
        omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, G, w.scale, out=out, lse=lse)
        omnimem_select_compressed(cache, cc, x.q, 4, 15, E, T, w.scale, workspace=ws_p, out=sel_p,
                                  score_mode=SCORE_PROB)

    say("graph: eager step")
    step()
    torch.cuda.synchronize()
    eager = [t.clone() for t in outputs]
    assert int(sel.cnt.min()) > 0 and int(sel_p.cnt.min()) > 0

    say("graph: capture")
    side = torch.cuda.Stream(device=dev)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    for rep in range(4):
        say(f"graph: replay {rep}")
        for t in outputs:
            t.fill_(-7)
        junk = torch.randn(1 << 20, device=dev).sum()   # the program's own eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for got, want in zip(outputs, eager):
            assert torch.equal(got, want), f"replay {rep} differs from the eager step"
        assert torch.isfinite(junk)

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(20):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    say(f"graph: {e0.elapsed_time(e1) / 20:.4f} ms per replayed step")
    assert np.isfinite(e0.elapsed_time(e1))
