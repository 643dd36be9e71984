"""omnimem_select_noalloc, the allocation-free variant of omnimem_select for callers
that cannot allocate device memory, through the C ABI: its scratch is the
library's static per-GPU array instead of a caller workspace.  Its outputs must
equal omnimem_select's bit for bit on the same inputs, call after call, including
a call on a smaller input right after a larger one (the array then still holds the
larger call's data) and a call that needs nearly the whole array."""
import pytest
import torch

from paper_2605_30519_amd import (OmniMemError, Selection, omnimem_select, omnimem_select_noalloc,
                                  omnimem_select_workspace_bytes, select_params, synth)
from paper_2605_30519_amd.omnimem import NOALLOC_SCRATCH_BYTES
from parity import say

pytestmark = pytest.mark.gpu
NAN = float("nan")


@pytest.fixture(scope="module")
def dev():
    d = torch.device("cuda:0")
    torch.cuda.set_device(d)
    return d


def poisoned_outputs(w, dev):
    H, R, K = w.heads, w.groups, w.top_k
    return Selection(torch.full((H, R, K), 12345, dtype=torch.int32, device=dev),
                     torch.full((H, R), -7, dtype=torch.int32, device=dev),
                     torch.full((H, R, K), NAN, dtype=torch.float32, device=dev), -1)


def compare(w, dev, seed):
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=seed, pad_value=NAN)
    need = omnimem_select_workspace_bytes(cache, w.query_tokens, select_params(
        w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale))
    say(f"noalloc {w.name}: H={w.heads} d={w.head_dim} Lq={w.query_tokens} n={w.history_chunks} G={w.group_size} "
        f"needs {need} bytes of {NOALLOC_SCRATCH_BYTES}")
    ref = omnimem_select(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    got = omnimem_select_noalloc(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks,
                                 w.scale, out=poisoned_outputs(w, dev))
    torch.cuda.synchronize()
    assert got.awe_active == ref.awe_active
    assert torch.equal(got.idx, ref.idx) and torch.equal(got.cnt, ref.cnt)
    assert torch.equal(got.score.view(torch.int32), ref.score.view(torch.int32))
    return need


def test_noalloc_matches_select(dev):
    bf16 = torch.bfloat16
    # the 1.3B layer at 20 chunks, then a smaller input, then the paper's small groups
    # on a short history (close to the whole array), then a small one again
    sizes = [
        compare(synth.WORKLOADS["wan1.3b_n20"], dev, 21),
        compare(synth.Workload("small", 3, 64, 300, 300, 64, 6, 6, 7, 130, 1, 2, bf16, True, 1, 7), dev, 3),
        compare(synth.Workload("g15", 12, 128, 4680, 4680, 64, 4, 4, 4, 15, 1, 3, bf16, True, 1, 12), dev, 4),
        compare(synth.Workload("tiny", 2, 64, 256, 256, 64, 8, 8, 4, 256, 1, 3, torch.float32, False, 1, 1), dev, 11),
    ]
    assert sizes[1] < sizes[0] and sizes[3] < sizes[2] <= NOALLOC_SCRATCH_BYTES
    assert sizes[2] > NOALLOC_SCRATCH_BYTES // 2


def test_noalloc_refuses_oversized(dev):
    w = synth.Workload("g15big", 12, 128, 4680, 4680, 64, 20, 20, 4, 15, 1, 3, torch.bfloat16, True, 1, 12)
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=5)
    out = poisoned_outputs(w, dev)
    with pytest.raises(OmniMemError) as e:
        omnimem_select_noalloc(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks,
                               w.scale, out=out)
    assert e.value.status == -5
    torch.cuda.synchronize()
    assert (out.idx == 12345).all() and (out.cnt == -7).all()   # nothing was launched
