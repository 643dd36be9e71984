"""Benchmark of OmniMem's memory-retrieval attention step on one MI355X.

A step = one chunk-layer: omnimem_select (query-shared top-K with Adaptive
Window Exclusion over the whole history) followed by omnimem_sparse_attn (per-head
scattered block-sparse attention), on the Wan2.1-1.3B-shaped layer: 12 heads x
128, a 4680-token chunk, 20 chunks of history (93,600 cached keys), 64-token
blocks, K = 64, one query group, 1-chunk window.  Four independent layer caches
(2.3 GB of K+V) are used in rotation, so no step finds its cache in the 256 MB
Infinity Cache.  Inputs are resident in HBM before the timed region.

Prints ONE JSON line: value = effective TFLOP/s of select + sparse attention
(attention flops over the valid selected keys + scoring flops, per step time),
ms_per_step = ms per chunk-layer, a roofline object for the dominant kernel
(measured with HIP events on the launch stream), the CPU oracle's throughput on
a bounded sample of the same workload, per-stage times, and a sweep over history
length (10/30/60/120 chunks) with the speedup over in-build dense attention.

Further objects in the same line, each skippable by a flag: the select stage by
cache state; the compressed-history step (pooled keys, CMP attention, the gated
three-branch forward of Eq. 1, and selection by probability-averaged scores);
the paper's small-group setting (G_q = 15); the LRU hot cache; the 30-layer
history ramp; achievable-peak probes; CPU-oracle extrapolations.  --prob-only G
times only the probability-score selection (a profiling target).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms per chunk-layer + effective TFLOP/s of select+sparse-attn vs history length"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
WORKLOAD = "wan1.3b_n20"
ROTATE_LAYERS = 4


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    # The MI355X's clock ramps up over the first fraction of a second of sustained
    # load (the attention kernel runs at ~1.8-1.9 GHz for the first milliseconds and
    # at ~2.15 GHz and above after ~50 ms), so the default warm-up covers ~0.4 s of
    # steps and the timed region (~0.1 s) measures the steady state that a
    # generation loop runs in.
    p.add_argument("--steps", type=int, default=500)
    p.add_argument("--warmup", type=int, default=2000)
    p.add_argument("--no-sweep", action="store_true", help="skip the history-length sweep")
    p.add_argument("--no-cpu-baseline", action="store_true", help="skip timing the CPU oracle")
    p.add_argument("--no-stress", action="store_true", help="skip the 14B-shaped union-gather comparison")
    p.add_argument("--no-ramp", action="store_true", help="skip the 30-layer, 1 -> 60 chunk ramp")
    p.add_argument("--no-compressed", action="store_true", help="skip the compressed-history path")
    p.add_argument("--no-lru", action="store_true", help="skip the LRU hot-cache measurement")
    p.add_argument("--no-small-group", action="store_true", help="skip the paper's small-group setting")
    p.add_argument("--no-probe", action="store_true", help="skip the achievable-peak probes (copy, GEMM)")
    p.add_argument("--attn-only", type=int, default=0, metavar="N",
                   help="only run N sparse-attention calls on the bench workload's first layer (a profiling "
                        "target), print their mean time, and exit")
    p.add_argument("--select-only", type=int, default=0, metavar="N",
                   help="only run N selections over the bench workload's rotated layer caches (a profiling "
                        "target), print their median time, and exit")
    p.add_argument("--small-group-only", action="store_true",
                   help="only run the small-group setting (G_q = 15, top-4: select and sparse attention, 150 "
                        "calls each; a profiling target), print its line, and exit")
    p.add_argument("--power-clock", action="store_true",
                   help="only sample socket power and GFX clock while the attention kernel (the bench layer's "
                        "queries, then Q = 0) and the MFMA issue loop (smooth, then random operands) each run "
                        "back to back for a few seconds, print the line, and exit")
    p.add_argument("--cu-fill", action="store_true",
                   help="only time the attention kernel with 228 and with 256 workgroups of 256 query rows "
                        "(one per CU), 64 or 57-58 key tiles each, sampling socket power and GFX clock, print "
                        "the line, and exit")
    p.add_argument("--prob-only", type=int, default=0, metavar="G",
                   help="only time selection by probability-averaged scores from the pooled history, "
                        "query groups of G rows (top-64 for one group per head, else top-4), and exit")
    return p.parse_args()


def prob_only(dev, G, reps=50):
    """Selection by probability-averaged scores alone, on the bench workload's first
    layer and its pooled history: a profiling target for those kernels."""
    import torch

    from paper_2605_30519_amd import (SCORE_PROB, CompressedCache, omnimem_compress_chunk, omnimem_select_compressed,
                                      synth)
    w = synth.WORKLOADS[WORKLOAD]
    n = w.history_chunks
    K = w.top_k if G >= w.query_tokens else 4
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=1000)
    cc = CompressedCache.allocate(cache, n)
    for c in range(n):
        omnimem_compress_chunk(cache, c, cc)
    sel = None
    for _ in range(20):
        sel = omnimem_select_compressed(cache, cc, x.q, K, G, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                                        out=sel, want_score=False, score_mode=SCORE_PROB)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        omnimem_select_compressed(cache, cc, x.q, K, G, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                                  out=sel, want_score=False, score_mode=SCORE_PROB)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    logit_fl = 2.0 * w.query_tokens * n * w.blocks_per_chunk * w.head_dim * w.heads
    print(json.dumps({"prob_select": {"workload": WORKLOAD, "group_size": G, "top_k": K, "select_ms": round(ms, 4),
                                      "logit_tflops": round(logit_fl / (ms * 1e-3) / 1e12, 2)}}), flush=True)


def attn_only(dev, calls, warm=200):
    """Sparse attention alone on the bench workload's first layer, back to back: a
    profiling target for the attention kernel."""
    import torch

    from paper_2605_30519_amd import omnimem_select, omnimem_sparse_attn, synth
    w = synth.WORKLOADS[WORKLOAD]
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=1000)
    sel = omnimem_select(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    out = torch.empty_like(x.q)
    lse = torch.empty((w.heads, w.query_tokens), dtype=torch.float32, device=dev)
    for _ in range(warm):
        omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale, out=out, lse=lse)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(calls):
        omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale, out=out, lse=lse)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / calls
    # the host's time per call (binding checks, descriptor, launch), over 100 calls
    # enqueued onto an idle GPU: far fewer than the queue holds, so none waits
    t0 = time.perf_counter()
    for _ in range(100):
        omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale, out=out, lse=lse)
    host_us = (time.perf_counter() - t0) / 100 * 1e6
    torch.cuda.synchronize()
    fl = attn_flops(sel.idx, sel.cnt, w, w.history_chunks)
    print(json.dumps({"attn_only": {"workload": WORKLOAD, "calls": calls, "ms": round(ms, 4),
                                    "tflops": round(fl / (ms * 1e-3) / 1e12, 1), "flops_per_call": fl,
                                    "host_us_per_call": round(host_us, 2)}}), flush=True)


def power_clock(dev, secs=6.0):
    """Socket power and GFX clock, read through torch.cuda (the SMI library) twice
    while each load runs back to back for `secs`: the attention kernel on the bench
    workload's first layer with its queries and with Q = 0 (all scores 0, so P is
    constant and few MFMA operand bits toggle), the MFMA issue loop of the probe
    library with smooth and with random operands, and its softmax-slot loop with
    operands in registers and from LDS.  The chip holds its clock only
    while its power stays within the limit, and MFMA power grows with the operand
    bits that toggle: this is what sets the clock at which the kernels run."""
    import ctypes
    import threading

    import torch

    from paper_2605_30519_amd import _build, omnimem_select, omnimem_sparse_attn, synth
    w = synth.WORKLOADS[WORKLOAD]
    x = synth.make_layer(w, 0, device=dev)
    cache = synth.page_layer(x.k, x.v, w.block_size, seed=1000)
    sel = omnimem_select(cache, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    out = torch.empty_like(x.q)
    lse = torch.empty((w.heads, w.query_tokens), dtype=torch.float32, device=dev)
    q0 = torch.zeros_like(x.q)
    fl = attn_flops(sel.idx, sel.cnt, w, w.history_chunks)
    P = ctypes.CDLL(_build.PROBE_LIB)
    P.omnimem_probe_mfma_bf16.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_void_p]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    sink = torch.zeros(4, dtype=torch.float32, device=dev)
    iters = 100000  # 256 workgroups of 4 waves: ~6 ms per launch
    mfma_fl = 256 * 4 * iters * 4 * 32768.0

    P.omnimem_probe_softmax_slot.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                             ctypes.c_void_p]
    slot_iters = 25000  # 8 slots per round: ~4 ms per launch
    slot_fl = 256 * 4 * slot_iters * 8 * 32768.0

    def mfma(operands):
        assert P.omnimem_probe_mfma_bf16(operands, iters, 256, 1, ctypes.c_void_p(sink.data_ptr()), stream) == 0

    def slot(lds):
        assert P.omnimem_probe_softmax_slot(lds, slot_iters, 256, ctypes.c_void_p(sink.data_ptr()), stream) == 0

    loads = [("attention", lambda: omnimem_sparse_attn(cache, x.q, sel.idx, sel.cnt, w.group_size, w.scale,
                                                       out=out, lse=lse), fl, 1000),
             ("attention_q0", lambda: omnimem_sparse_attn(cache, q0, sel.idx, sel.cnt, w.group_size, w.scale,
                                                          out=out, lse=lse), fl, 1000),
             ("mfma_smooth", lambda: mfma(0), mfma_fl, 20),
             ("mfma_random", lambda: mfma(1), mfma_fl, 20),
             ("softmax_slot", lambda: slot(0), slot_fl, 20),
             ("softmax_slot_lds", lambda: slot(1), slot_fl, 20)]
    res = {"workload": WORKLOAD, "seconds_per_load": secs}
    for name, call, flops, batch in loads:
        samples = []

        def sampler():
            for delay in (0.5 * secs, 0.25 * secs):
                time.sleep(delay)
                samples.append((float(torch.cuda.power_draw(dev)), float(torch.cuda.clock_rate(dev))))

        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(batch):
            call()
        torch.cuda.synchronize()
        th = threading.Thread(target=sampler)
        calls = 0
        t_stop = time.time() + secs
        th.start()
        e0.record()
        while time.time() < t_stop:
            for _ in range(batch):
                call()
            calls += batch
            torch.cuda.synchronize()
        e1.record()
        torch.cuda.synchronize()
        th.join()
        ms = e0.elapsed_time(e1) / calls
        res[name] = {"us_per_call": round(ms * 1e3, 1), "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
                     "socket_power_w": [s[0] for s in samples], "gfx_clock_mhz": [s[1] for s in samples]}
        log(f"{name}: {res[name]}")
    print(json.dumps({"power_clock": res}), flush=True)


def cu_fill(dev, secs=3.0):
    """What a split of each (head, group)'s key list over all 256 CUs could gain.  At
    the bench shape the 64-row kernel runs 228 workgroups (12 heads x 19 tiles of 256
    rows), one per CU, each over 64 key tiles, so 28 CUs idle.  A split that balanced
    the work would give every CU 57 tiles.  The kernel is timed on synthetic layers
    of the same per-workgroup shape (seeded normal K, V and Q; one query group per
    head; 64 or 57-58 blocks of 64 tokens drawn at random from a 20-chunk history of
    4680-token chunks, full blocks only): 12 heads x 4680 rows (228 workgroups) and
    16 heads x 4096 rows (256 workgroups), each run back to back for `secs` with
    socket power and GFX clock read twice.  The 256-workgroup runs at 57 and 58
    tiles price the balanced split before any merge of its partial results."""
    import threading

    import torch

    from paper_2605_30519_amd import omnimem_sparse_attn, synth
    n, S, d, B = 20, 4680, 128, 64
    Bpc = -(-S // B)
    full = torch.tensor([c * Bpc + o for c in range(n) for o in range(Bpc - 1)], dtype=torch.int32)
    scale = 1.0 / d ** 0.5
    caches = {}
    res = {"history": f"{n} chunks of {S} tokens, blocks of {B}", "seconds_per_case": secs}
    for H, lq, K in ((12, 4680, 64), (12, 4680, 57), (16, 4096, 64), (16, 4096, 57), (16, 4096, 58)):
        g = torch.Generator(device="cpu").manual_seed(1000 * H + K)
        if H not in caches:
            k = torch.randn((n, S, H, d), generator=g).to(torch.bfloat16).to(dev)
            v = torch.randn((n, S, H, d), generator=g).to(torch.bfloat16).to(dev)
            caches[H] = synth.page_layer(k, v, B, seed=H)
            del k, v
        cache = caches[H]
        q = torch.randn((lq, H, d), generator=g).to(torch.bfloat16).to(dev)
        idx = torch.stack([torch.sort(full[torch.randperm(full.numel(), generator=g)[:K]]).values for _ in range(H)])
        idx = idx.reshape(H, 1, K).contiguous().to(dev)
        cnt = torch.full((H, 1), K, dtype=torch.int32, device=dev)
        out = torch.empty_like(q)
        lse = torch.empty((H, lq), dtype=torch.float32, device=dev)

        def call():
            omnimem_sparse_attn(cache, q, idx, cnt, lq, scale, out=out, lse=lse)
        samples = []

        def sampler():
            for delay in (0.5 * secs, 0.25 * secs):
                time.sleep(delay)
                samples.append((float(torch.cuda.power_draw(dev)), float(torch.cuda.clock_rate(dev))))
        for _ in range(500):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        th = threading.Thread(target=sampler)
        calls, t_stop = 0, time.time() + secs
        th.start()
        e0.record()
        while time.time() < t_stop:
            for _ in range(500):
                call()
            calls += 500
            torch.cuda.synchronize()
        e1.record()
        torch.cuda.synchronize()
        th.join()
        us = e0.elapsed_time(e1) / calls * 1e3
        wgs = H * -(-lq // 256)
        fl = 4.0 * d * H * lq * K * B
        name = f"h{H}_rows{lq}_top{K}"
        res[name] = {"workgroups": wgs, "tiles_per_workgroup": K, "us_per_call": round(us, 1),
                     "tflops": round(fl / (us * 1e-6) / 1e12, 1), "ns_per_workgroup_tile": round(us * 1e3 / K, 1),
                     "socket_power_w": [s[0] for s in samples], "gfx_clock_mhz": [s[1] for s in samples]}
        log(f"{name}: {res[name]}")
        del q, idx, cnt, out, lse
    base = res["h12_rows4680_top64"]["us_per_call"]
    res["balanced_split_bound_speedup"] = round(base / res["h16_rows4096_top57"]["us_per_call"], 4)
    print(json.dumps({"cu_fill": res}), flush=True)


def select_only(dev, calls, warm=100):
    """omnimem_select alone over the bench workload's rotated layer caches (so that K
    is read from HBM, as in the bench), HIP events around each call: a profiling
    target for the selection kernels."""
    import numpy as np
    import torch

    from paper_2605_30519_amd import omnimem_select, synth
    w = synth.WORKLOADS[WORKLOAD]
    layers = []
    for layer in range(ROTATE_LAYERS):
        x = synth.make_layer(w, layer, device=dev)
        layers.append((x.q, synth.page_layer(x.k, x.v, w.block_size, seed=1000 + layer)))
        del x
    sels = [omnimem_select(c, q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
            for q, c in layers]

    def call(i):
        q, c = layers[i % ROTATE_LAYERS]
        omnimem_select(c, q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                       out=sels[i % ROTATE_LAYERS], want_score=False)
    for i in range(warm):
        call(i)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(calls)]
    torch.cuda.synchronize()
    for i in range(calls):
        ev[i][0].record()
        call(i)
        ev[i][1].record()
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in ev])
    sb = select_bytes(w, w.history_chunks, sels[0].awe_active)
    print(json.dumps({"select_only": {"workload": WORKLOAD, "calls": calls, "ms": round(float(np.median(t)), 4),
                                      "gbs": round(sb / (float(np.median(t)) * 1e-3) / 1e9, 1)}}), flush=True)


def attn_flops(idx, cnt, w, n_chunks):
    """4 * d * sum over (head, query row) of the valid keys in its selected blocks."""
    import torch
    Bpc, B, S = w.blocks_per_chunk, w.block_size, w.chunk_tokens
    o = torch.remainder(idx.long(), Bpc)
    valid = torch.where(o == Bpc - 1, S - o * B, torch.full_like(o, B))
    K = idx.shape[-1]
    keep = (torch.arange(K, device=idx.device)[None, None, :] < cnt[..., None].long()) & (idx >= 0)
    keys = (valid * keep).sum(-1)                                  # [H, R]
    rows = torch.tensor([min(w.group_size, w.query_tokens - r * w.group_size) for r in range(idx.shape[1])],
                        device=idx.device)
    return float(4 * w.head_dim * (keys * rows[None, :]).sum().item())


def select_bytes(w, n_chunks, awe):
    """Algorithmic HBM bytes of select: every candidate K block once (valid tokens), plus Q."""
    eb = 2
    Bpc = w.blocks_per_chunk
    cand_chunks = n_chunks - w.window_chunks if awe else n_chunks
    return cand_chunks * w.chunk_tokens * w.heads * w.head_dim * eb + w.query_tokens * w.heads * w.head_dim * eb


def score_flops(w, n_chunks):
    return 2.0 * w.groups * n_chunks * w.blocks_per_chunk * w.heads * w.head_dim


def source_digest(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def load_traffic(kernel):
    """HBM bytes per launch from committed rocprofv3 counter runs, if the kernel
    source has not changed since they were taken; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    src = os.path.join(ROOT, "paper_2605_30519_amd", "csrc", rec.get("source", ""))
    if not os.path.exists(src) or source_digest(src) != rec.get("source_sha256"):
        return None
    return rec.get("bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2605_30519_amd import (lib, omnimem_dense_attn, omnimem_select, omnimem_select_workspace_bytes,
                                      omnimem_sparse_attn, omnimem_union_gather_attn, select_params, synth)
    from paper_2605_30519_amd.omnimem import Selection, workspace_tensor

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lib()
    if args.small_group_only:
        print(json.dumps({"small_group": small_group_measure(dev)}))
        return
    if args.power_clock:
        power_clock(dev)
        return
    if args.cu_fill:
        cu_fill(dev)
        return
    if args.prob_only:
        prob_only(dev, args.prob_only)
        return
    if args.attn_only:
        attn_only(dev, args.attn_only)
        return
    if args.select_only:
        select_only(dev, args.select_only)
        return
    w = synth.WORKLOADS[WORKLOAD]
    n = w.history_chunks
    H, R, K = w.heads, w.groups, w.top_k

    # ---------------------------------------------------------------- inputs
    log(f"generating {ROTATE_LAYERS} layer caches of {n} chunks")
    layers = []
    for layer in range(ROTATE_LAYERS):
        x = synth.make_layer(w, layer, device=dev)
        cache = synth.page_layer(x.k, x.v, w.block_size, seed=1000 + layer)
        layers.append((x.q, cache))
        if layer == 0:
            x0 = x
        else:
            del x
    params = select_params(K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    ws = workspace_tensor(omnimem_select_workspace_bytes(layers[0][1], w.query_tokens, params), dev)
    sels = [Selection(torch.empty((H, R, K), dtype=torch.int32, device=dev),
                      torch.empty((H, R), dtype=torch.int32, device=dev), None, 0) for _ in layers]
    outs = [torch.empty_like(q) for q, _ in layers]
    lses = [torch.empty((H, w.query_tokens), dtype=torch.float32, device=dev) for _ in layers]
    torch.cuda.synchronize()

    def step(i, ev=None):
        q, cache = layers[i % ROTATE_LAYERS]
        s = sels[i % ROTATE_LAYERS]
        if ev is not None:
            ev[0].record()
        omnimem_select(cache, q, K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                       workspace=ws, out=s, want_score=False)
        if ev is not None:
            ev[1].record()
        omnimem_sparse_attn(cache, q, s.idx, s.cnt, w.group_size, w.scale, out=outs[i % ROTATE_LAYERS],
                            lse=lses[i % ROTATE_LAYERS])
        if ev is not None:
            ev[2].record()

    log(f"warmup {args.warmup} steps, then {args.steps} timed steps")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    flops_per_layer = [attn_flops(s.idx, s.cnt, w, n) for s in sels]
    awe = sels[0].awe_active

    # ---------------------------------------------------------------- timed region
    # the steps alone (no event between the stages), then the same number of steps
    # again with events around each stage for the per-stage split
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for i in range(args.steps):
        step(i)
    t_end.record()
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    # the same steps replayed from HIP graphs (one per rotated layer cache)
    graphs = []
    for i in range(ROTATE_LAYERS):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(i)
        graphs.append(g)
    for i in range(2 * ROTATE_LAYERS):
        graphs[i % ROTATE_LAYERS].replay()
    torch.cuda.synchronize()
    t_start.record()
    for i in range(args.steps):
        graphs[i % ROTATE_LAYERS].replay()
    t_end.record()
    torch.cuda.synchronize()
    graph_ms_per_step = t_start.elapsed_time(t_end) / args.steps
    del graphs
    sel_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    att_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    flops_steps = np.array([flops_per_layer[i % ROTATE_LAYERS] for i in range(args.steps)])
    sflops = score_flops(w, n)
    eff_tflops = float((flops_steps.sum() + sflops * args.steps) / (total_ms * 1e-3) / 1e12)

    attn_tflops = float(flops_steps.mean() / (att_ms.mean() * 1e-3) / 1e12)
    sbytes = select_bytes(w, n, awe)
    sel_gbs = float(sbytes / (sel_ms.mean() * 1e-3) / 1e9)
    attn_roof = {"kernel": "k_attn_bf16_r64", "bound": "mfma", "achieved": round(attn_tflops, 2),
                 "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                 "traffic": load_traffic("k_attn_bf16_r64"),
                 "per_launch": {"flops": flops_steps.mean(), "avg_ms": round(float(att_ms.mean()), 4)}}
    sel_roof = {"kernel": "select (k_qmean_partial+k_pool_score+k_topk)", "bound": "hbm",
                "achieved": round(sel_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(sel_gbs / PEAK_HBM_GBS, 4), "traffic": load_traffic("k_pool_score"),
                "per_launch": {"bytes": sbytes, "avg_ms": round(float(sel_ms.mean()), 4)}}
    dominant = attn_roof if att_ms.mean() >= sel_ms.mean() else sel_roof

    result = {
        "metric": METRIC,
        "value": round(eff_tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "Wan2.1-1.3B-shaped attention layer: 12 heads x 128, 4680-token chunk, "
                               "20-chunk history (93,600 keys) in 64-token blocks, top-64 per head, one query "
                               "group, 1-chunk excluded window",
                   "history_chunks": n, "heads": H, "head_dim": w.head_dim, "query_tokens": w.query_tokens,
                   "block_size": w.block_size, "top_k": K, "group_size": w.group_size,
                   "rotated_layer_caches": ROTATE_LAYERS},
        "roofline": dominant,
        "stages": {"select_ms": round(float(np.median(sel_ms)), 4),
                   "sparse_attn_ms": round(float(np.median(att_ms)), 4),
                   "select_ms_p10_p90": [round(float(np.percentile(sel_ms, 10)), 4),
                                         round(float(np.percentile(sel_ms, 90)), 4)],
                   "sparse_attn_ms_p10_p90": [round(float(np.percentile(att_ms, 10)), 4),
                                              round(float(np.percentile(att_ms, 90)), 4)],
                   "select_roofline": sel_roof, "attention_roofline": attn_roof, "awe_active": awe,
                   "graph_replay": {"ms_per_step": round(graph_ms_per_step, 4),
                                    "effective_tflops": round(float((flops_steps.mean() + sflops) /
                                                                    (graph_ms_per_step * 1e-3) / 1e12), 2)}},
    }

    # ---------------------------------------------------------------- select, cache state
    # the select stage with the 256 MB Infinity Cache (MALL) flushed before each call
    # by a 1 GiB write, and warm (the same layer back to back)
    result["stages"]["select_cache_state"] = select_cache_state(layers, sels, ws, w, sbytes)

    # ---------------------------------------------------------------- compressed history
    if not args.no_compressed:
        log("compressed-history path (pool the newest chunk + select from pooled keys + sparse attention)")
        result["compressed"] = compressed_measure(dev, layers, sels, outs, lses, w, args)

    # ---------------------------------------------------------------- small query groups
    if not args.no_small_group:
        log("small query groups (G_q = 15, top-4 per group, 3-chunk window)")
        result["small_group"] = small_group_measure(dev)

    # ---------------------------------------------------------------- LRU hot cache
    if not args.no_lru:
        log("LRU hot cache: reload bandwidth and LRU size vs a drifting working set")
        result["lru"] = lru_measure(dev, x0, w)

    # ---------------------------------------------------------------- sweep
    if not args.no_sweep:
        wl = synth.WORKLOADS["wan1.3b_long"]
        log("history sweep 10/30/60/120 chunks (generating 120 chunks)")
        del layers, sels, outs, lses
        torch.cuda.empty_cache()
        xl = synth.make_layer(wl, 0, device=dev)
        cl = synth.page_layer(xl.k, xl.v, wl.block_size, seed=77)
        del xl.k, xl.v
        wsl = workspace_tensor(omnimem_select_workspace_bytes(cl, wl.query_tokens, params), dev)
        sweep = []
        ccl = None
        if not args.no_compressed:
            from paper_2605_30519_amd import (CompressedCache, omnimem_cmp_attn, omnimem_compress_chunk,
                                              omnimem_select_compressed)
            ccl = CompressedCache.allocate(cl, 120)
            for c in range(120):
                omnimem_compress_chunk(cl, c, ccl)
        for hn in (10, 30, 60, 120):
            q = synth.queries(wl, 0, hn, xl.rel, dev)
            s = Selection(torch.empty((H, R, K), dtype=torch.int32, device=dev),
                          torch.empty((H, R), dtype=torch.int32, device=dev), None, 0)
            out = torch.empty_like(q)
            ls = torch.empty((H, wl.query_tokens), dtype=torch.float32, device=dev)
            reps = 5
            e = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps + 1)]
            for r in range(reps + 1):
                e[r][0].record()
                omnimem_select(cl, q, K, wl.group_size, wl.window_chunks, wl.awe_min_outside_chunks, wl.scale,
                               num_chunks=hn, workspace=wsl, out=s, want_score=False)
                e[r][1].record()
                omnimem_sparse_attn(cl, q, s.idx, s.cnt, wl.group_size, wl.scale, num_chunks=hn, out=out, lse=ls)
                e[r][2].record()
                omnimem_dense_attn(cl, q, 0, hn, wl.scale, num_chunks=hn, out=out, lse=ls)
                e[r][3].record()
            torch.cuda.synchronize()
            ts = np.median([e[r][0].elapsed_time(e[r][1]) for r in range(1, reps + 1)])
            ta = np.median([e[r][1].elapsed_time(e[r][2]) for r in range(1, reps + 1)])
            td = np.median([e[r][2].elapsed_time(e[r][3]) for r in range(1, reps + 1)])
            fl = attn_flops(s.idx, s.cnt, wl, hn)
            dense_fl = 4.0 * wl.head_dim * wl.heads * wl.query_tokens * hn * wl.chunk_tokens
            sweep.append({"history_chunks": hn, "cached_keys": hn * wl.chunk_tokens,
                          "select_ms": round(float(ts), 4), "sparse_attn_ms": round(float(ta), 4),
                          "ms_per_chunk_layer": round(float(ts + ta), 4),
                          "effective_tflops": round((fl + score_flops(wl, hn)) / ((ts + ta) * 1e-3) / 1e12, 2),
                          "select_gbs": round(select_bytes(wl, hn, s.awe_active) / (ts * 1e-3) / 1e9, 1),
                          "sparse_attn_tflops": round(fl / (ta * 1e-3) / 1e12, 2),
                          "dense_ms": round(float(td), 4),
                          "dense_tflops": round(dense_fl / (td * 1e-3) / 1e12, 2),
                          "speedup_vs_dense": round(float(td / (ts + ta)), 2)})
            if ccl is not None:
                e = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps + 1)]
                for r in range(reps + 1):
                    e[r][0].record()
                    omnimem_select_compressed(cl, ccl, q, K, wl.group_size, wl.window_chunks,
                                              wl.awe_min_outside_chunks, wl.scale, num_chunks=hn, workspace=wsl,
                                              out=s, want_score=False)
                    e[r][1].record()
                    omnimem_cmp_attn(ccl, hn, q, wl.scale, out=out, lse=ls)
                    e[r][2].record()
                torch.cuda.synchronize()
                tsc = np.median([e[r][0].elapsed_time(e[r][1]) for r in range(1, reps + 1)])
                tcm = np.median([e[r][1].elapsed_time(e[r][2]) for r in range(1, reps + 1)])
                cmp_fl = 4.0 * wl.head_dim * wl.heads * wl.query_tokens * hn * wl.blocks_per_chunk
                sweep[-1].update({"select_compressed_ms": round(float(tsc), 4),
                                  "cmp_attn_ms": round(float(tcm), 4),
                                  "cmp_attn_tflops": round(cmp_fl / (tcm * 1e-3) / 1e12, 2)})
        result["sweep"] = sweep
        del cl

    # ---------------------------------------------------------------- 30-layer ramp
    if not args.no_ramp:
        log("30-layer ramp, history 1 -> 60 chunks (generating 30 x 60 chunks)")
        if "layers" in locals():
            del layers, sels, outs, lses
        torch.cuda.empty_cache()
        result["ramp"] = ramp_measure(dev)

    # ---------------------------------------------------------------- achievable peaks
    if not args.no_probe:
        log("achievable-peak probes: HBM copy, bf16 GEMM")
        result["achievable"] = probe_peaks(dev, result)

    # ---------------------------------------------------------------- 14B comparator
    if not args.no_stress:
        log("14B-shaped union-gather comparison")
        result["stress"] = stress_comparison(dev)

    # ---------------------------------------------------------------- CPU oracle
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(x0, w, flops_per_layer[0] + sflops)
        log("oracle on subsamples of the 120-chunk dense attention and the 30-layer ramp (extrapolated)")
        del x0
        torch.cuda.empty_cache()
        result["cpu_baseline"]["extrapolated"] = oracle_extrapolations(dev)

    print(json.dumps(result), flush=True)


def compressed_measure(dev, layers, sels, outs, lses, w, args):
    """The chunk step with App. C's compressed history: each step pools only the
    newest chunk into the layer's compressed cache, selects from the pooled keys and
    runs the same sparse attention.  Same rotated layer caches and steps as the main
    measurement; the pooled history of the older chunks was built beforehand, as it
    is when each chunk is appended."""
    import numpy as np
    import torch

    from paper_2605_30519_amd import (CompressedCache, omnimem_cmp_attn, omnimem_compress_chunk, omnimem_dense_attn,
                                      omnimem_gated_combine, omnimem_select_compressed,
                                      omnimem_select_workspace_bytes, omnimem_sparse_attn, select_params)
    from paper_2605_30519_amd.omnimem import workspace_tensor
    n, K = w.history_chunks, w.top_k
    ccs = [CompressedCache.allocate(cache, n) for _, cache in layers]
    for (q, cache), cc in zip(layers, ccs):
        for c in range(n):
            omnimem_compress_chunk(cache, c, cc)
    params = select_params(K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    ws = workspace_tensor(omnimem_select_workspace_bytes(layers[0][1], w.query_tokens, params), dev)

    def step(i, ev=None):
        q, cache = layers[i % len(layers)]
        cc, s = ccs[i % len(layers)], sels[i % len(layers)]
        if ev is not None:
            ev[0].record()
        omnimem_compress_chunk(cache, n - 1, cc)
        if ev is not None:
            ev[1].record()
        omnimem_select_compressed(cache, cc, q, K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                                  workspace=ws, out=s, want_score=False)
        if ev is not None:
            ev[2].record()
        omnimem_sparse_attn(cache, q, s.idx, s.cnt, w.group_size, w.scale, out=outs[i % len(layers)],
                            lse=lses[i % len(layers)])
        if ev is not None:
            ev[3].record()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    flops = [attn_flops(s.idx, s.cnt, w, n) + score_flops(w, n) for s in sels]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(args.steps):
        step(i)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    med = lambda a, b: float(np.median([e[a].elapsed_time(e[b]) for e in evs]))
    # compression attention over the same pooled history (Eq. 1's CMP branch)
    q0, _ = layers[0]
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(5):
        omnimem_cmp_attn(ccs[0], n, q0, w.scale, out=outs[0], lse=lses[0])
    e[0].record()
    for _ in range(20):
        omnimem_cmp_attn(ccs[0], n, q0, w.scale, out=outs[0], lse=lses[0])
    e[1].record()
    torch.cuda.synchronize()
    cmp_ms = e[0].elapsed_time(e[1]) / 20
    cmp_fl = 4.0 * w.head_dim * w.heads * w.query_tokens * n * w.blocks_per_chunk

    # Eq. 1 in full: the selection step above, then CMP and SWA (the window's chunks)
    # and the sigmoid-gated sum of the three branches (synthetic gate logits)
    o_cmp = [torch.empty_like(o) for o in outs]
    o_swa = [torch.empty_like(o) for o in outs]
    gates = torch.randn((w.query_tokens, w.heads, 3), generator=torch.Generator(device=dev).manual_seed(7),
                        device=dev)
    fused = [torch.empty_like(o) for o in outs]

    def three_branch(i, ev=None):
        j = i % len(layers)
        q, cache = layers[j]
        if ev is not None:
            ev[0].record()
        step(i)
        if ev is not None:
            ev[1].record()
        omnimem_cmp_attn(ccs[j], n, q, w.scale, out=o_cmp[j], want_lse=False)
        if ev is not None:
            ev[2].record()
        omnimem_dense_attn(cache, q, n - w.window_chunks, n, w.scale, out=o_swa[j], want_lse=False)
        if ev is not None:
            ev[3].record()
        omnimem_gated_combine(o_cmp[j], outs[j], o_swa[j], gates, out=fused[j])
        if ev is not None:
            ev[4].record()

    for i in range(200):
        three_branch(i)
    torch.cuda.synchronize()
    reps = 100
    evs3 = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(reps)]
    t0.record()
    for i in range(reps):
        three_branch(i)
    t1.record()
    torch.cuda.synchronize()
    tb_ms = t0.elapsed_time(t1) / reps
    for i in range(reps):
        three_branch(i, evs3[i])
    torch.cuda.synchronize()
    med3 = lambda a, b: float(np.median([e[a].elapsed_time(e[b]) for e in evs3]))

    # selection by probability-averaged scores (score_mode SCORE_PROB), the workload's
    # groups and the paper's G = 15 with top-4
    from paper_2605_30519_amd import SCORE_PROB
    q0, c0 = layers[0]
    prob = {}
    for name, G, Kp in (("workload_groups", w.group_size, K), ("g15_top4", 15, 4)):
        pp = select_params(Kp, G, w.window_chunks, w.awe_min_outside_chunks, w.scale, SCORE_PROB)
        wsp = workspace_tensor(omnimem_select_workspace_bytes(c0, w.query_tokens, pp), dev)
        sp = None
        for _ in range(20):
            sp = omnimem_select_compressed(c0, ccs[0], q0, Kp, G, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                                           workspace=wsp, out=sp, want_score=False, score_mode=SCORE_PROB)
        e[0].record()
        for _ in range(50):
            omnimem_select_compressed(c0, ccs[0], q0, Kp, G, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                                      workspace=wsp, out=sp, want_score=False, score_mode=SCORE_PROB)
        e[1].record()
        torch.cuda.synchronize()
        pms = e[0].elapsed_time(e[1]) / 50
        logit_fl = 2.0 * w.query_tokens * n * w.blocks_per_chunk * w.head_dim * w.heads
        prob[name] = {"group_size": G, "top_k": Kp, "select_ms": round(pms, 4),
                      "logit_tflops": round(logit_fl / (pms * 1e-3) / 1e12, 2),
                      "mfma_tflops": round(4 * logit_fl / (pms * 1e-3) / 1e12, 2)}
        del wsp
    return {"step": "pool the newest chunk + select from the pooled keys + sparse attention",
            "ms_per_chunk_layer": round(ms, 4),
            "effective_tflops": round(float(np.mean(flops)) / (ms * 1e-3) / 1e12, 2),
            "compress_chunk_ms": round(med(0, 1), 4), "select_compressed_ms": round(med(1, 2), 4),
            "sparse_attn_ms": round(med(2, 3), 4),
            "cmp_attn_ms": round(cmp_ms, 4), "cmp_attn_tflops": round(cmp_fl / (cmp_ms * 1e-3) / 1e12, 2),
            "three_branch": {"step": "the compressed chunk step + CMP + SWA over the window + gated fusion (Eq. 1)",
                             "ms_per_chunk_layer": round(tb_ms, 4), "selection_step_ms": round(med3(0, 1), 4),
                             "cmp_attn_ms": round(med3(1, 2), 4), "swa_attn_ms": round(med3(2, 3), 4),
                             "gated_combine_ms": round(med3(3, 4), 4)},
            "prob_scores": prob}


def select_cache_state(layers, sels, ws, w, sbytes, reps=30):
    """Select alone, HIP events around each call, layers in rotation: (a) after a
    1 GiB read that evicts the MALL with clean lines; (b) after a 1 GiB write, which
    leaves the MALL full of dirty lines that the select's reads must first write
    back; (c) warm, one layer back to back; (d) as (a), replayed from a HIP graph."""
    import numpy as np
    import torch

    from paper_2605_30519_amd import omnimem_select
    K = w.top_k
    scratch = torch.empty(1 << 28, dtype=torch.float32, device=layers[0][0].device)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(3 * reps)]
    total = torch.zeros((), dtype=torch.float32, device=scratch.device)

    def sel(i, e):
        q, cache = layers[i % len(layers)]
        e[0].record()
        omnimem_select(cache, q, K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale, workspace=ws,
                       out=sels[i % len(layers)], want_score=False)
        e[1].record()

    scratch.fill_(1.0)
    for i in range(reps):
        total += scratch.sum()
        sel(i, ev[i])
    for i in range(reps):
        scratch.fill_(float(i))
        sel(i, ev[reps + i])
    for _ in range(3):
        sel(0, ev[2 * reps])
    for i in range(reps):
        sel(0, ev[2 * reps + i])
    torch.cuda.synchronize()
    # (d) as (a), each layer's select replayed from a HIP graph (no launch gaps
    # between its three kernels)
    graphs = []
    for i in range(len(layers)):
        g = torch.cuda.CUDAGraph()
        q, cache = layers[i]
        with torch.cuda.graph(g):
            omnimem_select(cache, q, K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale,
                           workspace=ws, out=sels[i], want_score=False)
        graphs.append(g)
    torch.cuda.synchronize()
    evg = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps)]
    for i in range(reps):
        total += scratch.sum()
        evg[i][0].record()
        graphs[i % len(layers)].replay()
        evg[i][1].record()
    torch.cuda.synchronize()
    del graphs
    out = {}
    for name, part in (("mall_evicted_by_1gib_read", ev[:reps]), ("after_1gib_write_dirty_mall", ev[reps:2 * reps]),
                       ("warm_same_layer", ev[2 * reps:]), ("mall_evicted_graph_replay", evg)):
        t = np.array([a.elapsed_time(b) for a, b in part])
        gbs = sbytes / (float(np.median(t)) * 1e-3) / 1e9
        out[name] = {"select_ms": round(float(np.median(t)), 4),
                     "p10_p90": [round(float(np.percentile(t, 10)), 4), round(float(np.percentile(t, 90)), 4)],
                     "achieved_gbs": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
    del scratch
    return out


def small_group_measure(dev, reps=50):
    """The paper's memory-module setting on the Wan2.1-1.3B-shaped layer: query
    groups of 15 rows (312 groups), the top-4 blocks per (head, group), a window of
    3 chunks excluded once 3 chunks lie outside it; 20 cached chunks in 64-token
    blocks.  Select and selection attention timed as in the main run."""
    import numpy as np
    import torch

    from paper_2605_30519_amd import omnimem_select, omnimem_sparse_attn, synth
    w = synth.Workload("wan1.3b_g15", 12, 128, 4680, 4680, 64, 20, 20, 4, 15, 3, 3, torch.bfloat16, True, 1, 21)
    x = synth.make_layer(w, 0, device=dev)
    c = synth.page_layer(x.k, x.v, w.block_size, seed=3)
    del x.k, x.v
    sel = omnimem_select(c, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    out = torch.empty_like(x.q)
    lse = torch.empty((w.heads, w.query_tokens), dtype=torch.float32, device=dev)
    for _ in range(100):
        omnimem_select(c, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale, out=sel,
                       want_score=False)
        omnimem_sparse_attn(c, x.q, sel.idx, sel.cnt, w.group_size, w.scale, out=out, lse=lse)
    torch.cuda.synchronize()
    e = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
    for r in range(reps):
        e[r][0].record()
        omnimem_select(c, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale, out=sel,
                       want_score=False)
        e[r][1].record()
        omnimem_sparse_attn(c, x.q, sel.idx, sel.cnt, w.group_size, w.scale, out=out, lse=lse)
        e[r][2].record()
    torch.cuda.synchronize()
    ts = float(np.median([x_[0].elapsed_time(x_[1]) for x_ in e]))
    ta = float(np.median([x_[1].elapsed_time(x_[2]) for x_ in e]))
    fl = attn_flops(sel.idx, sel.cnt, w, w.history_chunks)
    idx = sel.idx.cpu().numpy()
    gather = int((idx >= 0).sum()) * w.block_size * w.head_dim * 2 * 2
    return {"workload": "Wan2.1-1.3B-shaped layer, query groups of 15 rows (312 groups), top-4 blocks per "
                        "(head, group), 3-chunk window, 20 chunks of 64-token blocks",
            "select_ms": round(ts, 4), "sparse_attn_ms": round(ta, 4), "ms_per_chunk_layer": round(ts + ta, 4),
            "sparse_attn_tflops": round(fl / (ta * 1e-3) / 1e12, 2),
            "gathered_kv_bytes": gather, "gather_gbs": round(gather / (ta * 1e-3) / 1e9, 1)}


def lru_measure(dev, x, w, steps=60, sizes=(5, 6, 8, 10), recent=4, seed=17):
    """The GPU hot cache of App. B / App. F on the bench layer: its chunks in pinned
    host pools (allocated after binding the thread to the GPU's NUMA node), a GPU
    pool of `slots` chunk slots per head, residency per (head, chunk).

    Access pattern (synthetic, with locality): per head, 3 anchor chunks that change
    every 15 steps and one chunk drawn from a per-head set of `recent` chunks; each
    head's 64 blocks are drawn from those 4 chunks.  The window chunk, read by the
    SWA branch, is requested for every head as well.

    A step is Eq. 1's three-branch forward with reloads: the selected (head, chunk)
    pairs decoded on the GPU (Alg. 1 Step 1) and copied to the host, omnimem_lru_require,
    the CMP and SWA branches, omnimem_lru_wait, the SLC branch over the hot cache,
    and the gated fusion.  Two modes: reloads on the compute stream (serial), and on
    a second stream, overlapping the CMP and SWA branches (overlap).  HIP events on
    the compute stream bracket each step, host round trip included.  The SWA branch
    waits for the reloads only while its window chunk is not yet resident."""
    import numpy as np
    import torch

    from paper_2605_30519_amd import (CompressedCache, LruOffload, PagedKVCache, omnimem_cmp_attn,
                                      omnimem_compress_chunk, omnimem_dense_attn, omnimem_gated_combine,
                                      omnimem_numa_bind, omnimem_selected_chunks, omnimem_sparse_attn, synth)
    n, S, H, d = (int(s) for s in x.k.shape)
    B, K, Bpc = w.block_size, w.top_k, w.blocks_per_chunk
    saved_affinity = os.sched_getaffinity(0)
    node = omnimem_numa_bind(0)
    pools = []
    for t in (x.k, x.v):
        pad = Bpc * B - S
        y = torch.cat([t, torch.zeros((n, pad, H, d), dtype=t.dtype, device=t.device)], dim=1) if pad else t
        pinned = torch.empty((n * Bpc, H, B, d), dtype=t.dtype, pin_memory=True)
        pinned.copy_(y.reshape(n * Bpc, B, H, d).permute(0, 2, 1, 3).cpu())
        pools.append(pinned)
        del y
    full = synth.page_layer(x.k, x.v, B, seed=7)
    cc = CompressedCache.allocate(full, n)
    for c in range(n):
        omnimem_compress_chunk(full, c, cc)
    del full
    rng = np.random.default_rng(seed)
    win = n - w.window_chunks
    candidates = list(range(win))
    recent_sets = [rng.choice(candidates, recent, replace=False).tolist() for _ in range(H)]
    plan = []
    anchors = None
    for step in range(steps):
        if step % 15 == 0:
            anchors = [rng.choice([c for c in candidates if c not in recent_sets[h]], 3, replace=False).tolist()
                       for h in range(H)]
        idx = np.zeros((H, 1, K), np.int32)
        for h in range(H):
            chunks = anchors[h] + [int(rng.choice(recent_sets[h]))]
            blocks = np.array([c * Bpc + o for c in chunks for o in range(Bpc)])
            idx[h, 0] = np.sort(rng.choice(blocks, K, replace=False))
        plan.append(torch.tensor(idx, dtype=torch.int32, device=dev))
    cnt = torch.full((H, 1), K, dtype=torch.int32, device=dev)
    o_slc, o_cmp, o_swa, o_out = (torch.empty_like(x.q) for _ in range(4))
    lse = torch.empty((H, w.query_tokens), dtype=torch.float32, device=dev)
    gate = torch.randn((w.query_tokens, H, 3), generator=torch.Generator(device=dev).manual_seed(3), device=dev)
    slab = B * d * x.k.element_size()
    res = {"workload": f"bench layer, {n} chunks in pinned host pools, residency per (head, chunk); {steps} steps; "
                       f"per head 3 anchor chunks changing every 15 steps + 1 of {recent} recent chunks, {K} blocks "
                       f"per head drawn from them, window chunk for the SWA branch",
           "numa_node": node, "pcie_peak_gbs": 63.0, "modes": []}

    def pool_of(slots):
        return PagedKVCache(torch.empty((slots * Bpc, H, B, d), dtype=x.k.dtype, device=dev),
                            torch.empty((slots * Bpc, H, B, d), dtype=x.k.dtype, device=dev),
                            torch.zeros((H, n, Bpc), dtype=torch.int32, device=dev), S)

    # raw reload rates: every head's copy of every chunk (heads merge into whole-page
    # copies), then alternate heads only (one strided copy per head and chunk)
    for name, mask in (("whole_chunks", np.ones((H, n), np.uint8)),
                       ("every_other_head", (np.add.outer(np.arange(H), np.arange(n)) % 2 == 0).astype(np.uint8))):
        gpu = pool_of(n)
        lru = LruOffload(gpu, n, pools[0], pools[1])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        lru.require(mask)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        gbs = 2 * int(mask.sum()) * Bpc * slab / (ms * 1e-3) / 1e9
        res[f"reload_{name}_gbs"] = round(gbs, 1)
        res[f"reload_{name}_frac_of_pcie"] = round(gbs / 63.0, 3)
        lru.close()
        del gpu
    copy_stream = torch.cuda.Stream()
    for slots in sizes:
        for mode in ("serial", "overlap"):
            gpu = pool_of(slots)
            lru = LruOffload(gpu, slots, pools[0], pools[1])
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
            xs = copy_stream if mode == "overlap" else None
            for step, idx in enumerate(plan):
                evs[step][0].record()
                needed = omnimem_selected_chunks(gpu, idx, cnt).cpu()
                needed[:, win:] = 1                                 # the SWA window, every head
                # a window chunk already resident is a hit, untouched by this request's
                # reloads: the SWA branch then need not wait for them
                window_ready = all(lru.slot_of(h, c) >= 0 for h in range(H) for c in range(win, n))
                lru.require(needed, copy_stream=xs)
                omnimem_cmp_attn(cc, n, x.q, w.scale, out=o_cmp, lse=lse)
                if not window_ready:
                    lru.wait()
                omnimem_dense_attn(gpu, x.q, win, n, w.scale, out=o_swa, lse=lse)
                lru.wait()                                          # Alg. 1's WaitUntilReload
                omnimem_sparse_attn(gpu, x.q, idx, cnt, w.group_size, w.scale, out=o_slc, lse=lse)
                omnimem_gated_combine(o_cmp, o_slc, o_swa, gate, out=o_out)
                evs[step][1].record()
            torch.cuda.synchronize()
            st = lru.stats()
            t = np.array([e[0].elapsed_time(e[1]) for e in evs])
            pairs = st["hits"] + st["misses"]
            res["modes"].append({"lru_chunks_per_head": slots, "mode": mode,
                                 "hit_rate": round(st["hits"] / max(1, pairs), 4),
                                 "reloaded_pairs": st["misses"],
                                 "reloaded_gb_per_step": round(st["bytes_reloaded"] / steps / 1e9, 4),
                                 "ms_per_step": round(float(t.mean()), 4),
                                 "ms_per_step_median": round(float(np.median(t)), 4),
                                 "gpu_pool_gb": round(2 * slots * Bpc * H * slab / 1e9, 3)})
            lru.close()
            del gpu
    os.sched_setaffinity(0, saved_affinity)
    return res


def ramp_measure(dev, layers_n=30, warm_passes=20):
    """The full chunk step of a 30-layer model as its history grows from 1 to 60
    chunks: for each history length n, select + sparse attention over all 30 layers
    (independent seeds, every layer's K/V resident), timed as one pass."""
    import numpy as np
    import torch

    from paper_2605_30519_amd import omnimem_select, omnimem_select_workspace_bytes, omnimem_sparse_attn, synth
    from paper_2605_30519_amd import select_params
    from paper_2605_30519_amd.omnimem import Selection, workspace_tensor
    w = synth.WORKLOADS["wan1.3b_30layer"]
    H, R, K, N = w.heads, w.groups, w.top_k, w.history_chunks
    caches, rels = [], []
    for layer in range(layers_n):
        x = synth.make_layer(w, layer, device=dev)
        caches.append(synth.page_layer(x.k, x.v, w.block_size, seed=300 + layer))
        rels.append(x.rel)
        del x
    resident_gb = sum(c.k_pages.numel() * c.k_pages.element_size() * 2 for c in caches) / 1e9
    params = select_params(K, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
    ws = workspace_tensor(omnimem_select_workspace_bytes(caches[0], w.query_tokens, params), dev)
    sel = Selection(torch.empty((H, R, K), dtype=torch.int32, device=dev),
                    torch.empty((H, R), dtype=torch.int32, device=dev), None, 0)
    out = torch.empty((w.query_tokens, H, w.head_dim), dtype=w.dtype, device=dev)
    lse = torch.empty((H, w.query_tokens), dtype=torch.float32, device=dev)

    def chunk_step(n, qs, flops=None):
        awe = 0
        for layer in range(layers_n):
            omnimem_select(caches[layer], qs[layer], K, w.group_size, w.window_chunks, w.awe_min_outside_chunks,
                           w.scale, num_chunks=n, workspace=ws, out=sel, want_score=False)
            omnimem_sparse_attn(caches[layer], qs[layer], sel.idx, sel.cnt, w.group_size, w.scale, num_chunks=n,
                                out=out, lse=lse)
            if flops is not None:
                flops.append(attn_flops(sel.idx, sel.cnt, w, n) + score_flops(w, n))
            awe = sel.awe_active
        return awe

    q60 = [synth.queries(w, layer, N, rels[layer], dev) for layer in range(layers_n)]
    for _ in range(warm_passes):  # the clock's ramp, on the longest history
        chunk_step(N, q60)
    del q60
    torch.cuda.synchronize()
    steps = []
    for n in range(1, N + 1):
        qs = [synth.queries(w, layer, n, rels[layer], dev) for layer in range(layers_n)]
        flops = []
        chunk_step(n, qs, flops)  # untimed: selection results for the flop count
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        awe = chunk_step(n, qs)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        steps.append({"history_chunks": n, "awe_active": int(awe),
                      "ms_per_chunk_layer": round(ms / layers_n, 4),
                      "effective_tflops": round(float(np.sum(flops)) / (ms * 1e-3) / 1e12, 2)})
        del qs
    total = sum(x["ms_per_chunk_layer"] for x in steps) * layers_n
    return {"workload": "30 layers of the Wan2.1-1.3B-shaped attention layer, history 1 -> 60 chunks, "
                        "one chunk step (select + sparse attention over every layer) per history length",
            "layers": layers_n, "resident_kv_gb": round(resident_gb, 1), "total_ms": round(total, 2),
            "awe_first_on": next((x["history_chunks"] for x in steps if x["awe_active"]), None),
            "steps": steps}


def hip_probes(dev):
    """The HIP roofline probes of libomnimem_probe.so: MFMA issue loops (4
    independent v_mfma_f32_32x32x16_bf16 chains per wave, smooth or random operands;
    the same with the fp32 16x16x4 and 32x32x2 MFMAs), the attention kernel's MFMA
    slot with its softmax VALU work, a streaming read and a streaming copy of 1 GiB.  Best of a few launch shapes each; HIP events on the
    launch stream."""
    import ctypes

    import torch

    from paper_2605_30519_amd import _build
    P = ctypes.CDLL(_build.PROBE_LIB)
    P.omnimem_probe_mfma_bf16.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_void_p]
    P.omnimem_probe_mfma_f32.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_void_p, ctypes.c_void_p]
    P.omnimem_probe_softmax_slot.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                             ctypes.c_void_p]
    P.omnimem_probe_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_void_p]
    P.omnimem_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    sink = torch.zeros(4, dtype=torch.float32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(call, reps):
        for _ in range(2):
            assert call() == 0
        e0.record()
        for _ in range(reps):
            assert call() == 0
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    out = {"probe_library": os.path.basename(_build.PROBE_LIB)}
    for operands, key in ((0, "mfma_bf16"), (1, "mfma_bf16_random")):
        mfma = []
        for wgs, wps, iters in ((256, 1, 100000), (1024, 1, 25000), (512, 2, 50000)):
            ms = timed(lambda: P.omnimem_probe_mfma_bf16(operands, iters, wgs, wps, ctypes.c_void_p(sink.data_ptr()),
                                                         stream), 5)
            flops = wgs * 4 * wps * iters * 4 * 32768.0
            mfma.append({"workgroups": wgs, "waves_per_simd": wps, "tflops": round(flops / (ms * 1e-3) / 1e12, 1)})
        best = max(m["tflops"] for m in mfma)
        out[key] = mfma
        out[key + "_tflops"] = best
        # 2.5 PFLOP/s bf16 is 1024 flops per cycle per SIMD on 1024 SIMDs at 2.4 GHz
        out[key.replace("mfma_bf16", "mfma_implied_clock_ghz")] = round(best / PEAK_BF16_TFLOPS * 2.4, 3)
    # the attention kernel's MFMA slot (MFMA + fma + exp + add + half a pack), operands in
    # registers or the A operand from LDS; one wave per SIMD, 8 slots per round
    for lds, key in ((0, "softmax_slot"), (1, "softmax_slot_lds")):
        iters = 25000
        ms = timed(lambda: P.omnimem_probe_softmax_slot(lds, iters, 256, ctypes.c_void_p(sink.data_ptr()), stream), 5)
        out[key + "_tflops"] = round(256 * 4 * iters * 8 * 32768.0 / (ms * 1e-3) / 1e12, 1)
    # fp32 MFMA (the selection's score products): 16x16x4 and 32x32x2, against 157.3 TF
    f32 = []
    for shape, fl in ((0, 2048.0), (1, 4096.0)):
        for wgs, wps, iters in ((256, 1, 50000), (512, 2, 25000)):
            ms = timed(lambda: P.omnimem_probe_mfma_f32(shape, iters, wgs, wps, ctypes.c_void_p(sink.data_ptr()),
                                                        stream), 5)
            flops = wgs * 4 * wps * iters * 4 * fl
            f32.append({"shape": ["16x16x4", "32x32x2"][shape], "workgroups": wgs, "waves_per_simd": wps,
                        "tflops": round(flops / (ms * 1e-3) / 1e12, 1)})
    out["mfma_f32"] = f32
    out["mfma_f32_tflops"] = max(m["tflops"] for m in f32)
    nbytes = 1 << 30
    a = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
    b = torch.empty_like(a)
    reads, copies = [], []
    for wgs in (1024, 2048, 4096, 8192):
        ms = timed(lambda: P.omnimem_probe_read(ctypes.c_void_p(a.data_ptr()), nbytes, wgs,
                                                ctypes.c_void_p(sink.data_ptr()), stream), 10)
        reads.append({"workgroups": wgs, "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1)})
        ms = timed(lambda: P.omnimem_probe_copy(ctypes.c_void_p(a.data_ptr()), ctypes.c_void_p(b.data_ptr()), nbytes,
                                                wgs, stream), 10)
        copies.append({"workgroups": wgs, "gbs": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)})
    out["hbm_read"] = reads
    out["hbm_read_gbs"] = max(r["gbs"] for r in reads)
    out["hbm_copy"] = copies
    out["hbm_copy_gbs"] = max(c["gbs"] for c in copies)
    del a, b
    return out


def probe_peaks(dev, result):
    """Achievable peaks on this GPU, measured next to the spec ones: the HIP roofline
    probes (MFMA issue loop, streaming read and copy), a torch device copy and a
    large bf16 GEMM (the vendor library's MFMA rate)."""
    import torch
    out = {"hip": hip_probes(dev)}
    a = torch.empty(1 << 29, dtype=torch.bfloat16, device=dev).fill_(1.0)  # 1 GiB
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    reps = 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    out["torch_copy_gbs"] = round(2 * a.numel() * 2 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del a, b
    m = 8192
    x = torch.randn((m, m), device=dev).to(torch.bfloat16)
    y = torch.randn((m, m), device=dev).to(torch.bfloat16)
    z = torch.empty((m, m), dtype=torch.bfloat16, device=dev)
    for _ in range(20):
        torch.matmul(x, y, out=z)
    e0.record()
    for _ in range(reps):
        torch.matmul(x, y, out=z)
    e1.record()
    torch.cuda.synchronize()
    out["bf16_gemm_tflops"] = round(2.0 * m ** 3 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e12, 1)
    out["gemm_shape"] = f"{m}x{m}x{m} bf16, torch.matmul"
    att = result["stages"]["attention_roofline"]["achieved"]
    sel = result["stages"]["select_roofline"]["achieved"]
    out["attention_frac_of_mfma_probe"] = round(att / out["hip"]["mfma_bf16_tflops"], 4)
    out["attention_frac_of_mfma_random_probe"] = round(att / out["hip"]["mfma_bf16_random_tflops"], 4)
    out["attention_frac_of_softmax_slot_lds_probe"] = round(att / out["hip"]["softmax_slot_lds_tflops"], 4)
    out["attention_frac_of_gemm"] = round(att / out["bf16_gemm_tflops"], 4)
    out["select_frac_of_read_probe"] = round(sel / out["hip"]["hbm_read_gbs"], 4)
    return out


def stress_comparison(dev):
    import numpy as np
    import torch

    from paper_2605_30519_amd import omnimem_select, omnimem_sparse_attn, omnimem_union_gather_attn, synth
    from paper_2605_30519_amd.omnimem import omnimem_union_workspace_bytes, workspace_tensor
    w = synth.WORKLOADS["wan14b_stress"]
    x = synth.make_layer(w, 0, device=dev)
    c = synth.page_layer(x.k, x.v, w.block_size, seed=55)
    del x.k, x.v
    uws = workspace_tensor(omnimem_union_workspace_bytes(c), dev)
    reps = 5
    e = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps + 1)]
    for r in range(reps + 1):
        e[r][0].record()
        s = omnimem_select(c, x.q, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks, w.scale)
        e[r][1].record()
        out, lse = omnimem_sparse_attn(c, x.q, s.idx, s.cnt, w.group_size, w.scale)
        e[r][2].record()
        uo, ul, ub = omnimem_union_gather_attn(c, x.q, s.idx, s.cnt, w.group_size, w.scale, workspace=uws)
        e[r][3].record()
    torch.cuda.synchronize()
    med = lambda a, b: float(np.median([e[r][a].elapsed_time(e[r][b]) for r in range(1, reps + 1)]))
    nb = w.history_chunks * w.blocks_per_chunk
    U = int(ub.item())
    idx = s.idx.cpu().numpy()
    per_head = [len(set(idx[h][idx[h] >= 0].tolist())) for h in range(w.heads)]
    slab = w.block_size * w.head_dim * 2 * 2          # K and V of one (block, head), bf16
    t_sel, t_att, t_uni = med(0, 1), med(1, 2), med(2, 3)
    fl = attn_flops(s.idx, s.cnt, w, w.history_chunks)
    sbytes = select_bytes(w, w.history_chunks, s.awe_active)
    merged = w.heads * U * slab
    return {"workload": "Wan2.1-14B-shaped layer: 40 heads x 128, 4680-token chunk, 60-chunk history "
                        "(280,800 keys) in 128-token blocks, top-32 per (head, group), 3 query groups of 1560 rows",
            "select_ms": round(t_sel, 4), "select_gbs": round(sbytes / (t_sel * 1e-3) / 1e9, 1),
            "select_frac_of_hbm": round(sbytes / (t_sel * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "scattered_attn_ms": round(t_att, 4),
            "scattered_attn_tflops": round(fl / (t_att * 1e-3) / 1e12, 2),
            "scattered_attn_frac_of_mfma": round(fl / (t_att * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "ms_per_chunk_layer": round(t_sel + t_att, 4),
            "union_gather_attn_ms": round(t_uni, 4),
            "union_blocks": U, "candidate_blocks": nb - w.window_chunks * w.blocks_per_chunk,
            "union_fraction": round(U / (nb - w.window_chunks * w.blocks_per_chunk), 4),
            "scattered_kv_bytes": int(sum(per_head)) * slab, "merged_buffer_bytes": merged,
            "merged_over_scattered": round(merged / max(1, int(sum(per_head)) * slab), 2),
            "union_gather_over_scattered_time": round(t_uni / t_att, 2),
            "outputs_bit_equal": bool(torch.equal(uo.view(torch.int16), out.view(torch.int16)))}


def oracle_extrapolations(dev, rows=48, seed=9):
    """The fp64 oracle where a whole run is far too long for the CPU: timed on a
    deterministic sample and scaled up, each result labelled extrapolated.
    - dense attention over 120 chunks (561,600 keys): `rows` sampled (head, row)
      pairs, scaled to all 56,160;
    - the 30-layer ramp: one layer's selection (whole) and sparse attention
      (`rows` sampled pairs) at history 1, 4, 30 and 60, interpolated linearly over
      n = 1..60 and multiplied by 30 layers."""
    import numpy as np
    import torch

    import oracle
    from paper_2605_30519_amd import synth
    rng = np.random.default_rng(seed)
    out = {}
    wl = synth.WORKLOADS["wan1.3b_long"]
    x = synth.make_layer(wl, 0, device=dev)
    q, k, v = x.q.cpu(), x.k.cpu(), x.v.cpu()
    del x
    torch.cuda.empty_cache()
    total = wl.heads * wl.query_tokens
    hs, qs = rng.integers(0, wl.heads, rows), rng.integers(0, wl.query_tokens, rows)
    t0 = time.perf_counter()
    oracle.dense_attn(q, k, v, wl.block_size, 0, wl.history_chunks, wl.scale, hs=hs, qs=qs)
    dt = time.perf_counter() - t0
    out["dense_n120_s"] = {"value": round(dt * total / rows, 1), "sample_rows": rows, "sample_s": round(dt, 2),
                           "label": "extrapolated"}
    del q, k, v
    w = synth.WORKLOADS["wan1.3b_30layer"]
    x = synth.make_layer(w, 0, device=dev)
    k, v = x.k.cpu(), x.v.cpu()
    total = w.heads * w.query_tokens
    per_step = {}
    for n in (1, 4, 30, 60):
        q = synth.queries(w, 0, n, x.rel, dev).cpu()
        t0 = time.perf_counter()
        ref = oracle.select(q, k[:n], w.block_size, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks,
                            w.scale)
        t1 = time.perf_counter()
        hs, qs = rng.integers(0, w.heads, rows), rng.integers(0, w.query_tokens, rows)
        oracle.sparse_attn(q, k[:n], v[:n], w.block_size, ref["idx"], ref["cnt"], w.group_size, w.scale, hs=hs, qs=qs)
        t2 = time.perf_counter()
        per_step[n] = (t1 - t0) + (t2 - t1) * total / rows
    del x, k, v
    torch.cuda.empty_cache()
    ns = sorted(per_step)
    ramp = sum(float(np.interp(n, ns, [per_step[m] for m in ns])) for n in range(1, w.history_chunks + 1))
    out["ramp_30_layers_s"] = {"value": round(ramp * w.layers, 1),
                               "per_step_s": {str(n): round(t, 2) for n, t in per_step.items()},
                               "label": "extrapolated"}
    return out


def cpu_baseline(x, w, step_flops, reps=3):
    """The fp64 oracle on the host cores: one whole chunk-layer (selection over the
    full history for every head, then selection attention for every query row of
    every head), repeated `reps` times; the median time is reported."""
    import numpy as np

    import oracle

    q, k, v = x.q.cpu(), x.k.cpu(), x.v.cpu()
    oracle.lib()
    hh, qq = np.meshgrid(np.arange(w.heads), np.arange(w.query_tokens), indexing="ij")
    times, sel_t = [], []
    for _ in range(reps):
        t0 = time.perf_counter()
        ref = oracle.select(q, k, w.block_size, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks,
                            w.scale)
        t1 = time.perf_counter()
        oracle.sparse_attn(q, k, v, w.block_size, ref["idx"], ref["cnt"], w.group_size, w.scale, hs=hh.ravel(),
                           qs=qq.ravel())
        t2 = time.perf_counter()
        times.append(t2 - t0)
        sel_t.append(t1 - t0)
    full_s = float(np.median(times))
    threads = oracle.lib().oracle_max_threads()
    # the same on one core: selection whole, attention on every 16th query row
    # (all heads), scaled to all rows
    with oracle.threads(1):
        t0 = time.perf_counter()
        ref = oracle.select(q, k, w.block_size, w.top_k, w.group_size, w.window_chunks, w.awe_min_outside_chunks,
                            w.scale)
        t1 = time.perf_counter()
        sub = qq.ravel() % 16 == 0
        oracle.sparse_attn(q, k, v, w.block_size, ref["idx"], ref["cnt"], w.group_size, w.scale,
                           hs=hh.ravel()[sub], qs=qq.ravel()[sub])
        t2 = time.perf_counter()
    attn1 = (t2 - t1) * sub.size / int(sub.sum())
    return {"value": round(step_flops / full_s / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"one whole chunk-layer of the same workload (selection for all {w.heads} heads over the "
                      f"20-chunk history + selection attention for all {w.heads * w.query_tokens} (head, row) "
                      f"pairs), fp64, median of {reps} runs, {sum(times):.1f} s in total",
            "ms_per_chunk_layer": round(full_s * 1e3, 1), "select_s": round(float(np.median(sel_t)), 3),
            "sparse_attn_s": round(float(np.median(times) - np.median(sel_t)), 3),
            "one_core": {"select_s": round(t1 - t0, 3), "sparse_attn_s_extrapolated": round(attn1, 2),
                         "ms_per_chunk_layer_extrapolated": round((t1 - t0 + attn1) * 1e3, 1),
                         "sample": "selection whole; attention on every 16th query row of every head, "
                                   "time scaled to all rows (extrapolated)"}}


if __name__ == "__main__":
    main()
