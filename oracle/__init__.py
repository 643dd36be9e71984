"""fp64 CPU oracle for OmniMem's memory-retrieval attention step (arXiv 2605.30519).

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's
CPU-baseline leg use this package; the product library never does.  It shares no
code with the GPU path.  The arithmetic lives in ``omnimem_oracle.c`` (plain C,
double precision); this module only marshals arrays through ctypes.

Data model (App. A, App. C of the paper):
  q       : [Lq, H, d]       current-chunk queries
  k, v    : [n, S, H, d]     history, chunk by chunk (logical order, no paging)
  resident: [n * Bpc] bool   False = the block is not on the GPU and is skipped
Arrays may be numpy float64/float32 or torch float64/float32/bfloat16 (CPU);
bf16 values are passed as their raw bit patterns and widened exactly in C.

Parity pins: every function here is pinned by ``tests/test_oracle_pins.py``
(worked examples, closed forms, brute force and invariants).
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "omnimem_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_vp = ctypes.c_void_p


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (OpenMP, -O2).  Returns the library path."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _configure(L):
    c_int = ctypes.c_int
    L.oracle_blocks_per_chunk.argtypes = [c_int, c_int]
    L.oracle_awe_active.argtypes = [c_int] * 5
    L.oracle_candidates.argtypes = [c_int, c_int, c_int, c_int, c_int, _u8p, _u8p]
    L.oracle_pool_keys.argtypes = [c_int] * 5 + [c_int, _vp, _f64p]
    L.oracle_proxy_queries.argtypes = [c_int] * 4 + [c_int, _vp, _f64p]
    L.oracle_query_scores.argtypes = [c_int] * 6 + [c_int, _vp, c_int, _vp, ctypes.c_double, _f64p]
    L.oracle_select.argtypes = ([c_int] * 6 + [c_int, _vp, c_int, _vp, _u8p] + [c_int] * 4 +
                                [ctypes.c_double, c_int, c_int, _i32p, _i32p, _f64p, _f64p])
    L.oracle_select_prob.argtypes = ([c_int] * 5 + [c_int, _vp, _f64p, _u8p] + [c_int] * 4 +
                                     [ctypes.c_double, c_int, c_int, _i32p, _i32p, _f64p, _f64p])
    L.oracle_sparse_attn.argtypes = ([c_int] * 6 + [c_int, _vp, c_int, _vp, _vp, _u8p, _i32p, _i32p,
                                     c_int, c_int, ctypes.c_double, c_int, _i32p, _i32p, _f64p, _f64p])
    L.oracle_dense_attn.argtypes = ([c_int] * 6 + [c_int, _vp, c_int, _vp, _vp, _u8p, c_int, c_int,
                                    ctypes.c_double, c_int, _i32p, _i32p, _f64p, _f64p])
    L.oracle_union.argtypes = [c_int, c_int, c_int, ctypes.c_int64, _i32p, _i32p, _i32p, _i32p]
    L.oracle_set_threads.argtypes = [c_int]
    L.oracle_max_threads.restype = c_int
    return L


@contextlib.contextmanager
def threads(n: int):
    """Run the oracle's OpenMP regions on n threads inside the block (timing only)."""
    L = lib()
    prev = L.oracle_max_threads()
    L.oracle_set_threads(n)
    try:
        yield
    finally:
        L.oracle_set_threads(prev)


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build()
            _lib = _configure(ctypes.CDLL(_LIB_PATH))
    return _lib


@contextlib.contextmanager
def using_library(path: str):
    """Temporarily route every oracle call through another build of the C source
    (the mutation tests load deliberately broken copies this way)."""
    global _lib
    lib()
    alt = _configure(ctypes.CDLL(path))
    with _lock:
        prev, _lib = _lib, alt
    try:
        yield
    finally:
        with _lock:
            _lib = prev


# ----------------------------------------------------------------- marshalling

def _as_input(x):
    """Return (element-type code, contiguous host array kept alive, pointer)."""
    try:
        import torch
    except ImportError:  # pragma: no cover
        torch = None
    if torch is not None and isinstance(x, torch.Tensor):
        x = x.detach().cpu().contiguous()
        if x.dtype == torch.bfloat16:
            arr = x.view(torch.int16).numpy()
            return 2, arr, arr.ctypes.data_as(_vp)
        if x.dtype == torch.float32:
            arr = x.numpy()
            return 1, arr, arr.ctypes.data_as(_vp)
        arr = x.to(torch.float64).numpy()
        return 0, arr, arr.ctypes.data_as(_vp)
    arr = np.ascontiguousarray(x)
    if arr.dtype == np.float32:
        return 1, arr, arr.ctypes.data_as(_vp)
    arr = np.ascontiguousarray(arr, dtype=np.float64)
    return 0, arr, arr.ctypes.data_as(_vp)


def _i32(x):
    arr = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    return arr, arr.ctypes.data_as(_i32p)


def _u8_or_null(resident):
    if resident is None:
        return None, ctypes.cast(None, _u8p)
    arr = np.ascontiguousarray(np.asarray(resident, dtype=np.uint8))
    return arr, arr.ctypes.data_as(_u8p)


def _check(rc, what):
    if rc < 0:
        raise ValueError(f"oracle {what}: invalid arguments")
    return rc


def _kv_shape(k):
    n, S, H, d = (int(s) for s in k.shape)
    return n, S, H, d


# ------------------------------------------------------------------ functions

def blocks_per_chunk(S: int, B: int) -> int:
    return _check(lib().oracle_blocks_per_chunk(S, B), "blocks_per_chunk")


def awe_active(n: int, E: int, T_out: int, K: int, Bpc: int) -> bool:
    """Adaptive Window Exclusion state (Eq. 2 guard and App. B activation rule)."""
    return bool(_check(lib().oracle_awe_active(n, E, T_out, K, Bpc), "awe_active"))


def candidates(n, Bpc, K, E, T_out, resident=None):
    """Candidate mask Omega over the n*Bpc history blocks (Eq. 2).  Returns (omega, awe)."""
    keep, rp = _u8_or_null(resident)
    omega = np.zeros(max(n * Bpc, 1), dtype=np.uint8)
    awe = _check(lib().oracle_candidates(n, Bpc, K, E, T_out, rp, omega.ctypes.data_as(_u8p)), "candidates")
    return omega[: n * Bpc].astype(bool), bool(awe)


def pool_keys(k, B: int):
    """Block-mean pooled keys, [H, n*Bpc, d] float64."""
    n, S, H, d = _kv_shape(k)
    et, keep, p = _as_input(k)
    Bpc = blocks_per_chunk(S, B)
    out = np.zeros((H, n * Bpc, d))
    _check(lib().oracle_pool_keys(H, d, S, n, B, et, p, out.ctypes.data_as(_f64p)), "pool_keys")
    return out


def proxy_queries(q, G_q: int):
    """Group-mean proxy queries, [H, R, d] float64 (Eq. 3)."""
    Lq, H, d = (int(s) for s in q.shape)
    et, keep, p = _as_input(q)
    R = -(-Lq // G_q)
    out = np.zeros((H, R, d))
    _check(lib().oracle_proxy_queries(H, d, Lq, G_q, et, p, out.ctypes.data_as(_f64p)), "proxy_queries")
    return out


def query_scores(q, k, B: int, scale: float):
    """Per-query compression scores s[h, q, b] (Eq. 2), [H, Lq, n*Bpc] float64."""
    n, S, H, d = _kv_shape(k)
    Lq = int(q.shape[0])
    etq, kq, pq = _as_input(q)
    etk, kk, pk = _as_input(k)
    Bpc = blocks_per_chunk(S, B)
    out = np.zeros((H, Lq, n * Bpc))
    _check(lib().oracle_query_scores(H, d, S, n, B, Lq, etq, pq, etk, pk, scale, out.ctypes.data_as(_f64p)),
           "query_scores")
    return out


def select(q, k, B: int, top_k: int, group_size: int, window_chunks: int, awe_min_outside_chunks: int,
           scale: float, resident=None, heads=None, want_all_scores=False):
    """Query-shared top-K block selection with Adaptive Window Exclusion (Eq. 2, Eq. 3).

    Returns dict(idx [H,R,K] int32 ascending with -1 padding, cnt [H,R], score [H,R,K] float64,
    awe bool, all_scores [H,R,N_b] (NaN outside Omega) if requested).  ``heads`` = (h0, h1)
    restricts the computation to a head range (other rows are left at -1 / 0)."""
    n, S, H, d = _kv_shape(k)
    Lq = int(q.shape[0])
    R = -(-Lq // group_size)
    Bpc = blocks_per_chunk(S, B)
    h0, h1 = (0, H) if heads is None else heads
    etq, kq, pq = _as_input(q)
    etk, kk, pk = _as_input(k)
    keep, rp = _u8_or_null(resident)
    idx = np.full((H, R, top_k), -1, dtype=np.int32)
    cnt = np.zeros((H, R), dtype=np.int32)
    score = np.full((H, R, top_k), -np.inf)
    alls = np.zeros((H, R, n * Bpc)) if want_all_scores else None
    awe = lib().oracle_select(H, d, S, n, B, Lq, etq, pq, etk, pk, rp, top_k, group_size, window_chunks,
                              awe_min_outside_chunks, scale, h0, h1, idx.ctypes.data_as(_i32p),
                              cnt.ctypes.data_as(_i32p), score.ctypes.data_as(_f64p),
                              alls.ctypes.data_as(_f64p) if alls is not None else ctypes.cast(None, _f64p))
    _check(awe, "select")
    out = dict(idx=idx, cnt=cnt, score=score, awe=bool(awe))
    if alls is not None:
        out["all_scores"] = alls
    return out


def select_prob(q, kc, n: int, Bpc: int, top_k: int, group_size: int, window_chunks: int,
                awe_min_outside_chunks: int, scale: float, resident=None, heads=None, want_all_scores=False):
    """Selection by the probability-averaged compression score: each query's softmax over
    all n*Bpc pooled keys kc ([H, n*Bpc, d], float64), averaged over its group (Eq. 3),
    then the top-K over Omega (Eq. 2).  Same outputs as ``select``; the scores are the
    group-mean probabilities."""
    kc = np.ascontiguousarray(np.asarray(kc, dtype=np.float64))
    H, N, d = (int(s) for s in kc.shape)
    if N != n * Bpc:
        raise ValueError(f"kc holds {N} pooled keys, expected n*Bpc = {n * Bpc}")
    Lq = int(q.shape[0])
    R = -(-Lq // group_size)
    h0, h1 = (0, H) if heads is None else heads
    etq, kq, pq = _as_input(q)
    keep, rp = _u8_or_null(resident)
    idx = np.full((H, R, top_k), -1, dtype=np.int32)
    cnt = np.zeros((H, R), dtype=np.int32)
    score = np.full((H, R, top_k), -np.inf)
    alls = np.zeros((H, R, N)) if want_all_scores else None
    awe = lib().oracle_select_prob(H, d, n, Bpc, Lq, etq, pq, kc.ctypes.data_as(_f64p), rp, top_k, group_size,
                                   window_chunks, awe_min_outside_chunks, scale, h0, h1, idx.ctypes.data_as(_i32p),
                                   cnt.ctypes.data_as(_i32p), score.ctypes.data_as(_f64p),
                                   alls.ctypes.data_as(_f64p) if alls is not None else ctypes.cast(None, _f64p))
    _check(awe, "select_prob")
    out = dict(idx=idx, cnt=cnt, score=score, awe=bool(awe))
    if alls is not None:
        out["all_scores"] = alls
    return out


def _rows(H, Lq, hs, qs):
    if hs is None:
        hh, qq = np.meshgrid(np.arange(H), np.arange(Lq), indexing="ij")
        hs, qs = hh.ravel(), qq.ravel()
    return _i32(hs), _i32(qs)


def sparse_attn(q, k, v, B: int, idx, cnt, group_size: int, scale: float, resident=None, hs=None, qs=None):
    """Selection attention over per-(head, group) block lists (Alg. 1, Step 2).

    Computes the sampled (head, query) rows (hs[i], qs[i]) -- all rows if None.
    Returns (out [m, d] float64, lse [m] float64, hs, qs)."""
    n, S, H, d = _kv_shape(k)
    Lq = int(q.shape[0])
    idx_a, idx_p = _i32(idx)
    cnt_a, cnt_p = _i32(cnt)
    top_k = int(idx_a.shape[-1])
    (hs_a, hs_p), (qs_a, qs_p) = _rows(H, Lq, hs, qs)
    m = int(hs_a.shape[0])
    etq, kq, pq = _as_input(q)
    etk, kk, pk = _as_input(k)
    etv, kv, pv = _as_input(v)
    if etk != etv:
        raise ValueError("k and v must share a dtype")
    keep, rp = _u8_or_null(resident)
    out = np.zeros((max(m, 1), d))
    lse = np.zeros(max(m, 1))
    _check(lib().oracle_sparse_attn(H, d, S, n, B, Lq, etq, pq, etk, pk, pv, rp, idx_p, cnt_p, top_k, group_size,
                                    scale, m, hs_p, qs_p, out.ctypes.data_as(_f64p), lse.ctypes.data_as(_f64p)),
           "sparse_attn")
    return out[:m], lse[:m], hs_a, qs_a


def dense_attn(q, k, v, B: int, chunk_begin: int, chunk_end: int, scale: float, resident=None, hs=None, qs=None):
    """Dense attention over history chunks [chunk_begin, chunk_end) (full history or SWA window)."""
    n, S, H, d = _kv_shape(k)
    Lq = int(q.shape[0])
    (hs_a, hs_p), (qs_a, qs_p) = _rows(H, Lq, hs, qs)
    m = int(hs_a.shape[0])
    etq, kq, pq = _as_input(q)
    etk, kk, pk = _as_input(k)
    etv, kv, pv = _as_input(v)
    if etk != etv:
        raise ValueError("k and v must share a dtype")
    keep, rp = _u8_or_null(resident)
    out = np.zeros((max(m, 1), d))
    lse = np.zeros(max(m, 1))
    _check(lib().oracle_dense_attn(H, d, S, n, B, Lq, etq, pq, etk, pk, pv, rp, chunk_begin, chunk_end, scale, m,
                                   hs_p, qs_p, out.ctypes.data_as(_f64p), lse.ctypes.data_as(_f64p)), "dense_attn")
    return out[:m], lse[:m], hs_a, qs_a


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (ties to even), returned as float64.
    An 8-bit significand: the frexp mantissa m in [0.5, 1) is rounded to a multiple of
    2^-8 with numpy's half-to-even rounding (normal range; values are not clamped)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.round(m * 256.0) / 256.0, e)


def cmp_cache(k, v, B: int, round_to=None):
    """The compressed history of App. C: one pooled key and value per block of every
    chunk, the plain block mean of Sec. 3.1 / App. B (pool_keys applied to K and to V),
    in block order: [H, n*Bpc, d] each.  round_to="bf16" rounds them to the stored
    dtype (a bf16 cache holds the pooled values in bf16)."""
    kc, vc = pool_keys(k, B), pool_keys(v, B)
    if round_to == "bf16":
        kc, vc = round_bf16(kc), round_bf16(vc)
    elif round_to is not None:
        raise ValueError(f"unknown rounding {round_to!r}")
    return kc, vc


def cmp_attn(q, kc, vc, scale: float, hs=None, qs=None):
    """Compression attention, the CMP branch of Eq. 1: query i of head h attends to the
    N pooled tokens kc[h], vc[h] ([H, N, d]) as one contiguous sequence (plain softmax
    attention over them).  Evaluated as dense attention over a one-chunk history of N
    tokens.  Returns (out [m, d], lse [m], hs, qs); N = 0 gives O = 0 and lse = -inf."""
    kc = np.asarray(kc, dtype=np.float64)
    vc = np.asarray(vc, dtype=np.float64)
    H, N, d = kc.shape
    Lq = int(q.shape[0])
    if N == 0:
        (hs_a, _), (qs_a, _) = _rows(H, Lq, hs, qs)
        m = int(hs_a.shape[0])
        return np.zeros((m, d)), np.full(m, -np.inf), hs_a, qs_a
    k1 = np.ascontiguousarray(kc.transpose(1, 0, 2))[None]   # [1, N, H, d]
    v1 = np.ascontiguousarray(vc.transpose(1, 0, 2))[None]
    return dense_attn(q, k1, v1, N, 0, 1, scale, hs=hs, qs=qs)


def gated_combine(o_cmp, o_slc, o_swa, gate_logits):
    """Eq. 1's fusion of the three branches: o = sum over c in (CMP, SLC, SWA) of
    g^c * Attn_c, each coefficient g^c in [0, 1] a sigmoid of its gate logit (App. B:
    learned per-branch sigmoid gates).  o_*: [Lq, H, d] or None (an absent branch
    contributes nothing); gate_logits: [Lq, H, 3] in the order CMP, SLC, SWA.
    float64 throughout."""
    gl = np.asarray(gate_logits, dtype=np.float64)
    out = None
    for c, o in enumerate((o_cmp, o_slc, o_swa)):
        if o is None:
            continue
        z = np.exp(-np.abs(gl[..., c]))                  # sigmoid without overflow
        g = np.where(gl[..., c] >= 0, 1.0 / (1.0 + z), z / (1.0 + z))
        term = g[..., None] * np.asarray(o, dtype=np.float64)
        out = term if out is None else out + term
    if out is None:
        raise ValueError("no branch given")
    return out


def lru_simulate(requests, slots: int):
    """The hot cache's replacement policy (App. B: least recently used chunks stay on
    the GPU; App. F varies the number of slots), for one head.  `requests` is a
    sequence of collections of chunk ids.  Per request, its distinct chunks are taken
    in ascending id: a resident chunk is a hit and becomes the most recently used;
    then each other chunk takes the lowest free slot, or else the slot of the least
    recently used resident chunk that the request does not name, and becomes the most
    recently used.  A request naming more than `slots` chunks is an error.
    Returns dict(slot_of={chunk: slot} after the last request, hits, misses,
    evictions, per_request=[(hits, misses), ...])."""
    if slots < 1:
        raise ValueError("slots must be >= 1")
    order = []            # resident chunks, least recently used first
    slot_of = {}
    hits = misses = evictions = 0
    per_request = []
    for req in requests:
        want = sorted(set(int(c) for c in req))
        if len(want) > slots:
            raise ValueError(f"a request names {len(want)} chunks, more than {slots} slots")
        h0, m0 = hits, misses
        for c in want:
            if c in slot_of:
                order.remove(c)
                order.append(c)
                hits += 1
        for c in want:
            if c in slot_of:
                continue
            free = sorted(set(range(slots)) - set(slot_of.values()))
            if free:
                s = free[0]
            else:
                victim = next(v for v in order if v not in want)
                s = slot_of.pop(victim)
                order.remove(victim)
                evictions += 1
            slot_of[c] = s
            order.append(c)
            misses += 1
        per_request.append((hits - h0, misses - m0))
    return dict(slot_of=slot_of, hits=hits, misses=misses, evictions=evictions, per_request=per_request)


def union(idx, cnt, n_blocks: int):
    """Eq. 4 unions: returns (per-head |U_h| [H], cross-head |U|)."""
    idx_a, idx_p = _i32(idx)
    cnt_a, cnt_p = _i32(cnt)
    H, R, K = (int(s) for s in idx_a.shape)
    per = np.zeros(H, dtype=np.int32)
    tot = np.zeros(1, dtype=np.int32)
    _check(lib().oracle_union(H, R, K, n_blocks, idx_p, cnt_p, per.ctypes.data_as(_i32p), tot.ctypes.data_as(_i32p)),
           "union")
    return per, int(tot[0])
