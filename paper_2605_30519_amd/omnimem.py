"""Python binding of libomnimem.so (ctypes).  Argument marshalling only: every
step of the computation runs in the HIP kernels behind the C ABI declared in
include/omnimem.h.  PyTorch supplies device memory and the current stream.

The functions carry the C names: omnimem_select, omnimem_sparse_attn,
omnimem_dense_attn, omnimem_union_gather_attn, the compressed-history calls
omnimem_compress_chunk, omnimem_select_compressed and omnimem_cmp_attn, Eq. 1's
gated fusion omnimem_gated_combine, plus the host-side helpers.
"""
from __future__ import annotations

import ctypes
import math
import os
import threading
from dataclasses import dataclass
from typing import Optional

import torch

from . import _build

BF16, F32 = 0, 1
_DTYPES = {torch.bfloat16: BF16, torch.float32: F32}

_lock = threading.Lock()
_lib = None


class OmniMemError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {omnimem_status_string(status)} (status {status})")
        self.status = status


class omnimem_kv_cache_t(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32),
        ("num_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("chunk_tokens", ctypes.c_int32),
        ("num_chunks", ctypes.c_int32),
        ("num_pages", ctypes.c_int64),
        ("k_pages", ctypes.c_void_p),
        ("v_pages", ctypes.c_void_p),
        ("page_table", ctypes.c_void_p),
        ("page_table_head_stride", ctypes.c_int64),
    ]


class omnimem_select_params_t(ctypes.Structure):
    _fields_ = [
        ("top_k", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("window_chunks", ctypes.c_int32),
        ("awe_min_outside_chunks", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("score_mode", ctypes.c_int32),
    ]


SCORE_LOGIT = 0  # the group-mean logit (the default)
SCORE_PROB = 1   # the group mean of each query's softmax probability (compressed history only)


class omnimem_lru_stats_t(ctypes.Structure):
    _fields_ = [
        ("hits", ctypes.c_int64),
        ("misses", ctypes.c_int64),
        ("evictions", ctypes.c_int64),
        ("bytes_reloaded", ctypes.c_int64),
    ]


class omnimem_cmp_cache_t(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32),
        ("num_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("chunk_tokens", ctypes.c_int32),
        ("capacity_chunks", ctypes.c_int32),
        ("k_mean", ctypes.c_void_p),
        ("k_pages", ctypes.c_void_p),
        ("v_pages", ctypes.c_void_p),
        ("page_table", ctypes.c_void_p),
        ("num_pages", ctypes.c_int64),
        ("k_lo", ctypes.c_void_p),
    ]


EXPORTED = [
    "omnimem_blocks_per_chunk",
    "omnimem_awe_active",
    "omnimem_select_workspace_bytes",
    "omnimem_select",
    "omnimem_select_noalloc",
    "omnimem_sparse_attn",
    "omnimem_dense_attn",
    "omnimem_union_workspace_bytes",
    "omnimem_union_gather_attn",
    "omnimem_status_string",
    "omnimem_compress_chunk",
    "omnimem_select_compressed",
    "omnimem_cmp_attn",
    "omnimem_gated_combine",
    "omnimem_selected_chunks",
    "omnimem_lru_create",
    "omnimem_lru_destroy",
    "omnimem_lru_require",
    "omnimem_lru_wait",
    "omnimem_lru_stats",
    "omnimem_lru_slot_of",
    "omnimem_numa_bind",
]


class _Present:
    """Attribute sink for a symbol a partial build does not export (sanitizer tests)."""


def _configure(L, required: bool = True):
    """Declares every exported function's signature on the loaded library L.  With
    required=False, functions L does not export are skipped (a host-only test build)."""
    if not required:
        class _Partial:
            def __init__(self, lib):
                self._lib = lib

            def __getattr__(self, name):
                try:
                    return getattr(self._lib, name)
                except AttributeError:
                    f = _Present()
                    object.__setattr__(self, name, f)
                    return f
        _configure(_Partial(L))
        return L
    i32, i64, vp, f32, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_size_t
    kvp = ctypes.POINTER(omnimem_kv_cache_t)
    pp = ctypes.POINTER(omnimem_select_params_t)
    L.omnimem_blocks_per_chunk.argtypes = [i32, i32]
    L.omnimem_blocks_per_chunk.restype = i32
    L.omnimem_awe_active.argtypes = [i32] * 5
    L.omnimem_awe_active.restype = i32
    L.omnimem_select_workspace_bytes.argtypes = [kvp, i32, pp]
    L.omnimem_select_workspace_bytes.restype = sz
    L.omnimem_select.argtypes = [kvp, vp, i32, pp, vp, vp, vp, ctypes.POINTER(i32), vp, sz, vp]
    L.omnimem_select.restype = i32
    L.omnimem_select_noalloc.argtypes = [kvp, vp, i32, pp, vp, vp, vp, ctypes.POINTER(i32), vp]
    L.omnimem_select_noalloc.restype = i32
    L.omnimem_sparse_attn.argtypes = [kvp, vp, i32, vp, vp, i32, i32, f32, vp, vp, vp]
    L.omnimem_sparse_attn.restype = i32
    L.omnimem_dense_attn.argtypes = [kvp, vp, i32, i32, i32, f32, vp, vp, vp]
    L.omnimem_dense_attn.restype = i32
    L.omnimem_union_workspace_bytes.argtypes = [kvp]
    L.omnimem_union_workspace_bytes.restype = sz
    L.omnimem_union_gather_attn.argtypes = [kvp, vp, i32, vp, vp, i32, i32, f32, vp, vp, vp, vp, sz, vp]
    L.omnimem_union_gather_attn.restype = i32
    L.omnimem_status_string.argtypes = [i32]
    L.omnimem_status_string.restype = ctypes.c_char_p
    ccp = ctypes.POINTER(omnimem_cmp_cache_t)
    L.omnimem_compress_chunk.argtypes = [kvp, i32, ccp, vp]
    L.omnimem_compress_chunk.restype = i32
    L.omnimem_select_compressed.argtypes = [kvp, ccp, vp, i32, pp, vp, vp, vp, ctypes.POINTER(i32), vp, sz, vp]
    L.omnimem_select_compressed.restype = i32
    L.omnimem_cmp_attn.argtypes = [ccp, i32, vp, i32, f32, vp, vp, vp]
    L.omnimem_cmp_attn.restype = i32
    L.omnimem_gated_combine.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]
    L.omnimem_gated_combine.restype = i32
    L.omnimem_lru_create.argtypes = [kvp, i32, vp, vp, i32, vp, ctypes.POINTER(vp)]
    L.omnimem_lru_create.restype = i32
    L.omnimem_lru_destroy.argtypes = [vp]
    L.omnimem_lru_destroy.restype = None
    L.omnimem_lru_require.argtypes = [vp, vp, i32, vp, vp, ctypes.POINTER(i32)]
    L.omnimem_lru_require.restype = i32
    L.omnimem_lru_wait.argtypes = [vp, vp]
    L.omnimem_lru_wait.restype = i32
    L.omnimem_lru_stats.argtypes = [vp, ctypes.POINTER(omnimem_lru_stats_t)]
    L.omnimem_lru_stats.restype = i32
    L.omnimem_lru_slot_of.argtypes = [vp, i32, i32]
    L.omnimem_lru_slot_of.restype = i32
    L.omnimem_selected_chunks.argtypes = [kvp, vp, vp, i32, i32, vp, vp]
    L.omnimem_selected_chunks.restype = i32
    L.omnimem_numa_bind.argtypes = [i32, ctypes.POINTER(i32)]
    L.omnimem_numa_bind.restype = i32
    return L


def lib():
    """The loaded libomnimem.so.  Builds it if it has never been built; there is no
    fallback: without the HIP library nothing in this module runs."""
    global _lib
    with _lock:
        if _lib is None:
            if not _build.is_built():
                _build.build()
            _lib = _configure(ctypes.CDLL(_build.LIB))
    return _lib


def library_path() -> str:
    return os.path.realpath(_build.LIB)


# ----------------------------------------------------------------------- cache

@dataclass
class PagedKVCache:
    """One layer's paged KV cache (device tensors owned by the caller).

    k_pages, v_pages: [num_pages, H, B, d] (bf16 or fp32); page_table: [n, Bpc] int32
    shared by every head, or [H, n, Bpc] with one table per head (the (page, h) slab
    then holds head h's block); negative = block not resident."""
    k_pages: torch.Tensor
    v_pages: torch.Tensor
    page_table: torch.Tensor
    chunk_tokens: int

    @property
    def num_heads(self) -> int:
        return int(self.k_pages.shape[1])

    @property
    def block_size(self) -> int:
        return int(self.k_pages.shape[2])

    @property
    def head_dim(self) -> int:
        return int(self.k_pages.shape[3])

    @property
    def num_chunks(self) -> int:
        return int(self.page_table.shape[-2])

    @property
    def per_head_tables(self) -> bool:
        return self.page_table.dim() == 3

    @property
    def blocks_per_chunk(self) -> int:
        return -(-self.chunk_tokens // self.block_size)

    @property
    def num_blocks(self) -> int:
        return self.num_chunks * self.blocks_per_chunk

    @property
    def dtype(self) -> torch.dtype:
        return self.k_pages.dtype

    def descriptor(self, num_chunks: Optional[int] = None, with_table: bool = True) -> omnimem_kv_cache_t:
        """C descriptor; `num_chunks` < n exposes only the oldest chunks (a shorter history);
        with_table=False passes a NULL page table (selection from pooled keys only)."""
        kp, vp, pt = self.k_pages, self.v_pages, self.page_table
        if kp.dtype not in _DTYPES or vp.dtype != kp.dtype:
            raise TypeError(f"unsupported page dtype {kp.dtype}")
        for t in (kp, vp, pt):
            if not t.is_contiguous():
                raise ValueError("cache tensors must be contiguous")
        if pt.dtype != torch.int32:
            raise TypeError("page_table must be int32")
        if kp.dim() != 4 or vp.shape != kp.shape:
            raise ValueError("k_pages and v_pages must share one [num_pages, H, B, d] shape")
        num_pages, H, B, d = (int(x) for x in kp.shape)
        bpc = -(-self.chunk_tokens // B)
        pt_shape = tuple(pt.shape)
        if not (len(pt_shape) == 2 or (len(pt_shape) == 3 and pt_shape[0] == H)) or pt_shape[-1] != bpc:
            raise ValueError(f"page_table must be [n, {bpc}] or [{H}, n, {bpc}] (blocks per chunk)")
        _on_gpu(kp, v_pages=vp, page_table=pt)
        total = pt_shape[-2]
        n = total if num_chunks is None else int(num_chunks)
        if n > total:
            raise ValueError("num_chunks exceeds the page table")
        return omnimem_kv_cache_t(
            _DTYPES[kp.dtype], H, d, B, self.chunk_tokens, n, num_pages, kp.data_ptr(), vp.data_ptr(),
            pt.data_ptr() if with_table else None, total * bpc if len(pt_shape) == 3 else 0)


def _current_raw_stream():
    """The current device's current stream as a raw handle: torch's own accessor for
    it when this torch has one (it builds no Stream object), else the public API."""
    try:
        return torch._C._cuda_getCurrentRawStream(torch._C._cuda_getDevice())
    except AttributeError:
        return torch.cuda.current_stream().cuda_stream


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(_current_raw_stream())
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(None)


def _check(status: int, what: str):
    if status != 0:
        raise OmniMemError(status, what)


def _default_scale(cache: PagedKVCache, scale):
    return 1.0 / math.sqrt(cache.head_dim) if scale is None else float(scale)


# Argument checks.  The C ABI receives raw pointers, so shapes, dtypes, devices and
# contiguity of tensors can only be checked here; every check runs before anything
# is launched.  Shape and dtype are checked before the device, so that the checks
# themselves can be exercised on a machine without a GPU.

def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _on_gpu(like: torch.Tensor, like_name: str = "the cache", **tensors):
    """Every given tensor (None = absent) lives on the GPU that holds `like`."""
    if like.is_cuda:  # the common case, without building any message
        dev = like.get_device()
        if all(t is None or (t.is_cuda and t.get_device() == dev) for t in tensors.values()):
            return
    _need(like.is_cuda, f"{like_name} must live on a GPU")
    for name, t in tensors.items():
        if t is None:
            continue
        _need(t.is_cuda, f"{name} must be a GPU tensor")
        _need(t.device == like.device, f"{name} must be on {like.device}, not {t.device}")


def _check_tensor(name: str, t, shape, dtype):
    if isinstance(t, torch.Tensor) and t.dtype == dtype and tuple(t.shape) == tuple(shape) and t.is_contiguous():
        return  # the common case, without building any message
    _need(isinstance(t, torch.Tensor), f"{name} must be a tensor")
    _need(tuple(t.shape) == tuple(shape), f"{name} must have shape {tuple(shape)}, not {tuple(t.shape)}")
    _need(t.dtype == dtype, f"{name} must be {dtype}, not {t.dtype}")
    _need(t.is_contiguous(), f"{name} must be contiguous")


def _check_q(cache: "PagedKVCache", q) -> int:
    """q: [lq, H, d] in the cache's dtype, contiguous.  Returns lq."""
    _need(isinstance(q, torch.Tensor) and q.dim() == 3, "q must be a [lq, H, d] tensor")
    lq = int(q.shape[0])
    _check_tensor("q", q, (lq, cache.num_heads, cache.head_dim), cache.dtype)
    return lq


def _check_outputs(q: torch.Tensor, out, lse):
    lq, H, d = (int(s) for s in q.shape)
    if out is not None:
        _check_tensor("out", out, (lq, H, d), q.dtype)
    if lse is not None:
        _check_tensor("lse", lse, (H, lq), torch.float32)


def _check_lists(q: torch.Tensor, idx, cnt, group_size: int) -> int:
    """idx [H, R, K] and cnt [H, R] int32 for R = ceil(lq / group_size).  Returns K."""
    _need(int(group_size) >= 1, "group_size must be >= 1")
    lq, H = int(q.shape[0]), int(q.shape[1])
    R = -(-lq // int(group_size))
    _need(isinstance(idx, torch.Tensor) and idx.dim() == 3, "idx must be an [H, R, K] tensor")
    K = int(idx.shape[-1])
    _need(K >= 1, "idx must hold at least one entry per row")
    _check_tensor("idx", idx, (H, R, K), torch.int32)
    _check_tensor("cnt", cnt, (H, R), torch.int32)
    return K


def _check_workspace(ws, need: int, like: torch.Tensor):
    _need(isinstance(ws, torch.Tensor) and ws.dim() == 1, "workspace must be a 1-D uint8 tensor")
    _check_tensor("workspace", ws, (int(ws.shape[0]),), torch.uint8)
    _need(ws.numel() >= need, f"workspace holds {ws.numel()} bytes, {need} needed")
    _on_gpu(like, workspace=ws)


def _check_selection_out(sel: "Selection", H: int, R: int, K: int):
    _check_tensor("out.idx", sel.idx, (H, R, K), torch.int32)
    _check_tensor("out.cnt", sel.cnt, (H, R), torch.int32)
    if sel.score is not None:
        _check_tensor("out.score", sel.score, (H, R, K), torch.float32)


# --------------------------------------------------------------- host helpers

def omnimem_blocks_per_chunk(chunk_tokens: int, block_size: int) -> int:
    return int(lib().omnimem_blocks_per_chunk(chunk_tokens, block_size))


def omnimem_awe_active(num_chunks: int, window_chunks: int, awe_min_outside_chunks: int, top_k: int,
                       blocks_per_chunk: int) -> int:
    return int(lib().omnimem_awe_active(num_chunks, window_chunks, awe_min_outside_chunks, top_k, blocks_per_chunk))


def omnimem_status_string(status: int) -> str:
    return lib().omnimem_status_string(status).decode()


def select_params(top_k, group_size, window_chunks, awe_min_outside_chunks, scale,
                  score_mode: int = SCORE_LOGIT) -> omnimem_select_params_t:
    return omnimem_select_params_t(top_k, group_size, window_chunks, awe_min_outside_chunks, scale, score_mode)


def omnimem_select_workspace_bytes(cache: PagedKVCache, lq: int, params: omnimem_select_params_t,
                                   num_chunks: Optional[int] = None) -> int:
    d = cache.descriptor(num_chunks)
    return int(lib().omnimem_select_workspace_bytes(ctypes.byref(d), lq, ctypes.byref(params)))


def omnimem_union_workspace_bytes(cache: PagedKVCache, num_chunks: Optional[int] = None) -> int:
    d = cache.descriptor(num_chunks)
    return int(lib().omnimem_union_workspace_bytes(ctypes.byref(d)))


# ------------------------------------------------------------------ the calls

@dataclass
class Selection:
    idx: torch.Tensor      # [H, R, K] int32, ascending, -1 padded
    cnt: torch.Tensor      # [H, R] int32
    score: Optional[torch.Tensor]  # [H, R, K] float32
    awe_active: int


def workspace_tensor(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 256-byte (or better) aligned blocks
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def omnimem_select(cache: PagedKVCache, q: torch.Tensor, top_k: int, group_size: int, window_chunks: int,
                   awe_min_outside_chunks: int, scale: Optional[float] = None, *, num_chunks: Optional[int] = None,
                   want_score: bool = True, workspace: Optional[torch.Tensor] = None,
                   out: Optional[Selection] = None, stream=None) -> Selection:
    lq = _check_q(cache, q)
    H = cache.num_heads
    _need(int(top_k) >= 1 and int(group_size) >= 1, "top_k and group_size must be >= 1")
    params = select_params(top_k, group_size, window_chunks, awe_min_outside_chunks, _default_scale(cache, scale))
    R = -(-lq // group_size)
    if out is not None:
        _check_selection_out(out, H, R, int(top_k))
    desc = cache.descriptor(num_chunks)
    dev = q.device
    if out is None:
        out = Selection(torch.empty((H, R, top_k), dtype=torch.int32, device=dev),
                        torch.empty((H, R), dtype=torch.int32, device=dev),
                        torch.empty((H, R, top_k), dtype=torch.float32, device=dev) if want_score else None, 0)
    _check_selection_out(out, H, R, int(top_k))
    _on_gpu(cache.k_pages, q=q, idx=out.idx, cnt=out.cnt, score=out.score)
    need = int(lib().omnimem_select_workspace_bytes(ctypes.byref(desc), lq, ctypes.byref(params)))
    if workspace is None:
        workspace = workspace_tensor(need, dev)
    _check_workspace(workspace, need, q)
    awe = ctypes.c_int32(0)
    st = lib().omnimem_select(ctypes.byref(desc), _ptr(q), lq, ctypes.byref(params), _ptr(out.idx), _ptr(out.cnt),
                              _ptr(out.score), ctypes.byref(awe), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "omnimem_select")
    out.awe_active = int(awe.value)
    return out


NOALLOC_SCRATCH_BYTES = 8 << 20   # OMNIMEM_NOALLOC_SCRATCH_BYTES


def omnimem_select_noalloc(cache: PagedKVCache, q: torch.Tensor, top_k: int, group_size: int, window_chunks: int,
                           awe_min_outside_chunks: int, scale: Optional[float] = None, *, out: Selection,
                           num_chunks: Optional[int] = None, stream=None) -> Selection:
    """omnimem_select with the library's static per-GPU scratch instead of a
    workspace: nothing is allocated, so `out` (idx, cnt and optionally score) must be
    given.  Runs on the current device; calls that overlap on one GPU race."""
    lq = _check_q(cache, q)
    H = cache.num_heads
    _need(int(top_k) >= 1 and int(group_size) >= 1, "top_k and group_size must be >= 1")
    _need(out is not None, "out must be given: this call allocates nothing")
    R = -(-lq // group_size)
    _check_selection_out(out, H, R, int(top_k))
    params = select_params(top_k, group_size, window_chunks, awe_min_outside_chunks, _default_scale(cache, scale))
    desc = cache.descriptor(num_chunks)
    _on_gpu(cache.k_pages, q=q, idx=out.idx, cnt=out.cnt, score=out.score)
    awe = ctypes.c_int32(0)
    st = lib().omnimem_select_noalloc(ctypes.byref(desc), _ptr(q), lq, ctypes.byref(params), _ptr(out.idx),
                                      _ptr(out.cnt), _ptr(out.score), ctypes.byref(awe), _stream(stream))
    _check(st, "omnimem_select_noalloc")
    out.awe_active = int(awe.value)
    return out


def omnimem_sparse_attn(cache: PagedKVCache, q: torch.Tensor, idx: torch.Tensor, cnt: torch.Tensor,
                        group_size: int, scale: Optional[float] = None, *, num_chunks: Optional[int] = None,
                        out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                        stream=None):
    lq = _check_q(cache, q)
    H = cache.num_heads
    top_k = _check_lists(q, idx, cnt, group_size)
    _check_outputs(q, out, lse)
    desc = cache.descriptor(num_chunks)
    _on_gpu(cache.k_pages, q=q, idx=idx, cnt=cnt, out=out, lse=lse)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((H, lq), dtype=torch.float32, device=q.device)
    st = lib().omnimem_sparse_attn(ctypes.byref(desc), _ptr(q), lq, _ptr(idx), _ptr(cnt), top_k,
                                   group_size, _default_scale(cache, scale), _ptr(out), _ptr(lse), _stream(stream))
    _check(st, "omnimem_sparse_attn")
    return out, lse


def omnimem_dense_attn(cache: PagedKVCache, q: torch.Tensor, chunk_begin: int, chunk_end: int,
                       scale: Optional[float] = None, *, num_chunks: Optional[int] = None,
                       out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                       stream=None):
    lq = _check_q(cache, q)
    H = cache.num_heads
    _check_outputs(q, out, lse)
    desc = cache.descriptor(num_chunks)
    _on_gpu(cache.k_pages, q=q, out=out, lse=lse)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((H, lq), dtype=torch.float32, device=q.device)
    st = lib().omnimem_dense_attn(ctypes.byref(desc), _ptr(q), lq, chunk_begin, chunk_end,
                                  _default_scale(cache, scale), _ptr(out), _ptr(lse), _stream(stream))
    _check(st, "omnimem_dense_attn")
    return out, lse


def omnimem_union_gather_attn(cache: PagedKVCache, q: torch.Tensor, idx: torch.Tensor, cnt: torch.Tensor,
                              group_size: int, scale: Optional[float] = None, *, num_chunks: Optional[int] = None,
                              workspace: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                              lse: Optional[torch.Tensor] = None, stream=None):
    lq = _check_q(cache, q)
    H = cache.num_heads
    top_k = _check_lists(q, idx, cnt, group_size)
    _check_outputs(q, out, lse)
    desc = cache.descriptor(num_chunks)
    _on_gpu(cache.k_pages, q=q, idx=idx, cnt=cnt, out=out, lse=lse)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((H, lq), dtype=torch.float32, device=q.device)
    union_blocks = torch.zeros(1, dtype=torch.int32, device=q.device)
    need = int(lib().omnimem_union_workspace_bytes(ctypes.byref(desc)))
    if workspace is None:
        workspace = workspace_tensor(need, q.device)
    _check_workspace(workspace, need, q)
    st = lib().omnimem_union_gather_attn(ctypes.byref(desc), _ptr(q), lq, _ptr(idx), _ptr(cnt), top_k,
                                         group_size, _default_scale(cache, scale), _ptr(out), _ptr(lse),
                                         _ptr(union_blocks), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "omnimem_union_gather_attn")
    return out, lse, union_blocks


# ------------------------------------------------------- compressed history

CMP_PAGE_TOKENS = 64


@dataclass
class CompressedCache:
    """One layer's compressed history (device tensors): k_mean [H, cap*Bpc, d] fp32,
    k_pages / v_pages [pages, H, 64, d] in the full cache's dtype, page_table [pages],
    and for bf16 caches optionally k_lo [pages, H, 64, d] bf16, the pooled keys'
    rounding residual (the probability-averaged scores then skip splitting k_mean)."""
    k_mean: torch.Tensor
    k_pages: torch.Tensor
    v_pages: torch.Tensor
    page_table: torch.Tensor
    block_size: int
    chunk_tokens: int
    capacity_chunks: int
    k_lo: Optional[torch.Tensor] = None

    @classmethod
    def allocate(cls, cache: PagedKVCache, capacity_chunks: int) -> "CompressedCache":
        H, d, dev = cache.num_heads, cache.head_dim, cache.k_pages.device
        tokens = capacity_chunks * cache.blocks_per_chunk
        pages = max(1, -(-tokens // CMP_PAGE_TOKENS))
        k_lo = None
        if cache.dtype == torch.bfloat16:
            k_lo = torch.zeros((pages, H, CMP_PAGE_TOKENS, d), dtype=torch.bfloat16, device=dev)
        return cls(torch.zeros((H, max(tokens, 1), d), dtype=torch.float32, device=dev),
                   torch.zeros((pages, H, CMP_PAGE_TOKENS, d), dtype=cache.dtype, device=dev),
                   torch.zeros((pages, H, CMP_PAGE_TOKENS, d), dtype=cache.dtype, device=dev),
                   torch.zeros(pages, dtype=torch.int32, device=dev),
                   cache.block_size, cache.chunk_tokens, int(capacity_chunks), k_lo)

    def check_against(self, cache: PagedKVCache):
        """The pooled tensors must match the full cache's heads, dim, dtype and GPU."""
        H, d = cache.num_heads, cache.head_dim
        tokens = max(self.capacity_chunks * cache.blocks_per_chunk, 1)
        pages = max(1, -(-tokens // CMP_PAGE_TOKENS))
        _need(self.block_size == cache.block_size and self.chunk_tokens == cache.chunk_tokens,
              "compressed cache geometry differs from the full cache")
        _need(self.k_mean.dim() == 3, "k_mean must be [H, capacity*Bpc, d]")
        _check_tensor("k_mean", self.k_mean, (H, int(self.k_mean.shape[1]), d), torch.float32)
        _need(int(self.k_mean.shape[1]) >= tokens, "k_mean holds fewer pooled tokens than the capacity")
        for name, t in (("cmp k_pages", self.k_pages), ("cmp v_pages", self.v_pages)):
            _need(t.dim() == 4, f"{name} must be [pages, H, {CMP_PAGE_TOKENS}, d]")
            _check_tensor(name, t, (int(t.shape[0]), H, CMP_PAGE_TOKENS, d), cache.dtype)
            _need(int(t.shape[0]) >= pages, f"{name} holds fewer pages than the capacity needs")
        _check_tensor("cmp page_table", self.page_table, (int(self.page_table.shape[0]),), torch.int32)
        if self.k_lo is not None:
            _need(cache.dtype == torch.bfloat16, "k_lo exists for bf16 caches only")
            _check_tensor("cmp k_lo", self.k_lo, tuple(int(x) for x in self.k_pages.shape), torch.bfloat16)
        _on_gpu(cache.k_pages, k_mean=self.k_mean, cmp_k_pages=self.k_pages, cmp_v_pages=self.v_pages,
                cmp_page_table=self.page_table, cmp_k_lo=self.k_lo)

    def descriptor(self) -> omnimem_cmp_cache_t:
        return omnimem_cmp_cache_t(
            _DTYPES[self.k_pages.dtype], int(self.k_pages.shape[1]), int(self.k_pages.shape[3]), self.block_size,
            self.chunk_tokens, self.capacity_chunks, self.k_mean.data_ptr(), self.k_pages.data_ptr(),
            self.v_pages.data_ptr(), self.page_table.data_ptr(), int(self.k_pages.shape[0]),
            self.k_lo.data_ptr() if self.k_lo is not None else None)


def omnimem_compress_chunk(cache: PagedKVCache, chunk: int, cc: CompressedCache, *,
                           num_chunks: Optional[int] = None, stream=None) -> None:
    cc.check_against(cache)
    desc = cache.descriptor(num_chunks)
    cdesc = cc.descriptor()
    _check(lib().omnimem_compress_chunk(ctypes.byref(desc), int(chunk), ctypes.byref(cdesc), _stream(stream)),
           "omnimem_compress_chunk")


def omnimem_select_compressed(cache: PagedKVCache, cc: CompressedCache, q: torch.Tensor, top_k: int, group_size: int,
                              window_chunks: int, awe_min_outside_chunks: int, scale: Optional[float] = None, *,
                              num_chunks: Optional[int] = None, want_score: bool = True,
                              workspace: Optional[torch.Tensor] = None, out: Optional[Selection] = None,
                              all_candidates: bool = False, score_mode: int = SCORE_LOGIT,
                              stream=None) -> Selection:
    """all_candidates=True ignores residency (NULL page table): every block of the
    history is a candidate, as when an LRU hot cache reloads what is selected.
    score_mode=SCORE_PROB ranks by group-mean softmax probabilities over the pooled
    keys instead of group-mean logits."""
    lq = _check_q(cache, q)
    H = cache.num_heads
    _need(int(top_k) >= 1 and int(group_size) >= 1, "top_k and group_size must be >= 1")
    cc.check_against(cache)
    params = select_params(top_k, group_size, window_chunks, awe_min_outside_chunks, _default_scale(cache, scale),
                           score_mode)
    R = -(-lq // group_size)
    if out is not None:
        _check_selection_out(out, H, R, int(top_k))
    desc = cache.descriptor(num_chunks, with_table=not all_candidates)
    cdesc = cc.descriptor()
    dev = q.device
    if out is None:
        out = Selection(torch.empty((H, R, top_k), dtype=torch.int32, device=dev),
                        torch.empty((H, R), dtype=torch.int32, device=dev),
                        torch.empty((H, R, top_k), dtype=torch.float32, device=dev) if want_score else None, 0)
    _check_selection_out(out, H, R, int(top_k))
    _on_gpu(cache.k_pages, q=q, idx=out.idx, cnt=out.cnt, score=out.score)
    need = int(lib().omnimem_select_workspace_bytes(ctypes.byref(desc), lq, ctypes.byref(params)))
    if workspace is None:
        workspace = workspace_tensor(need, dev)
    _check_workspace(workspace, need, q)
    awe = ctypes.c_int32(0)
    st = lib().omnimem_select_compressed(ctypes.byref(desc), ctypes.byref(cdesc), _ptr(q), lq, ctypes.byref(params),
                                         _ptr(out.idx), _ptr(out.cnt), _ptr(out.score), ctypes.byref(awe),
                                         _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "omnimem_select_compressed")
    out.awe_active = int(awe.value)
    return out


def omnimem_cmp_attn(cc: CompressedCache, n_chunks: int, q: torch.Tensor, scale: Optional[float] = None, *,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                     stream=None):
    H, d = int(cc.k_pages.shape[1]), int(cc.k_pages.shape[3])
    _need(isinstance(q, torch.Tensor) and q.dim() == 3, "q must be a [lq, H, d] tensor")
    lq = int(q.shape[0])
    _check_tensor("q", q, (lq, H, d), cc.k_pages.dtype)
    _check_outputs(q, out, lse)
    _on_gpu(cc.k_pages, "the compressed cache", q=q, out=out, lse=lse, v_pages=cc.v_pages, page_table=cc.page_table)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((H, lq), dtype=torch.float32, device=q.device)
    sc = 1.0 / math.sqrt(d) if scale is None else float(scale)
    cdesc = cc.descriptor()
    st = lib().omnimem_cmp_attn(ctypes.byref(cdesc), int(n_chunks), _ptr(q), lq, sc, _ptr(out), _ptr(lse),
                                _stream(stream))
    _check(st, "omnimem_cmp_attn")
    return out, lse


def omnimem_gated_combine(o_cmp: Optional[torch.Tensor], o_slc: Optional[torch.Tensor],
                          o_swa: Optional[torch.Tensor], gate_logits: torch.Tensor, *,
                          out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Eq. 1: out = sum_c sigmoid(gate_logits[..., c]) * o_c over the given branches
    (CMP, SLC, SWA); gate_logits [lq, H, 3] float32."""
    ref = next(o for o in (o_cmp, o_slc, o_swa) if o is not None)
    lq, H, d = (int(s) for s in ref.shape)
    for o in (o_cmp, o_slc, o_swa):
        if o is not None and (o.shape != ref.shape or o.dtype != ref.dtype or not o.is_contiguous()):
            raise ValueError("branch outputs must share shape, dtype and be contiguous")
    if gate_logits.dtype != torch.float32 or tuple(gate_logits.shape) != (lq, H, 3) or not gate_logits.is_contiguous():
        raise ValueError("gate_logits must be a contiguous float32 [lq, H, 3] tensor")
    if out is not None:
        _check_tensor("out", out, (lq, H, d), ref.dtype)
    _on_gpu(ref, "the branch outputs", o_cmp=o_cmp, o_slc=o_slc, o_swa=o_swa, gate_logits=gate_logits, out=out)
    if out is None:
        out = torch.empty_like(ref)
    st = lib().omnimem_gated_combine(_DTYPES[ref.dtype], lq, H, d, _ptr(o_cmp), _ptr(o_slc), _ptr(o_swa),
                                     _ptr(gate_logits), _ptr(out), _stream(stream))
    _check(st, "omnimem_gated_combine")
    return out


# ------------------------------------------------------------ LRU hot cache

def omnimem_selected_chunks(cache: PagedKVCache, sel_idx: torch.Tensor, sel_cnt: torch.Tensor, *,
                            num_chunks: Optional[int] = None, out: Optional[torch.Tensor] = None,
                            stream=None) -> torch.Tensor:
    """Alg. 1 Step 1's chunk decode on the device: [H, n] uint8, 1 where some group of
    head h selected a block of chunk c."""
    _need(isinstance(sel_idx, torch.Tensor) and sel_idx.dim() == 3, "idx must be an [H, R, K] tensor")
    H, R, K = (int(s) for s in sel_idx.shape)
    _need(H == cache.num_heads, f"idx must have {cache.num_heads} heads")
    _check_tensor("idx", sel_idx, (H, R, K), torch.int32)
    _check_tensor("cnt", sel_cnt, (H, R), torch.int32)
    n = cache.num_chunks if num_chunks is None else int(num_chunks)
    if out is not None:
        _check_tensor("out", out, (H, n), torch.uint8)
    desc = cache.descriptor(num_chunks)
    _on_gpu(cache.k_pages, idx=sel_idx, cnt=sel_cnt, out=out)
    if out is None:
        out = torch.empty((H, n), dtype=torch.uint8, device=sel_idx.device)
    _check(lib().omnimem_selected_chunks(ctypes.byref(desc), _ptr(sel_idx), _ptr(sel_cnt), R, K, _ptr(out),
                                         _stream(stream)), "omnimem_selected_chunks")
    return out


def omnimem_numa_bind(device: int = 0) -> int:
    """Binds the calling thread to the NUMA node of GPU `device` (affinity and memory
    policy); returns the node, or -1 when there is none to bind."""
    node = ctypes.c_int32(-1)
    _check(lib().omnimem_numa_bind(int(device), ctypes.byref(node)), "omnimem_numa_bind")
    return int(node.value)


class LruOffload:
    """GPU hot cache of full-resolution history chunks with a per-(head, chunk) LRU
    (the library's host runtime).  `gpu` is the GPU pool as a PagedKVCache with
    per-head tables: k_pages / v_pages of at least slots*Bpc pages, page_table
    [H, n, Bpc] (written by the runtime only).  k_host / v_host: pinned CPU tensors
    [host_chunks*Bpc, H, B, d], chunk c in pages [c*Bpc, (c+1)*Bpc)."""

    def __init__(self, gpu: PagedKVCache, slots: int, k_host: torch.Tensor, v_host: torch.Tensor, stream=None):
        _need(gpu.per_head_tables, "the GPU pool needs per-head page tables [H, n, Bpc]")
        for t in (k_host, v_host):
            if t.device.type != "cpu" or not t.is_pinned() or not t.is_contiguous() or t.dtype != gpu.dtype:
                raise ValueError("host pools must be contiguous pinned CPU tensors of the cache dtype")
            if tuple(t.shape[1:]) != tuple(gpu.k_pages.shape[1:]) or t.shape[0] % gpu.blocks_per_chunk:
                raise ValueError("host pools must hold whole chunks in the cache's page layout")
        self.gpu, self.k_host, self.v_host = gpu, k_host, v_host   # kept alive with the state
        self.slots = int(slots)
        self.host_chunks = int(k_host.shape[0]) // gpu.blocks_per_chunk
        desc = gpu.descriptor()
        h = ctypes.c_void_p()
        _check(lib().omnimem_lru_create(ctypes.byref(desc), self.slots, k_host.data_ptr(), v_host.data_ptr(),
                                        self.host_chunks, _stream(stream), ctypes.byref(h)), "omnimem_lru_create")
        self._h = h

    def require(self, needed, compute_stream=None, copy_stream=None) -> int:
        """needed: [H, n] host uint8 array or tensor (1 = make resident).  Reloads run on
        copy_stream (default: the compute stream) after the work already enqueued on
        compute_stream (default: the current stream)."""
        if isinstance(needed, torch.Tensor):
            needed = needed.detach()
            _need(needed.device.type == "cpu", "needed must be a host tensor (copy it from the GPU first)")
            arr = needed.to(torch.uint8).contiguous().numpy()
        else:
            import numpy as np
            arr = np.ascontiguousarray(np.asarray(needed, dtype=np.uint8))
        _need(arr.ndim == 2 and arr.shape[0] == self.gpu.num_heads, f"needed must be [{self.gpu.num_heads}, n]")
        cs = _stream(compute_stream)
        xs = cs if copy_stream is None else _stream(copy_stream)
        got = ctypes.c_int32(0)
        _check(lib().omnimem_lru_require(self._h, arr.ctypes.data_as(ctypes.c_void_p), int(arr.shape[1]), cs, xs,
                                         ctypes.byref(got)), "omnimem_lru_require")
        return int(got.value)

    def wait(self, stream=None):
        """Orders `stream` (default: the current stream) after the last reloads."""
        _check(lib().omnimem_lru_wait(self._h, _stream(stream)), "omnimem_lru_wait")

    def stats(self) -> dict:
        st = omnimem_lru_stats_t()
        _check(lib().omnimem_lru_stats(self._h, ctypes.byref(st)), "omnimem_lru_stats")
        return {"hits": st.hits, "misses": st.misses, "evictions": st.evictions, "bytes_reloaded": st.bytes_reloaded}

    def slot_of(self, head: int, chunk: int) -> int:
        return int(lib().omnimem_lru_slot_of(self._h, int(head), int(chunk)))

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().omnimem_lru_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
