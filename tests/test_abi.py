"""The C ABI without a GPU: the library loads, exports every symbol that
include/omnimem.h declares, and rejects invalid arguments on the host before
anything is launched (so none of these calls reaches the HIP runtime)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT
from paper_2605_30519_amd import omnimem as om

HEADER = os.path.join(ROOT, "include", "omnimem.h")
FAKE = 0x10000  # aligned, never dereferenced: every call below fails validation first


def abi():
    """The library the validation cases run against: libomnimem.so here; the
    sanitizer test swaps in a host-only build of the same checks."""
    return om.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(omnimem_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = om.lib()
    names = declared_functions()
    assert set(names) == set(om.EXPORTED), names
    for name in names:
        assert hasattr(L, name), name


def test_only_the_abi_is_exported():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", om.library_path()], capture_output=True, text=True).stdout
    exported = sorted({line.split()[-1] for line in out.splitlines() if " T " in line})
    assert [n for n in exported if n.startswith("omnimem_")] == declared_functions()
    assert not [n for n in exported if "omnimem" in n and not n.startswith("omnimem_")]


def test_host_helpers():
    L = om.lib()
    assert L.omnimem_blocks_per_chunk(4680, 64) == 74
    assert L.omnimem_blocks_per_chunk(4680, 128) == 37
    assert L.omnimem_blocks_per_chunk(0, 64) == -1
    # tiny fp32 workload: exclusion from a 4-chunk history on
    assert [L.omnimem_awe_active(n, 1, 3, 4, 4) for n in range(9)] == [0, 0, 0, 0, 1, 1, 1, 1, 1]
    assert L.omnimem_awe_active(10, 1, 0, 36, 4) == 1 and L.omnimem_awe_active(10, 1, 0, 37, 4) == 0
    assert L.omnimem_awe_active(-1, 1, 3, 4, 4) == -1
    assert L.omnimem_status_string(0) == b"ok"
    assert L.omnimem_status_string(-3) == b"workspace too small"
    assert b"static" in L.omnimem_status_string(-5)
    assert L.omnimem_status_string(7) == b"unknown status"


def test_awe_matches_oracle_truth_table():
    import oracle
    L = om.lib()
    for n in range(0, 9):
        for E in range(0, 4):
            for T in range(0, 5):
                for K in (1, 4, 9, 40):
                    for Bpc in (1, 4, 74):
                        assert L.omnimem_awe_active(n, E, T, K, Bpc) == int(oracle.awe_active(n, E, T, K, Bpc))


def cache(**kw):
    d = dict(dtype=0, num_heads=2, head_dim=64, block_size=64, chunk_tokens=256, num_chunks=3, num_pages=12,
             k_pages=FAKE, v_pages=FAKE, page_table=FAKE)
    d.update(kw)
    return om.omnimem_kv_cache_t(**d)


def params(**kw):
    d = dict(top_k=4, group_size=256, window_chunks=1, awe_min_outside_chunks=3, scale=0.125)
    d.update(kw)
    return om.omnimem_select_params_t(**d)


EINVAL, EUNSUP, EWS = -1, -2, -3

CACHE_CASES = [
    (dict(dtype=7), EUNSUP),
    (dict(head_dim=96), EUNSUP),
    (dict(block_size=32), EUNSUP),
    (dict(num_heads=0), EINVAL),
    (dict(chunk_tokens=0), EINVAL),
    (dict(num_chunks=-1), EINVAL),
    (dict(num_pages=-1), EINVAL),
    (dict(page_table=0), EINVAL),
    (dict(k_pages=0), EINVAL),
    (dict(k_pages=FAKE + 8), EINVAL),
    (dict(page_table_head_stride=-1), EINVAL),
    (dict(page_table_head_stride=11), EINVAL),     # per-head tables hold all n*Bpc = 12 blocks
    (dict(page_table=FAKE + 2), EINVAL),
]


@pytest.mark.parametrize("kw,want", CACHE_CASES)
def test_cache_validation(kw, want):
    L = abi()
    c = cache(**kw)
    st = L.omnimem_sparse_attn(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 256, 0.125, FAKE, None, None)
    assert st == want
    st = L.omnimem_dense_attn(ctypes.byref(c), FAKE, 256, 0, 1, 0.125, FAKE, None, None)
    assert st == want


def test_select_validation():
    L = abi()
    c = cache()
    ws = L.omnimem_select_workspace_bytes(ctypes.byref(c), 256, ctypes.byref(params()))
    assert ws > 0 and ws % 256 == 0
    assert L.omnimem_select_workspace_bytes(None, 256, ctypes.byref(params())) == 0
    assert L.omnimem_select_workspace_bytes(ctypes.byref(c), 256, ctypes.byref(params(top_k=0))) == 0

    def call(p=params(), lq=256, q=FAKE, idx=FAKE, cnt=FAKE, work=FAKE, nbytes=ws):
        return L.omnimem_select(ctypes.byref(c), q, lq, ctypes.byref(p), idx, cnt, None, None, work, nbytes, None)

    assert call(p=params(top_k=0)) == EINVAL
    assert call(p=params(group_size=0)) == EINVAL
    assert call(p=params(window_chunks=-1)) == EINVAL
    assert call(p=params(awe_min_outside_chunks=-2)) == EINVAL
    assert call(p=params(scale=0.0)) == EINVAL
    assert call(p=params(scale=float("nan"))) == EINVAL
    assert call(lq=-1) == EINVAL
    assert call(q=0) == EINVAL
    assert call(q=FAKE + 2) == EINVAL
    assert call(idx=0) == EINVAL
    assert call(cnt=0) == EINVAL
    assert call(work=0) == EINVAL
    assert call(work=FAKE + 16) == EINVAL           # workspace must be 256-byte aligned
    assert call(nbytes=ws - 1) == EWS
    # lq = 0 is a no-op that still reports the exclusion state
    awe = ctypes.c_int32(-5)
    st = L.omnimem_select(ctypes.byref(c), None, 0, ctypes.byref(params()), None, None, None, ctypes.byref(awe), None,
                          0, None)
    assert st == 0 and awe.value == 0            # 3 chunks, 2 outside the window < 3
    c4 = cache(num_chunks=5)
    st = L.omnimem_select(ctypes.byref(c4), None, 0, ctypes.byref(params()), None, None, None, ctypes.byref(awe), None,
                          0, None)
    assert st == 0 and awe.value == 1


def cmp_cache(**kw):
    d = dict(dtype=0, num_heads=2, head_dim=64, block_size=64, chunk_tokens=256, capacity_chunks=3,
             k_mean=FAKE, k_pages=FAKE, v_pages=FAKE, page_table=FAKE, num_pages=1, k_lo=None)
    d.update(kw)
    return om.omnimem_cmp_cache_t(**d)


def test_compressed_cache_validation():
    """The compressed cache's checks, k_lo (the pooled keys' residual pages) included:
    it may be absent, exists for bf16 caches only and must be 16-byte aligned."""
    L = abi()

    def compress(cc, kv=None):
        kv = kv or cache()
        return L.omnimem_compress_chunk(ctypes.byref(kv), 0, ctypes.byref(cc), None)

    def select(cc, kv=None):
        kv = kv or cache()
        p = params(score_mode=1)
        return L.omnimem_select_compressed(ctypes.byref(kv), ctypes.byref(cc), FAKE, 256, ctypes.byref(p), FAKE,
                                           FAKE, None, None, FAKE, 1 << 20, None)

    assert select(cmp_cache(capacity_chunks=2)) == EINVAL        # fewer chunks than the history
    assert compress(cmp_cache(capacity_chunks=0)) == EINVAL      # chunk 0 beyond the capacity
    for call in (compress, select):
        # every case is refused before anything is launched (the pointers are fake)
        assert call(cmp_cache(num_heads=3)) == EINVAL            # geometry differs from the full cache
        assert call(cmp_cache(num_pages=0)) == EINVAL            # 12 pooled tokens need one page
        assert call(cmp_cache(k_mean=FAKE + 4)) == EINVAL
        assert call(cmp_cache(k_lo=FAKE + 8)) == EINVAL          # misaligned residual pages
        assert call(cmp_cache(dtype=1, k_lo=FAKE), cache(dtype=1)) == EINVAL  # fp32 caches keep no residual


def test_attention_validation():
    L = abi()
    c = cache()
    sp = L.omnimem_sparse_attn
    assert sp(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 0, 256, 0.125, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 0, 0.125, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 256, -1.0, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE, 256, 0, FAKE, 4, 256, 0.125, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE, 256, FAKE, 0, 4, 256, 0.125, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 256, 0.125, 0, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE + 4, 256, FAKE, FAKE, 4, 256, 0.125, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), FAKE, -3, FAKE, FAKE, 4, 256, 0.125, FAKE, None, None) == EINVAL
    assert sp(ctypes.byref(c), None, 0, None, None, 4, 256, 0.125, None, None, None) == 0   # empty: no-op
    dn = L.omnimem_dense_attn
    assert dn(ctypes.byref(c), FAKE, 256, 2, 1, 0.125, FAKE, None, None) == EINVAL
    assert dn(ctypes.byref(c), FAKE, 256, 0, 4, 0.125, FAKE, None, None) == EINVAL
    assert dn(ctypes.byref(c), FAKE, 256, -1, 1, 0.125, FAKE, None, None) == EINVAL
    ug = L.omnimem_union_gather_attn
    uws = L.omnimem_union_workspace_bytes(ctypes.byref(c))
    # 12 blocks x 2 heads x (64 x 64 bf16) x (K + V) plus two int32 tables
    assert uws >= 12 * 2 * 64 * 64 * 2 * 2
    assert ug(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 256, 0.125, FAKE, None, FAKE, FAKE, uws - 1, None) == EWS
    assert ug(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 256, 0.125, FAKE, None, 0, FAKE, uws, None) == EINVAL


def test_select_noalloc_validation():
    """The allocation-free selection shares omnimem_select's checks and refuses a
    problem larger than its static scratch before touching the device."""
    L = abi()
    c = cache()

    def call(kv=c, p=params(), lq=256, q=FAKE, idx=FAKE, cnt=FAKE):
        return L.omnimem_select_noalloc(ctypes.byref(kv), q, lq, ctypes.byref(p), idx, cnt, None, None, None)

    assert call(p=params(top_k=0)) == EINVAL
    assert call(p=params(score_mode=1)) == EINVAL
    assert call(q=0) == EINVAL and call(idx=0) == EINVAL and call(cnt=0) == EINVAL
    assert call(q=FAKE + 2) == EINVAL
    assert call(kv=cache(head_dim=96)) == EUNSUP
    # the paper's small groups (G = 15) on a 20-chunk 1.3B layer need about 33 MB
    big = cache(num_heads=12, head_dim=128, block_size=64, chunk_tokens=4680, num_chunks=20, num_pages=1480)
    need = L.omnimem_select_workspace_bytes(ctypes.byref(big), 4680, ctypes.byref(params(top_k=4, group_size=15)))
    assert need > om.NOALLOC_SCRATCH_BYTES
    assert call(kv=big, lq=4680, p=params(top_k=4, group_size=15)) == -5
    awe = ctypes.c_int32(-5)
    assert L.omnimem_select_noalloc(ctypes.byref(c), None, 0, ctypes.byref(params()), None, None, None,
                                    ctypes.byref(awe), None) == 0 and awe.value == 0


def test_per_head_tables_and_chunk_decode_validation():
    """Per-head page tables are accepted where they are supported and refused by the
    union-gather comparator; the chunk decode checks its lists and mask."""
    L = abi()
    c = cache(page_table_head_stride=12)
    assert L.omnimem_sparse_attn(ctypes.byref(c), None, 0, None, None, 4, 256, 0.125, None, None, None) == 0
    uws = L.omnimem_union_workspace_bytes(ctypes.byref(c))
    assert L.omnimem_union_gather_attn(ctypes.byref(c), FAKE, 256, FAKE, FAKE, 4, 256, 0.125, FAKE, None, FAKE, FAKE,
                                       uws, None) == EUNSUP
    sc = L.omnimem_selected_chunks
    assert sc(ctypes.byref(c), FAKE, FAKE, 1, 0, FAKE, None) == EINVAL          # top_k < 1
    assert sc(ctypes.byref(c), FAKE, FAKE, -1, 4, FAKE, None) == EINVAL         # groups < 0
    assert sc(ctypes.byref(c), 0, FAKE, 1, 4, FAKE, None) == EINVAL             # no idx
    assert sc(ctypes.byref(c), FAKE, FAKE + 2, 1, 4, FAKE, None) == EINVAL      # misaligned cnt
    assert sc(ctypes.byref(c), FAKE, FAKE, 1, 4, 0, None) == EINVAL             # no mask
    assert sc(ctypes.byref(cache(num_chunks=0)), FAKE, FAKE, 1, 4, 0, None) == 0  # empty history: nothing to do
    assert sc(ctypes.byref(cache(head_dim=96)), FAKE, FAKE, 1, 4, FAKE, None) == EUNSUP


def test_gated_combine_validation():
    L = abi()
    g = L.omnimem_gated_combine
    assert g(2, 8, 2, 64, FAKE, None, None, FAKE, FAKE, None) == EUNSUP        # dtype
    assert g(0, 8, 2, 96, FAKE, None, None, FAKE, FAKE, None) == EUNSUP        # head_dim
    assert g(0, -1, 2, 64, FAKE, None, None, FAKE, FAKE, None) == EINVAL
    assert g(0, 8, 2, 64, None, None, None, FAKE, FAKE, None) == EINVAL        # no branch
    assert g(0, 8, 2, 64, FAKE, FAKE + 8, None, FAKE, FAKE, None) == EINVAL    # misaligned branch
    assert g(0, 8, 2, 64, FAKE, None, None, FAKE + 2, FAKE, None) == EINVAL    # misaligned gates
    assert g(0, 8, 2, 64, FAKE, None, None, FAKE, None, None) == EINVAL        # no output
    assert g(0, 0, 2, 64, None, None, None, None, None, None) == 0             # empty: no-op


def test_probe_library_exports_its_header():
    """The roofline probes (a measurement library outside the attention ABI) load and
    export exactly what include/omnimem_probe.h declares."""
    import subprocess
    from paper_2605_30519_amd import _build
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "omnimem_probe.h")).read(), flags=re.S)
    declared = sorted(set(re.findall(r"\b(omnimem_probe_[a-z_0-9]+)\s*\(", text)))
    assert declared
    ctypes.CDLL(_build.PROBE_LIB)
    out = subprocess.run(["nm", "-D", "--defined-only", _build.PROBE_LIB], capture_output=True, text=True).stdout
    exported = sorted({line.split()[-1] for line in out.splitlines() if " T " in line and "omnimem" in line})
    assert exported == declared


def test_probe_argument_checks():
    """Every probe refuses bad arguments with -1 before it touches the GPU (so this
    runs without one)."""
    from paper_2605_30519_amd import _build
    P = ctypes.CDLL(_build.PROBE_LIB)
    P.omnimem_probe_mfma_bf16.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_void_p]
    P.omnimem_probe_mfma_f32.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_void_p, ctypes.c_void_p]
    P.omnimem_probe_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
    P.omnimem_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    sink = ctypes.c_void_p(0x1000)
    assert P.omnimem_probe_mfma_bf16(0, 0, 1, 1, sink, None) == -1       # no iterations
    assert P.omnimem_probe_mfma_bf16(1, 1, 1, 3, sink, None) == -1       # three waves per SIMD
    assert P.omnimem_probe_mfma_bf16(0, 1, 1, 1, None, None) == -1       # no sink
    assert P.omnimem_probe_mfma_bf16(2, 1, 1, 1, sink, None) == -1       # unknown operand kind
    P.omnimem_probe_softmax_slot.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                             ctypes.c_void_p]
    assert P.omnimem_probe_softmax_slot(2, 1, 1, sink, None) == -1       # unknown operand source
    assert P.omnimem_probe_softmax_slot(0, 0, 1, sink, None) == -1       # no iterations
    assert P.omnimem_probe_softmax_slot(1, 1, 0, sink, None) == -1       # no workgroups
    assert P.omnimem_probe_softmax_slot(0, 1, 1, None, None) == -1       # no sink
    assert P.omnimem_probe_mfma_f32(2, 1, 1, 1, sink, None) == -1        # unknown shape
    assert P.omnimem_probe_mfma_f32(0, 1, 0, 1, sink, None) == -1        # no workgroups
    assert P.omnimem_probe_mfma_f32(1, 1, 1, 1, None, None) == -1        # no sink
    buf = ctypes.c_void_p(0x10000)
    assert P.omnimem_probe_copy(buf, None, 64, 1, None) == -1            # no destination
    assert P.omnimem_probe_copy(buf, buf, 24, 1, None) == -1             # not a multiple of 16
    assert P.omnimem_probe_copy(ctypes.c_void_p(0x10008), buf, 64, 1, None) == -1  # misaligned
    assert P.omnimem_probe_read(buf, 64, 0, sink, None) == -1            # no workgroups
    assert P.omnimem_probe_read(buf, 64, 1, None, None) == -1            # no sink


def test_scratch_guard_reads_resource_remarks():
    """The build's check that the 64-row attention kernel keeps everything in
    registers: it reads the compiler's per-kernel resource remarks and names a
    listed kernel that reports scratch memory or spilled VGPRs (canned remarks in
    the compiler's format, so this runs without compiling)."""
    from paper_2605_30519_amd import _build

    def remarks(name, scratch, spill):
        pre = "attention.hip:836:1: remark: "
        return "\n".join([f"{pre}Function Name: {name} [-Rpass-analysis=kernel-resource-usage]",
                          f"{pre}    VGPRs: 256 [-Rpass-analysis=kernel-resource-usage]",
                          f"{pre}    ScratchSize [bytes/lane]: {scratch} [-Rpass-analysis=kernel-resource-usage]",
                          f"{pre}    VGPRs Spill: {spill} [-Rpass-analysis=kernel-resource-usage]"])
    r64 = "_ZN7omnimem12_GLOBAL__N_115k_attn_bf16_r64ILi128EEEvNS0_8AttnArgsE"
    other = "_ZN7omnimem12_GLOBAL__N_110k_attn_f32ILi64EEEvNS0_8AttnArgsE"
    kernels = _build.NO_SCRATCH["attention.hip"]
    assert _build.scratch_users(remarks(r64, 0, 0) + "\n" + remarks(other, 64, 3), kernels) == []
    bad = _build.scratch_users(remarks(other, 0, 0) + "\n" + remarks(r64, 1088, 0), kernels)
    assert bad == [f"{r64}: ScratchSize [bytes/lane]: 1088"]
    bad = _build.scratch_users(remarks(r64, 0, 5), kernels)
    assert bad == [f"{r64}: VGPRs Spill: 5"]
