"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): the argument checks of every entry point (validate.cpp, plan.cpp), the
LRU bookkeeping of the hot cache (lru_core.cpp) and the NUMA binding helpers
(numa.cpp) are built with both sanitizers into a host-only shim library
(tests/host_shim.cpp) and driven in a child interpreter that preloads the
sanitizer runtime:
  * every bad-argument case of tests/test_abi.py, which must return the same
    statuses as the real library;
  * random request sequences through the LRU bookkeeping, against the oracle's
    model of the policy, head by head, including requests whose copies are not all
    committed (the state must stay consistent);
  * CPU lists and NUMA nodes read from a fake sysfs tree.
Any out-of-bounds access, use after free or undefined operation aborts the child."""
import os
import subprocess
import sys

import pytest

from conftest import ROOT

CSRC = os.path.join(ROOT, "paper_2605_30519_amd", "csrc")
HERE = os.path.dirname(os.path.abspath(__file__))
SOURCES = [os.path.join(CSRC, f) for f in ("validate.cpp", "plan.cpp", "lru_core.cpp", "numa.cpp")]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


CHILD = r'''
import ctypes, os, sys
import numpy as np
sys.path[:0] = [{repo!r}, {tests!r}]
import oracle
import test_abi
from paper_2605_30519_amd import omnimem as om

shim = om._configure(ctypes.CDLL({so!r}), required=False)
test_abi.abi = lambda: shim

# 1. the ABI test's bad-argument cases
for kw, want in test_abi.CACHE_CASES:
    test_abi.test_cache_validation(kw, want)
test_abi.test_host_helpers()
test_abi.test_select_validation()
test_abi.test_attention_validation()
test_abi.test_select_noalloc_validation()
test_abi.test_per_head_tables_and_chunk_decode_validation()
test_abi.test_gated_combine_validation()
test_abi.test_compressed_cache_validation()
print("validation ok")

# 2. the LRU bookkeeping against the oracle's policy model, per head
i32p = ctypes.POINTER(ctypes.c_int32)
shim.shim_lru_new.restype = ctypes.c_void_p
shim.shim_lru_new.argtypes = [ctypes.c_int] * 3
shim.shim_lru_free.argtypes = [ctypes.c_void_p]
shim.shim_lru_plan.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, i32p, ctypes.c_int,
                               ctypes.POINTER(ctypes.c_int)]
shim.shim_lru_commit.argtypes = [ctypes.c_void_p] + [ctypes.c_int] * 4
shim.shim_lru_slot_of.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int]
shim.shim_lru_chunk_in.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int]
shim.shim_lru_counts.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)]
assert shim.shim_lru_new(0, 2, 3) is None and shim.shim_lru_new(2, 0, 3) is None

def plan(core, needed):
    cap = needed.size + 1
    buf = (ctypes.c_int32 * (4 * cap))()
    count = ctypes.c_int(0)
    arr = np.ascontiguousarray(needed, dtype=np.uint8)
    rc = shim.shim_lru_plan(core, arr.ctypes.data_as(ctypes.c_void_p), arr.shape[1], buf, cap,
                            ctypes.byref(count))
    return rc, [tuple(buf[4 * i: 4 * i + 4]) for i in range(count.value)]

rng = np.random.default_rng(5)
for trial in range(40):
    H, slots, chunks = int(rng.integers(1, 4)), int(rng.integers(1, 6)), int(rng.integers(1, 12))
    core = shim.shim_lru_new(H, slots, chunks)
    reqs = [[] for _ in range(H)]
    for step in range(30):
        n = int(rng.integers(0, chunks + 1))
        needed = (rng.random((H, n)) < rng.uniform(0.05, 0.6)).astype(np.uint8)
        over = [h for h in range(H) if needed[h].sum() > slots]
        counts_before = (ctypes.c_int64 * 3)()
        shim.shim_lru_counts(core, counts_before)
        rc, loads = plan(core, needed)
        if over:
            assert rc == -1 and loads == []
            after = (ctypes.c_int64 * 3)()
            shim.shim_lru_counts(core, after)
            assert list(after) == list(counts_before)
            continue
        assert rc == 0
        for h in range(H):
            reqs[h].append(np.nonzero(needed[h])[0].tolist())
        for (h, c, s, old) in loads:
            shim.shim_lru_commit(core, h, c, s, old)
        for h in range(H):
            ref = oracle.lru_simulate(reqs[h], slots)
            got = {{c: shim.shim_lru_slot_of(core, h, c) for c in range(chunks) if shim.shim_lru_slot_of(core, h, c) >= 0}}
            assert got == ref["slot_of"], (trial, step, h, got, ref["slot_of"])
    counts = (ctypes.c_int64 * 3)()
    shim.shim_lru_counts(core, counts)
    refs = [oracle.lru_simulate(reqs[h], slots) for h in range(H)]
    assert list(counts) == [sum(r["hits"] for r in refs), sum(r["misses"] for r in refs),
                            sum(r["evictions"] for r in refs)], (list(counts), refs)
    shim.shim_lru_free(core)

# uncommitted loads (copies that could not be enqueued) leave their slots free and
# their chunks non-resident; the two tables stay inverse to each other
core = shim.shim_lru_new(2, 3, 8)
for step in range(25):
    needed = (rng.random((2, 8)) < 0.3).astype(np.uint8)
    for h in range(2):
        while needed[h].sum() > 3:
            needed[h, np.nonzero(needed[h])[0][0]] = 0
    rc, loads = plan(core, needed)
    assert rc == 0
    for (h, c, s, old) in loads[: len(loads) // 2]:
        shim.shim_lru_commit(core, h, c, s, old)
    for (h, c, s, old) in loads[len(loads) // 2:]:
        assert shim.shim_lru_slot_of(core, h, c) == -1 and shim.shim_lru_chunk_in(core, h, s) == -1
    for h in range(2):
        for s in range(3):
            c = shim.shim_lru_chunk_in(core, h, s)
            assert c < 0 or shim.shim_lru_slot_of(core, h, c) == s
        for c in range(8):
            s = shim.shim_lru_slot_of(core, h, c)
            assert s < 0 or shim.shim_lru_chunk_in(core, h, s) == c
assert plan(core, np.ones((2, 9), np.uint8))[0] == -1       # n beyond the chunks
shim.shim_lru_free(core)
print("lru ok")

# 3. CPU lists and NUMA nodes from a fake sysfs tree
mask = (ctypes.c_uint64 * 2)()
shim.shim_parse_cpu_list.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_uint64), ctypes.c_int]
assert shim.shim_parse_cpu_list(b"0-3,8,10-11\n", mask, 2) == 7 and mask[0] == 0b110100001111
assert shim.shim_parse_cpu_list(b"64-65", mask, 2) == 2 and mask[1] == 3 and mask[0] == 0
for bad in (b"3-1", b"1,,2", b"a", b"1-", b"128", b"1,"):
    assert shim.shim_parse_cpu_list(bad, mask, 2) == -1, bad
root = {root!r}
dev = os.path.join(root, "bus", "pci", "devices", "0000:c1:00.0")
os.makedirs(dev)
open(os.path.join(dev, "numa_node"), "w").write("1\n")
shim.shim_numa_node_of_pci.argtypes = [ctypes.c_char_p, ctypes.c_char_p]
assert shim.shim_numa_node_of_pci(root.encode(), b"0000:C1:00.0") == 1
assert shim.shim_numa_node_of_pci(root.encode(), b"0000:c2:00.0") == -1
assert shim.shim_numa_node_of_pci(root.encode(), b"../../etc") == -1
open(os.path.join(dev, "numa_node"), "w").write("-1\n")
assert shim.shim_numa_node_of_pci(root.encode(), b"0000:c1:00.0") == -1
mine = sorted(os.sched_getaffinity(0))
for node, cpus in ((0, ",".join(str(c) for c in mine)), (1, "4000-4001")):
    d = os.path.join(root, "devices", "system", "node", f"node{{node}}")
    os.makedirs(d)
    open(os.path.join(d, "cpulist"), "w").write(cpus + "\n")
shim.shim_bind_thread_to_node.argtypes = [ctypes.c_char_p, ctypes.c_int]
assert shim.shim_bind_thread_to_node(root.encode(), 1) in (-1, 1)    # CPUs beyond the mask or none shared
assert shim.shim_bind_thread_to_node(root.encode(), 7) == -1         # no such node
assert shim.shim_bind_thread_to_node(root.encode(), 0) in (0, -1)    # -1 only if set_mempolicy is not allowed
assert sorted(os.sched_getaffinity(0)) == mine
print("numa ok")
'''


def test_host_code_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    so = tmp_path / "libomnimem_host_san.so"
    subprocess.check_call(["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-o", str(so),
                           os.path.join(HERE, "host_shim.cpp"), *SOURCES])
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    code = CHILD.format(repo=ROOT, tests=HERE, so=str(so), root=str(tmp_path / "sys"))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0 and "numa ok" in r.stdout, (r.stdout[-2000:], r.stderr[-4000:])
