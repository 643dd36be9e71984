"""Builds libomnimem.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJ_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libomnimem.so")
PROBE_LIB = os.path.join(PKG, "libomnimem_probe.so")
SOURCES = ["api.hip", "select.hip", "prob.hip", "attention.hip", "union_gather.hip", "fuse.hip", "offload.hip"]
# host-only C++ (no HIP): argument checks, work plans, the LRU bookkeeping and the
# NUMA binding, built by the host compiler; tests also build them under sanitizers
HOST_SOURCES = ["validate.cpp", "plan.cpp", "lru_core.cpp", "numa.cpp"]
HEADERS = ["device_common.h", "launch.h", "plan.h", "validate.h", "lru_core.h", "numa.h"]
CXX = os.environ.get("CXX", "g++")
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-O3",
    "--offload-arch=gfx950",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    "-Wall",
    # no packed fp32 instructions in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


# Per-source extra flags for attention.hip.  The 64-row attention kernel needs more
# than 256 registers per lane; MFMA results in arch VGPRs (not accumulation
# registers) keep its softmax VALU work free of register-file copies.  Without
# IEEE-mode NaN quieting, fmaxf over MFMA results maps to plain v_max3 (no NaN is
# ever produced or consumed on purpose there).
EXTRA_FLAGS = {"attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans", "-mno-amdgpu-ieee"]}

# Kernels that must keep every value in registers.  The 64-row attention kernel
# issues its P.V MFMAs from inline asm with O in fixed accumulation registers, and its
# hazard waits assume that nothing else touches those registers while an MFMA runs; a
# spill or a private array moved to scratch memory would add such accesses (and be
# slow).  The build fails if the compiler reports scratch use for them.
NO_SCRATCH = {"attention.hip": ("k_attn_bf16_r64",)}
RESOURCE_REMARK = "-Rpass-analysis=kernel-resource-usage"


def scratch_users(remarks: str, kernels) -> list:
    """Kernels among `kernels` (name fragments) whose resource remarks report a
    nonzero scratch size or spilled VGPRs."""
    bad, name = [], None
    for line in remarks.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif name and any(k in name for k in kernels):
            for key in ("ScratchSize [bytes/lane]:", "VGPRs Spill:"):
                if key in line and int(line.split(key)[1].split()[0]) != 0:
                    bad.append(f"{name}: {key} {line.split(key)[1].split()[0]}")
    return bad


def build(verbose: bool = False) -> str:
    """Compile every source (in parallel) and link libomnimem.so.  Always rebuilds."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    procs = []
    for src in SOURCES:
        obj = os.path.join(OBJ_DIR, src.replace(".hip", ".o"))
        remark = [RESOURCE_REMARK] if src in NO_SCRATCH else []
        cmd = [HIPCC, *FLAGS, *EXTRA_FLAGS.get(src, []), *remark, "-c", os.path.join(CSRC, src), "-o", obj]
        procs.append((src, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    for src in HOST_SOURCES:
        obj = os.path.join(OBJ_DIR, src.replace(".cpp", ".host.o"))
        cmd = [CXX, *HOST_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        procs.append((src, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    objs = []
    errors = []
    for src, obj, p in procs:
        out, _ = p.communicate()
        if p.returncode == 0 and src in NO_SCRATCH:
            bad = scratch_users(out, NO_SCRATCH[src])
            if bad:
                errors.append(f"{src}: kernels that must not use scratch memory do:\n" + "\n".join(bad))
        out = "\n".join(line for line in out.splitlines()
                        if "packed-fp32-ops" not in line and "kernel-resource-usage" not in line)
        if p.returncode != 0:
            errors.append(f"{src}:\n{out}")
        elif verbose and out.strip():
            print(out)
        objs.append(obj)
    if errors:
        raise RuntimeError("hipcc failed:\n" + "\n".join(errors))
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    # the roofline probes: a library of their own, outside the attention ABI
    tmp = PROBE_LIB + ".tmp%d" % os.getpid()
    subprocess.check_call([HIPCC, *FLAGS, "-shared", os.path.join(CSRC, "probe.hip"), "-o", tmp],
                          stderr=subprocess.DEVNULL if not verbose else None)
    os.replace(tmp, PROBE_LIB)
    return LIB


def is_built() -> bool:
    return os.path.exists(LIB) and os.path.exists(PROBE_LIB)
