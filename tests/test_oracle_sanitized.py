"""The oracle's C source under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): built with both, loaded in a child interpreter with the sanitizer runtime
preloaded, and driven through the whole pin battery.  Any out-of-bounds access,
use after free or undefined operation aborts the child with a report."""
import os
import subprocess
import sys

import pytest

import oracle

SRC = os.path.join(os.path.dirname(oracle.__file__), "omnimem_oracle.c")
HERE = os.path.dirname(os.path.abspath(__file__))


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


CHILD = """
import sys
sys.path[:0] = [{repo!r}, {tests!r}]
import oracle
from oracle_pins import ALL_PINS
with oracle.using_library({so!r}):
    for pin in ALL_PINS:
        pin()
print("pins ok:", len(ALL_PINS))
"""


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    so = tmp_path / "liboracle_san.so"
    subprocess.check_call(["gcc", "-O1", "-g", "-fopenmp", "-fPIC", "-shared", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-o", str(so), SRC,
                           "-lm"])
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    code = CHILD.format(repo=os.path.dirname(HERE), tests=HERE, so=str(so))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0 and "pins ok" in r.stdout, (r.stdout[-2000:], r.stderr[-4000:])
