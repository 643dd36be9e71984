"""bench.py's command line, on the CPU: a request for more than one GPU is refused
with a message before anything touches a GPU, and every measurement mode parses."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def run(*args):
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus 1" in r.stderr
    assert r.stdout == ""


def test_world_size_above_one_is_refused():
    env = dict(os.environ, WORLD_SIZE="2")
    r = subprocess.run([sys.executable, BENCH], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_modes_are_listed():
    r = run("--help")
    assert r.returncode == 0
    for flag in ("--steps", "--warmup", "--attn-only", "--select-only", "--small-group-only", "--power-clock",
                 "--cu-fill", "--prob-only", "--no-sweep", "--no-cpu-baseline", "--no-stress"):
        assert flag in r.stdout, flag
