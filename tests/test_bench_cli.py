"""bench.py's command-line contract without a GPU: more than one GPU is refused with
a message, and every workload the benchmark documents is selectable."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def _run(*args):
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_workloads_are_listed():
    r = _run("--help")
    assert r.returncode == 0
    for wl in ("llada8b_bf16_p512_w32", "llada8b_bf16_p1024_w64_spec", "llada8b_w8_p4096_w64_spec",
               "llada8b_bf16_e2e128", "llada8b_bf16_e2e128_mbsd", "llada8b_bf16_prefill512", "dream7b_bf16_p512_w32",
               "llada8b_q4_p512_w32"):
        assert wl in r.stdout
