"""bench.py's host-side contract, on the CPU: one JSON line is a GPU matter, but the
argument handling that decides what runs is not."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT, capture_output=True,
                          text=True, timeout=300)


def test_bench_measures_one_gpu_only():
    # This library is a single-GPU kernel library: asking for more GPUs ends with a message
    # (before any device is touched), not with a number.
    r = _bench("--gpus", "2")
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr


def test_bench_defaults_to_the_largest_single_gpu_workload():
    r = _bench("--help")
    assert r.returncode == 0
    for name in ("tiny_fp32", "smollm2_prefill", "llama7b_qkv_prefill", "llama7b_swiglu_decode", "layernorm_linear",
                 "mla_kv_down"):
        assert name in r.stdout
    assert "default workload is the largest single-GPU configuration" in r.stdout.replace("\n", " ")
