"""bench.py's command line, on the CPU: the options parse, and a request for
more than one GPU, or for a workload that is not a whole decoder layer, ends
with a message before any GPU work."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)


def test_help_lists_the_options():
    p = _bench("--help")
    assert p.returncode == 0
    for opt in ("--gpus", "--steps", "--warmup", "--ratios", "--no-cpu-baseline",
                "--no-fused-attention", "--no-decode", "--copy-probe-mib", "--no-policies",
                "--no-attention-chain", "--no-mlp-chain", "--no-pv", "--no-paper-kernels",
                "--no-layer-forward", "--no-decode-batched", "--workload"):
        assert opt in p.stdout


def test_more_than_one_gpu_is_refused():
    p = _bench("--gpus", "2")
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_parity_workloads_are_refused():
    # the step is a whole decoder layer; the single-product workloads are
    # parity-test cases, refused before any GPU work
    for wk in ("mlp_1b", "linear_f32", "attn_4k", "no_such_workload"):
        p = _bench("--workload", wk)
        assert p.returncode != 0
        assert wk in p.stderr
