"""bench.py's command line, on the CPU: the options parse, and a request for
more than one GPU ends with a message and exit status 2 before any GPU work."""
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
                "--no-fused-attention", "--no-decode", "--copy-probe-mib"):
        assert opt in p.stdout


def test_more_than_one_gpu_is_refused():
    p = _bench("--gpus", "2")
    assert p.returncode == 2
    assert "one GPU" in p.stderr
