"""bench.py's command line on the CPU: more than one GPU is refused with a
message (the benchmark measures one GPU), and the copy probe and configurations
are listed."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=300, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _bench("--gpus", "2")
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_help_lists_every_workload():
    r = _bench("--help")
    assert r.returncode == 0
    for cfg in ("jacobi-1d", "jacobi-2d", "pagerank-rmat", "jacobi-3d", "allgatherv", "allreduce",
                "hypercube", "threshold", "mf"):
        assert cfg in r.stdout
