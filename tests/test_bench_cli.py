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


def test_byte_model_and_host_fields():
    """The sweep's algorithmic bytes follow the model 12 nnz + 28 n + 4 (col
    and val per nonzero, row_ptr, the x view, b, the written iterate); the
    CPU baseline names the cores this process may use."""
    sys.path.insert(0, ROOT)
    import bench
    assert bench.sweep_bytes(64_000_000, 447_040_000) == 12 * 447_040_000 + 28 * 64_000_000 + 4
    # compact forms: one value per column in place of one per nonzero; values
    # by diagonal and a mask byte per row in place of columns and row pointers
    n, nnz = 4_194_304, 67_108_864
    assert (bench.format_sweep_bytes(n, nnz, "column values", 0)
            == bench.sweep_bytes(n, nnz) - 8 * nnz + 8 * n)
    n, nnz = 64_000_000, 447_040_000
    assert (bench.format_sweep_bytes(n, nnz, "diagonals", 7)
            == 56 * n + n + 24 * n)
    assert bench.format_sweep_bytes(n, nnz, "general", 7) == bench.sweep_bytes(n, nnz)
    cores, model = bench.host_cpu()
    assert cores == len(os.sched_getaffinity(0)) and cores >= 1
    assert model is None or isinstance(model, str)
