"""CPU checks of the benchmark script's command line (no GPU needed)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_parses_and_imports():
    sys.path.insert(0, ROOT)
    import bench  # noqa: F401  (a syntax error or a broken module fails here)

    assert callable(bench.main) and callable(bench.cpu_baseline)


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
