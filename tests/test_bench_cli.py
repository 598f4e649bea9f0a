"""Host side of the benchmark: one GPU only, refused before any GPU work."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_algorithmic_bytes_count_distinct_rows_once():
    sys.path.insert(0, ROOT)
    import bench
    N, d, k, u = 32768, 4096, 64, 28993
    # X once, distinct E rows once, Z, U, ids
    assert bench.algorithmic_bytes("compress", N, d, k, u) == N * d * 2 + u * d * 2 + N * k * 4 + d * k * 2 + 4 * N
    assert bench.algorithmic_bytes("decompress", N, d, k, u) == bench.algorithmic_bytes("compress", N, d, k, u)
    assert bench.algorithmic_bytes("project_grad", N, d, k, u) == N * d * 2 + N * k * 4 + d * k * 2
