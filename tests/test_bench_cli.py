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


def test_traffic_summary_from_counter_files(tmp_path, monkeypatch):
    """profiles/traffic.json is rebuilt from two rocprofv3 counter files:
    each op's median counter, scaled by the known-size copy."""
    import csv
    import json
    import bench
    cols = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    dec = "ssn::decompress_mfma_bf16<2, true, 0, 64, 1, 8, true, false, false, 1, 1, 1>(float const*)"
    pg = "ssn::compress_rows_bf16<4, false, true, 8, 1, true, false, true, 4, false>(unsigned short const*)"
    tab = pg
    cp = "__amd_rocclr_copyBuffer"
    fetch = [(cp, 1, 131072.0), (dec, 131072, 140000.0), (dec, 131072, 150000.0), (dec, 131072, 145000.0),
             (pg, 131072, 133000.0), (tab, 524288, 526000.0), ("other_kernel", 64, 1.0)]
    write = [(cp, 1, 262144.0), (dec, 131072, 262144.0), (dec, 131072, 262144.0), (dec, 131072, 262144.0),
             (pg, 131072, 7000.0), (tab, 524288, 32768.0), ("other_kernel", 64, 1.0)]
    paths = []
    for name, rows, counter in (("f.csv", fetch, "FETCH_SIZE"), ("w.csv", write, "WRITE_SIZE")):
        p = tmp_path / name
        with open(p, "w", newline="") as f:
            w = csv.writer(f)
            w.writerow(cols)
            for i, (k, g, v) in enumerate(rows):
                w.writerow([i, g, k, counter, v])
        paths.append(str(p))
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    bench.summarize_traffic(*paths)
    t = json.load(open(tmp_path / "traffic.json"))
    assert t["kernel_source_hash"] == bench.kernel_source_hash()
    assert abs(t["calibration"]["fetch_scale"] - 2.0) < 1e-9
    assert abs(t["calibration"]["write_scale"] - 1.0) < 1e-9
    d = t["kernels"]["decompress"]
    assert d["read_bytes"] == int(145000.0 * 1024 * 2.0) and d["write_bytes"] == 262144 * 1024
    assert t["kernels"]["project_grad"]["grid"] == 131072
    assert t["kernels"]["project_table"]["read_bytes"] == int(526000.0 * 1024 * 2.0)
    assert set(t["kernels"]) == {"decompress", "project_grad", "project_table"}


def test_counter_summary_table(tmp_path, capsys):
    """The general counter table: medians per kernel and grid, FETCH_SIZE /
    WRITE_SIZE scaled by the largest copy of each file (small copies of the
    same run are ignored), L2 hit share from TCC_HIT_sum / TCC_MISS_sum, and
    kernels outside the library left out."""
    import csv
    import bench
    cols = ["Dispatch_Id", "Grid_Size", "Kernel_Name", "Counter_Name", "Counter_Value"]
    sp = "void ssn::sparta_copy4(float const*, float*, long)"
    cp = "__amd_rocclr_copyBuffer"

    def write(name, rows):
        p = tmp_path / name
        with open(p, "w", newline="") as f:
            w = csv.writer(f)
            w.writerow(cols)
            for i, (k, g, c, v) in enumerate(rows):
                w.writerow([i, g, k, c, v])
        return str(p)

    fetch = write("f.csv", [(cp, 131072, "FETCH_SIZE", 131072.0), (cp, 512, "FETCH_SIZE", 2.0),
                            (cp, 512, "FETCH_SIZE", 2.0), (cp, 512, "FETCH_SIZE", 2.0),
                            (sp, 1000, "FETCH_SIZE", 30000.0), (sp, 1000, "FETCH_SIZE", 31000.0),
                            (sp, 1000, "FETCH_SIZE", 32000.0), ("torch_kernel", 64, "FETCH_SIZE", 5.0)])
    wr = write("w.csv", [(cp, 131072, "WRITE_SIZE", 262144.0), (sp, 1000, "WRITE_SIZE", 62500.0)])
    l2 = write("l.csv", [(sp, 1000, "TCC_HIT_sum", 300.0), (sp, 1000, "TCC_MISS_sum", 100.0)])
    bench.summarize_counters([fetch, wr, l2], 256)
    out = capsys.readouterr().out
    rows = [r for r in out.splitlines() if r.startswith("| `")]
    assert len(rows) == 1 and "torch_kernel" not in out
    cells = [c.strip() for c in rows[0].strip("|").split("|")]
    head = [c.strip() for c in [r for r in out.splitlines() if r.startswith("| kernel")][0].strip("|").split("|")]
    got = dict(zip(head, cells))
    assert got["op"] == "sparta" and got["grid (threads)"] == "1000" and got["dispatches"] == "3"
    assert got["FETCH_SIZE"] == "31000" and got["WRITE_SIZE"] == "62500"
    assert got["scaled MB read"] == f"{31000 * 1024 * 2.0 / 1e6:.1f}"
    assert got["scaled MB written"] == f"{62500 * 1024 * 1.0 / 1e6:.1f}"
    assert got["L2 hit %"] == "75.0"
