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


def test_bench_has_no_undefined_names():
    """Every name bench.py reads is bound in its own scope, an enclosing
    scope, the module or the builtins: the bench only runs on a GPU, so a
    stray name would otherwise surface there first."""
    import ast
    import builtins

    src = open(os.path.join(ROOT, "bench.py"), encoding="utf-8").read()
    tree = ast.parse(src)

    def bound_names(node):
        """Names bound directly in the scope of `node` (not in nested scopes)."""
        names = set()
        if isinstance(node, (ast.FunctionDef, ast.AsyncFunctionDef, ast.Lambda)):
            a = node.args
            for arg in a.posonlyargs + a.args + a.kwonlyargs:
                names.add(arg.arg)
            if a.vararg:
                names.add(a.vararg.arg)
            if a.kwarg:
                names.add(a.kwarg.arg)
        body = node.body if isinstance(node.body, list) else [node.body]
        stack = list(body)
        while stack:
            n = stack.pop()
            if isinstance(n, (ast.FunctionDef, ast.AsyncFunctionDef, ast.ClassDef)):
                names.add(n.name)
                stack.extend(n.decorator_list)
                continue
            if isinstance(n, ast.Lambda):
                continue
            if isinstance(n, (ast.ListComp, ast.SetComp, ast.DictComp, ast.GeneratorExp)):
                continue
            if isinstance(n, ast.Name) and isinstance(n.ctx, (ast.Store, ast.Del)):
                names.add(n.id)
            elif isinstance(n, (ast.Import, ast.ImportFrom)):
                for al in n.names:
                    names.add((al.asname or al.name).split(".")[0])
            elif isinstance(n, ast.ExceptHandler) and n.name:
                names.add(n.name)
            elif isinstance(n, (ast.Global, ast.Nonlocal)):
                names.update(n.names)
            stack.extend(ast.iter_child_nodes(n))
        return names

    module_names = bound_names(tree) | set(dir(builtins)) | {"__file__", "__name__"}
    missing = []

    def visit(node, env):
        if isinstance(node, (ast.FunctionDef, ast.AsyncFunctionDef, ast.Lambda)):
            for dflt in node.args.defaults + node.args.kw_defaults:
                if dflt is not None:
                    visit(dflt, env)
            env = env | bound_names(node)
            body = node.body if isinstance(node.body, list) else [node.body]
            for n in body:
                visit(n, env)
            return
        if isinstance(node, (ast.ListComp, ast.SetComp, ast.DictComp, ast.GeneratorExp)):
            inner = set(env)
            for gen in node.generators:
                visit(gen.iter, inner)
                for t in ast.walk(gen.target):
                    if isinstance(t, ast.Name):
                        inner.add(t.id)
                for cond in gen.ifs:
                    visit(cond, inner)
            for part in ([node.key, node.value] if isinstance(node, ast.DictComp) else [node.elt]):
                visit(part, inner)
            return
        if isinstance(node, ast.Name) and isinstance(node.ctx, ast.Load) and node.id not in env:
            missing.append(f"{node.id} (line {node.lineno})")
        for child in ast.iter_child_nodes(node):
            visit(child, env)

    for n in tree.body:
        visit(n, module_names)
    assert not missing, "names read but never bound: " + ", ".join(missing)
