#!/usr/bin/env python3
"""Benchmark of the subspace-network stage-boundary codec on one MI355X.

One step = one microbatch through every codec operation of a pipeline stage
boundary, on the 8B-stage-shaped workload (N = 16 x 2048 = 32768 tokens,
d = 4096, k = 64, V = 131072, bf16 storage, fp32 coordinates):

    decompress (incoming coordinates -> activation), project_grad (gradient
    leaving through the input boundary), compress (activation leaving through
    the output boundary), expand_grad (incoming gradient coordinates).

Two independent microbatch input sets alternate between steps so that
consecutive steps gather different embedding rows, and within a step the
compressed microbatch draws its own token ids (the decompressed and the
compressed activations of a stage belong to different microbatches in a
pipeline), so compress never finds the rows decompress just gathered in the
caches.  Inputs are resident in HBM before the timed region starts.  The once-per-optimizer-step weight
re-projection (4 layers x (4096x4096 + 4096x14336)) is timed separately and
reported under "weights" (bf16 storage) and "weights_f32" (float32 master
weights).  The same step with compress against the projected
embedding table (Z = X U - (E U)[ids], table formed once outside the timed
region) is timed separately and reported under "variants"; the headline value
is the step with compress as written in Eq. (2).  The same step at the
paper's own stage shapes (Pluralis-8B d=5120, k=51, V=128,256, S=4096; the 1B
ablation model d=2048, k=40, S=2048; b = 1, 2 and 3 coalesced sequences) and the
weight re-projection at those shapes are reported under "paper_shapes", and
the k=64 points of the sweep (d=4096, N=4096..131072, Zipf(1.1) ids) under
"sweep_k64".

Prints ONE JSON line (rank 0).  `--gpus` above 1 is refused: this build runs
on one GPU.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
MFMA_F32_PEAK_TFLOPS = 157.3    # MI355X dense float32 MFMA
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ["paper_2607_13332_amd/csrc/codec_kernels.hip",
                  "paper_2607_13332_amd/csrc/f32_kernels.hip",
                  "paper_2607_13332_amd/csrc/f32_strips.h",
                  "paper_2607_13332_amd/csrc/f32_weights.hip",
                  "paper_2607_13332_amd/csrc/weights_kernels.hip",
                  "paper_2607_13332_amd/csrc/reparam_kernels.hip",
                  "paper_2607_13332_amd/csrc/sparta_kernels.hip",
                  "paper_2607_13332_amd/csrc/ssn_device.h"]


def _code_only(src: str) -> str:
    """C++ source without comments and whitespace (the kernel sources hold no
    string literals that contain comment markers)."""
    import re
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return "".join(src.split())


def kernel_source_hash() -> str:
    """Hash of the kernel sources' code (comments and layout do not change
    what the counters measure)."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=400)
    p.add_argument("--warmup", type=int, default=200,
                   help="untimed steps first (the GPU's clocks settle after ~30 ms of sustained load)")
    p.add_argument("--settle-seconds", type=float, default=3.0,
                   help="before the warmup steps, untimed steps for this long: the first GPU "
                        "process on an idle box runs at lower clocks for a while (the headline "
                        "step measured 336 us cold against 301 us in the next process)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-weights", action="store_true")
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the k=64 sweep points (d=4096, N=4096..131072, Zipf ids)")
    p.add_argument("--no-reparam", action="store_true",
                   help="skip the reparameterized-SSN projection timings")
    p.add_argument("--no-sparta", action="store_true",
                   help="skip the sparse-averaging round (320M-parameter block)")
    p.add_argument("--no-paper-shapes", action="store_true",
                   help="skip the timings at the paper's own stage shapes (d=5120 k=51, d=2048 k=40)")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target CPU time of the oracle baseline sample")
    p.add_argument("--tokens", type=int, default=0, help="override N (testing only)")
    p.add_argument("--only", choices=("reparam", "sparta", "sweep", "paper", "weights", "f32"), default=None,
                   help="profiling aid: run only this section and print its JSON (no headline; "
                        "keeps its kernels apart from the codec's in a kernel trace)")
    p.add_argument("--sweep-tokens", type=str, default="",
                   help="with --only sweep / paper / reparam: comma-separated token counts to keep")
    p.add_argument("--select", type=str, default="",
                   help="with --only sweep / paper / reparam: comma-separated workload names to "
                        "keep (e.g. paper8b_b1,paper8b_b3), so that launches of equal total grid "
                        "from different workloads stay apart in a counter run")
    p.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"), default=None,
                   help="no GPU work: turn the counter_collection.csv files of a rocprofv3 "
                        "--pmc FETCH_SIZE run and a --pmc WRITE_SIZE run of this bench "
                        "(with --copy-calib 256) into profiles/traffic.json and print the table")
    p.add_argument("--summarize-counters", nargs="+", metavar="COUNTER_CSV", default=None,
                   help="no GPU work: per-kernel table (median per dispatch of every counter) of "
                        "the counter_collection.csv files of rocprofv3 --pmc runs of this bench; "
                        "FETCH_SIZE / WRITE_SIZE are scaled to bytes by the device copy that "
                        "--copy-calib MIB ran in the same process")
    p.add_argument("--summarize-trace", metavar="TRACE_CSV", default=None,
                   help="no GPU work: per-kernel table (grid, calls, average / min / max us, "
                        "share of the traced time) of a rocprofv3 --kernel-trace csv")
    p.add_argument("--copy-calib", type=int, default=0, metavar="MIB",
                   help="before the timed region, run a plain device copy of MIB MiB three times "
                        "(a known-size kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE); "
                        "the live device-copy reference rate is then skipped")
    return p.parse_args()


def algorithmic_bytes(op: str, N: int, d: int, k: int, u: int, s: int = 2) -> int:
    """Bytes each op must move: activations/gradients once, distinct embedding
    rows once, coordinates once, the basis and ids once."""
    U = d * k * s
    if op == "compress":
        return N * d * s + u * d * s + N * k * 4 + U + 4 * N
    if op == "decompress":
        return N * k * 4 + u * d * s + N * d * s + U + 4 * N
    if op in ("project_grad", "expand_grad"):
        return N * d * s + N * k * 4 + U
    if op == "compress_projected":
        return N * d * s + u * k * 4 + N * k * 4 + U + 4 * N
    raise ValueError(op)


def op_u(op: str, s) -> int:
    """Distinct embedding rows an op of input set s gathers."""
    return s["u_c"] if op in ("compress", "compress_projected") else s["u"]


def load_traffic(kernel_key: str):
    """HBM bytes per launch measured by rocprofv3 PMC counters, if the stored
    measurement was taken on the current kernel sources."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    ent = t.get("kernels", {}).get(kernel_key)
    return None if ent is None else ent.get("bytes_per_launch")


def _template_args(kernel_name: str):
    """Template arguments of a demangled kernel name, as strings."""
    if "<" not in kernel_name:
        return []
    inner = kernel_name.split("<", 1)[1].rsplit(">", 1)[0]
    return [a.strip() for a in inner.split(",")]


def traffic_op(kernel_name: str, grid: int):
    """Which headline op a dispatch of the headline bench run belongs to."""
    a = _template_args(kernel_name)
    if "copyBuffer" in kernel_name:
        return "calibration"
    if "decompress_mfma_bf16" in kernel_name and a[:1] == ["2"]:
        return "decompress" if a[1] == "true" else "expand_grad"
    if "compress_rows_bf16" in kernel_name and a[:1] == ["4"]:
        if a[1] == "true":
            return "compress"
        if a[-1] == "true":
            return "compress_projected"
        # the gradient projection over N = 32768 rows, or the table over V rows
        return "project_grad" if grid == 32768 // 128 * 512 else "project_table"
    if "project_weights_cols_bf16" in kernel_name:
        return "project_weights"
    return None


def summarize_traffic(fetch_csv: str, write_csv: str, calib_bytes: int = 256 << 20):
    """profiles/traffic.json from two rocprofv3 counter runs of this bench.

    Each counter is read in KiB per dispatch; both are scaled by what they
    read for the plain device copy of known size that --copy-calib runs (on
    this GPU FETCH_SIZE counts half of a copy's reads).  Per op: the median
    over its dispatches."""
    import csv
    import statistics

    def per_op(path, counter):
        vals, names = {}, {}
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                grid = int(r["Grid_Size"])
                op = traffic_op(r["Kernel_Name"], grid)
                if op is None:
                    continue
                vals.setdefault(op, []).append(float(r["Counter_Value"]))
                name = r["Kernel_Name"]
                names[op] = ((name[5:] if name.startswith("void ") else name).split("(")[0], grid)
        return vals, names

    fv, names = per_op(fetch_csv, "FETCH_SIZE")
    wv, _ = per_op(write_csv, "WRITE_SIZE")
    fscale = calib_bytes / (statistics.median(fv["calibration"]) * 1024.0)
    wscale = calib_bytes / (statistics.median(wv["calibration"]) * 1024.0)
    out = {"kernel_source_hash": kernel_source_hash(),
           "calibration": {"kernel": "__amd_rocclr_copyBuffer (torch copy_ of "
                                     f"{calib_bytes >> 20} MiB)",
                           "known_bytes": calib_bytes, "fetch_scale": round(fscale, 4),
                           "write_scale": round(wscale, 4)},
           "kernels": {}}
    rows = []
    for op in ("project_grad", "project_table", "compress_projected", "compress", "expand_grad",
               "decompress", "project_weights"):
        if op not in fv or op not in wv:
            continue
        fk, wk = statistics.median(fv[op]), statistics.median(wv[op])
        rb, wb = int(fk * 1024 * fscale), int(wk * 1024 * wscale)
        name, grid = names[op]
        out["kernels"][op] = {"kernel": name, "grid": grid, "fetch_kib": round(fk, 1),
                              "write_kib": round(wk, 1), "read_bytes": rb, "write_bytes": wb,
                              "bytes_per_launch": rb + wb}
        rows.append(f"| {op} | `{name}` | {grid} | {len(fv[op])} | {fk:.0f} | {wk:.0f} | "
                    f"{rb / 1e6:.1f} | {wb / 1e6:.1f} | {(rb + wb) / 1e6:.1f} |")
    with open(os.path.join(PROFILES, "traffic.json"), "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(f"scales: fetch {fscale:.4f}, write {wscale:.4f}")
    print("| op | kernel | grid | dispatches | FETCH KiB | WRITE KiB | scaled MB read | "
          "scaled MB written | total MB |")
    print("|---|---|---|---|---|---|---|---|---|")
    print("\n".join(rows))


def summarize_counters(paths, calib_mib: int = 256):
    """Markdown table of rocprofv3 --pmc runs of this bench: one row per
    kernel of this library and grid, the median per dispatch of every
    counter collected.  FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are
    scaled to bytes by what the same counter read for the plain device copy
    of calib_mib MiB that --copy-calib runs in each process (the copy
    dispatches of the largest grid in that file); the L2 hit share is
    TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum) where both were collected."""
    import csv
    import statistics

    def short(name):
        return (name[5:] if name.startswith("void ") else name).split("(")[0]

    rows, counters, scale = {}, [], {}
    for path in paths:
        copies, recs = {}, []
        with open(path) as f:
            for r in csv.DictReader(f):
                name, c = short(r["Kernel_Name"]), r["Counter_Name"]
                key = (r["Dispatch_Id"], c)
                if "copyBuffer" in name:
                    copies.setdefault(int(r["Grid_Size"]), {})[key] = float(r["Counter_Value"])
                elif name.startswith("ssn::"):
                    recs.append((name, int(r["Grid_Size"]), key, c, float(r["Counter_Value"])))
        if copies:
            big = copies[max(copies)]
            for c in ("FETCH_SIZE", "WRITE_SIZE"):
                v = [x for (_, cc), x in big.items() if cc == c]
                if v and statistics.median(v) > 0:
                    scale[(path, c)] = calib_mib * 1024.0 / statistics.median(v)
        for name, grid, key, c, v in recs:
            if c not in counters:
                counters.append(c)
            rows.setdefault((name, grid), {}).setdefault(c, {})[(path,) + key] = v

    def med(ent, c):
        return statistics.median(ent[c].values()) if c in ent else None

    def scaled(ent, c):
        # bytes per dispatch: each run's median scaled by that run's copy
        per_run = {}
        for (path, _, _), v in ent.get(c, {}).items():
            per_run.setdefault(path, []).append(v)
        if not per_run or any((p, c) not in scale for p in per_run):
            return None
        return statistics.median([statistics.median(v) * 1024.0 * scale[(p, c)]
                                  for p, v in per_run.items()])

    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        fs = sorted({round(s, 3) for (p, cc), s in scale.items() if cc == c})
        if fs:
            print(f"{c} scale(s) from the {calib_mib} MiB copy: {', '.join(map(str, fs))}")
    has_bytes = any(c in counters for c in ("FETCH_SIZE", "WRITE_SIZE"))
    has_l2 = "TCC_HIT_sum" in counters and "TCC_MISS_sum" in counters
    head = ["kernel", "op", "grid (threads)", "dispatches"] + counters
    if has_bytes:
        head += ["scaled MB read", "scaled MB written", "total MB"]
    if has_l2:
        head += ["L2 hit %"]
    print("| " + " | ".join(head) + " |")
    print("|" + "---|" * len(head))
    for (name, grid), ent in sorted(rows.items(), key=lambda kv: (kernel_op(kv[0][0]), kv[0])):
        n = max(len(v) for v in ent.values())
        cells = [f"`{name}`", kernel_op(name), str(grid), str(n)]
        cells += ["" if med(ent, c) is None else f"{med(ent, c):.6g}" for c in counters]
        if has_bytes:
            rb, wb = scaled(ent, "FETCH_SIZE"), scaled(ent, "WRITE_SIZE")
            cells += ["" if rb is None else f"{rb / 1e6:.1f}", "" if wb is None else f"{wb / 1e6:.1f}",
                      "" if rb is None or wb is None else f"{(rb + wb) / 1e6:.1f}"]
        if has_l2:
            h, m = med(ent, "TCC_HIT_sum"), med(ent, "TCC_MISS_sum")
            cells += ["" if h is None or m is None or h + m == 0 else f"{100 * h / (h + m):.1f}"]
        print("| " + " | ".join(cells) + " |")


def kernel_op(kernel_name: str) -> str:
    """The library operation a kernel of this build serves (for trace tables)."""
    a = _template_args(kernel_name)
    if "project_weights_f32" in kernel_name and a[-1:] == ["true"]:
        return "factor_grad"                    # the strip kernel's factor-gradient mode
    for key, op in (("project_weights", "project_weights"), ("factor_grad_reduce", "factor_grad sum"),
                    ("factor_grad", "factor_grad"), ("reparam_backward_fused", "reparam backward (fused)"),
                    ("sum_partials", "range sum"), ("sparta", "sparta"), ("check_ids", "check_ids"),
                    ("pad_basis", "pad_basis"), ("copyBuffer", "device copy")):
        if key in kernel_name:
            return op
    if "decompress_f32" in kernel_name:
        # <KQ, HAS_E, GZ, SPAN>
        if a[2:3] == ["true"]:
            return "factored_embedding"
        return "decompress" if a[1:2] == ["true"] else "expand_grad"
    if "compress_f32" in kernel_name:
        # <KP, HAS_E, HAS_P, ...>
        if a[1:2] == ["true"]:
            return "compress"
        return "compress_projected" if a[2:3] == ["true"] else "project_grad"
    if "decompress" in kernel_name:
        if len(a) > 7 and a[7] == "true":
            return "factored_embedding"
        return "decompress" if a[1:2] == ["true"] else "expand_grad"
    if "compress_rows_bf16" in kernel_name or "compress_split_bf16" in kernel_name:
        if a[1:2] == ["true"]:
            return "compress"
        has_p = a[-1] == "true" if "compress_rows" in kernel_name else a[2:3] == ["true"]
        return "compress_projected" if has_p else "project_grad"
    if "compress_generic" in kernel_name:
        return "compress / project_grad (generic)"
    return "other"


def summarize_trace(trace_csv: str):
    """Markdown table of a rocprofv3 kernel trace: one row per kernel and
    grid (x, or x by y), sorted by total time; kernels outside this library
    (torch's input generation and copies) are left out."""
    import csv
    groups, total = {}, 0.0
    with open(trace_csv) as f:
        for r in csv.DictReader(f):
            us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            total += us
            name = r["Kernel_Name"]
            name = (name[5:] if name.startswith("void ") else name).split("(")[0]
            if not name.startswith("ssn::"):
                continue
            gy = r["Grid_Size_Y"]
            grid = r["Grid_Size_X"] if gy == "1" else f"{r['Grid_Size_X']}x{gy}"
            groups.setdefault((name, grid), []).append(us)
    print("| kernel | op | grid (threads, x or x by y) | calls | avg us | min us | max us | % time |")
    print("|---|---|---|---|---|---|---|---|")
    for (name, grid), ts in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{name}` | {kernel_op(name)} | {grid} | {len(ts)} | {sum(ts) / len(ts):.1f} | "
              f"{min(ts):.1f} | {max(ts):.1f} | {100 * sum(ts) / total:.2f} |")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(sample, cfg, seconds: float):
    """The float64 oracle on a bounded token sample, on this host's cores:
    BLAS threads set to the cores this process may run on."""
    from oracle import ssn_oracle as O
    cores = len(os.sched_getaffinity(0))

    def run(budget):
        n = sample["X"].shape[0]
        done, t0 = 0, time.perf_counter()
        while True:
            O.decompress(sample["Zin"], sample["ids"], sample["E"], sample["U"])
            O.project_grad(sample["G"], sample["U"])
            O.compress(sample["X"], sample["ids"], sample["E"], sample["U"])
            O.expand_grad(sample["GZin"], sample["U"])
            done += n
            el = time.perf_counter() - t0
            if el >= budget:
                return done, el

    try:
        from threadpoolctl import threadpool_limits
    except ImportError:
        threadpool_limits = None
    n = sample["X"].shape[0]
    if threadpool_limits is not None:
        with threadpool_limits(limits=cores):
            done, el = run(seconds)
    else:
        done, el = run(seconds)
    out = {"value": done / el, "unit": "tokens/s", "cores": cores, "kind": "oracle",
           "cpu_model": cpu_model(),
           "sample": f"{n} of the {cfg.N} tokens of one microbatch (d={cfg.d}, k={cfg.k}), "
                     f"all four codec ops in float64 with BLAS on {cores} threads, "
                     f"repeated {done // n}x over {el:.1f} s"}
    if threadpool_limits is not None:
        # the same oracle on one core, over a quarter of the time
        with threadpool_limits(limits=1):
            done1, el1 = run(seconds / 4)
        out["single_core_value"] = done1 / el1
    return out


def time_weights(wc, steps: int, dev, dtype: str = "bf16"):
    """W <- U (U^T W) over one stage's output projections, one batched launch,
    in the storage dtype `dtype` (bf16, or float32 master weights)."""
    import torch
    from paper_2607_13332_amd import inputs as I
    from paper_2607_13332_amd import ssn
    Ws = []
    for layer in range(wc.layers):
        for j, (dd, n) in enumerate(wc.shapes):
            Ws.append(I.weights_device(dd, n, wc.seed * 100 + 10 * layer + j, dev, dtype))
    Uw = I.to_device(I.store(I.gaussian_orthonormal_basis(wc.d, wc.k, wc.seed), dtype), dtype, dev)
    # a few untimed calls (the matrices were just written by the generator);
    # long back-to-back runs of this kernel drift slower on the box (power
    # management), which a once-per-optimizer-step operation never sees
    for _ in range(5):
        ssn.project_weights_batched(Ws, Uw)
    torch.cuda.synchronize()
    reps = 10
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record()
    for r in range(reps):       # back to back
        ssn.project_weights_batched(Ws, Uw)
        ev[r + 1].record()
    torch.cuda.synchronize()
    wms = sum(ev[r].elapsed_time(ev[r + 1]) for r in range(reps)) / reps
    # the same call after 20 ms of idle GPU, as once per optimizer step
    iso = []
    for r in range(5):
        time.sleep(0.02)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ssn.project_weights_batched(Ws, Uw)
        e1.record()
        torch.cuda.synchronize()
        iso.append(e0.elapsed_time(e1))
    iso_ms = sorted(iso)[len(iso) // 2]
    es = 2 if dtype == "bf16" else 4
    mfma_peak = MFMA_BF16_PEAK_TFLOPS if dtype == "bf16" else MFMA_F32_PEAK_TFLOPS
    wbytes = sum(2 * W.numel() * es for W in Ws) + wc.d * wc.k * es
    wflops = sum(4.0 * wc.d * wc.k * W.shape[1] for W in Ws)
    shapes = " + ".join(f"{a}x{b}" for a, b in wc.shapes)
    out = {
        "workload": f"W <- U(U^T W) for {wc.layers} layers x ({shapes}) {dtype}, k={wc.k}, one launch",
        "ms": round(wms, 5),
        "algorithmic_GBps": round(wbytes / (wms * 1e-3) / 1e9, 1),
        "frac_hbm_peak": round(wbytes / (wms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "mfma_TFLOPs": round(wflops / (wms * 1e-3) / 1e12, 2),
        "frac_mfma_peak": round(wflops / (wms * 1e-3) / 1e12 / mfma_peak, 4),
        "isolated_call": {"what": "median of 5 single calls, each after 20 ms of idle GPU",
                          "ms": round(iso_ms, 5),
                          "frac_hbm_peak": round(wbytes / (iso_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
    }
    if wc.name == I.WEIGHTS.name and dtype == "bf16":
        out["traffic"] = load_traffic("project_weights")
    if wc.k % 16 != 0:
        # U stored with zero columns up to whole 16-column tiles: the same
        # projection (the padding rows of U^T W are zero), aligned U paths
        kp = 16 * ((wc.k + 15) // 16)
        Up = torch.zeros((wc.d, kp), dtype=Uw.dtype, device=dev)
        Up[:, :wc.k] = Uw
        for _ in range(5):
            ssn.project_weights_batched(Ws, Up)
        ev[0].record()
        for r in range(reps):
            ssn.project_weights_batched(Ws, Up)
            ev[r + 1].record()
        torch.cuda.synchronize()
        pms = sum(ev[r].elapsed_time(ev[r + 1]) for r in range(reps)) / reps
        out["padded_basis"] = {"what": f"U stored zero-padded to {kp} columns", "ms": round(pms, 5),
                               "frac_hbm_peak": round(wbytes / (pms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        del Up
    del Ws
    torch.cuda.empty_cache()
    return out


def time_reparam(N: int, din: int, d: int, k: int, steps: int, dev, seed: int = 1040,
                 pad_to: int = 0, dtype: str = "bf16"):
    """Reparameterized-SSN projection of one layer: forward (H Zp) U^T and the
    backward (G U, (G U) Zp^T, H^T (G U)), storage dtype `dtype` (bf16 or
    f32).  pad_to > k: Zp and U stored with zero columns up to pad_to (the
    same layer: the padding columns of T, G U and the factor gradient stay
    zero)."""
    import numpy as np
    import torch
    from paper_2607_13332_amd import inputs as I
    from paper_2607_13332_amd import ssn
    sdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    es = 2 if dtype == "bf16" else 4
    g = torch.Generator(device=dev).manual_seed(seed)
    H = torch.randn((N, din), generator=g, device=dev).to(sdt)
    G = torch.randn((N, d), generator=g, device=dev).to(sdt)
    Zp = (0.02 * torch.randn((din, k), generator=g, device=dev)).to(sdt)
    U = I.to_device(I.store(I.gaussian_orthonormal_basis(d, k, seed), dtype), dtype, dev)
    kalg = k
    if pad_to > k:
        Zq = torch.zeros((din, pad_to), dtype=sdt, device=dev)
        Uq = torch.zeros((d, pad_to), dtype=sdt, device=dev)
        Zq[:, :k] = Zp
        Uq[:, :k] = U
        Zp, U, k = Zq, Uq, pad_to
    T = torch.empty((N, k), dtype=torch.float32, device=dev)
    Y = torch.empty((N, d), dtype=sdt, device=dev)
    GT = torch.empty((N, k), dtype=torch.float32, device=dev)
    GH = torch.empty((N, din), dtype=sdt, device=dev)
    GZ = torch.empty((din, k), dtype=torch.float32, device=dev)
    ws = torch.empty((max(4, ssn.reparam_workspace_bytes(dtype, N, din, k)) + 3) // 4,
                     dtype=torch.float32, device=dev)
    for _ in range(3):
        ssn.reparam_forward(H, Zp, U, T, Y)
        ssn.reparam_backward(H, Zp, U, G, GT, GH, GZ, ws)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record()
        ssn.reparam_forward(H, Zp, U, T, Y)
        ev[i][1].record()
        ssn.reparam_backward(H, Zp, U, G, GT, GH, GZ, ws)
        ev[i][2].record()
    torch.cuda.synchronize()
    fwd = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    bwd = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    fb = es * N * din + es * N * d + 8.0 * N * kalg + es * (din + d) * kalg
    bb = es * N * d + 2 * es * N * din + 12.0 * N * kalg + es * (din + d) * kalg + 4.0 * din * kalg
    pad = f", stored zero-padded to {k} columns" if k != kalg else ""
    out = {"workload": f"one projection layer: H [{N}, {din}], Zp [{din}, {kalg}], "
                       f"U [{d}, {kalg}]{pad}, {dtype}",
           "forward_ms": round(fwd, 5),
           "forward_frac_hbm_peak": round(fb / (fwd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "backward_ms": round(bwd, 5),
           "backward_frac_hbm_peak": round(bb / (bwd * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "tokens_per_s_fwd_bwd": round(N / ((fwd + bwd) * 1e-3), 1)}
    del H, G, Zp, U, T, Y, GT, GH, GZ, ws
    torch.cuda.empty_cache()
    return out


def time_sparta(cfg, steps: int, dev):
    """One sparse-averaging round over a block of float32 master weights
    (section 4.2): snapshot, the reducer's average with per-sender deltas,
    the receive step (buffer += delta) and the delta rule, for a rotating
    segment and for a sorted random index set of the same size."""
    import torch
    from paper_2607_13332_amd import inputs as I
    from paper_2607_13332_amd import ssn
    m, R = cfg.m, cfg.R
    theta = I.sparta_replica_device(cfg.n, cfg.seed, dev)
    first, _ = ssn.sparta_segment(cfg.n, 7)
    Ilist = I.sparta_positions_device(cfg.n, m, cfg.seed, dev)
    snap = torch.empty(m, dtype=torch.float32, device=dev)
    ssn.sparta_snapshot(theta, first=first, m=m, out=snap)
    chunks = I.sparta_chunks_device(snap, R, cfg.seed)
    acc = torch.empty(m, dtype=torch.float32, device=dev)
    deltas = [torch.empty(m, dtype=torch.float32, device=dev) for _ in range(R)]
    w = [1.0] * R
    ops = {
        "snapshot_segment": (lambda: ssn.sparta_snapshot(theta, first=first, m=m, out=snap), 8 * m),
        "snapshot_list": (lambda: ssn.sparta_snapshot(theta, I=Ilist, out=snap), 16 * m),
        "average": (lambda: ssn.sparta_average(chunks, w, acc=acc, deltas=deltas), 4 * m * (2 * R + 1)),
        "receive_segment": (lambda: ssn.delta_rule(theta, deltas[0], None, first=first), 12 * m),
        "apply_segment": (lambda: ssn.delta_rule(theta, acc, snap, first=first), 16 * m),
        "apply_list": (lambda: ssn.delta_rule(theta, acc, snap, I=Ilist), 24 * m),
    }
    reps = max(10, steps)
    out = {"workload": f"{cfg.n / 1e6:.0f}M float32 parameters, p = 1/{cfg.segments} "
                       f"({m / 1e6:.0f}M per round), {R} senders",
           "per_op": {}}
    total = 0.0
    for name, (fn, nbytes) in ops.items():
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        gbs = nbytes / (ms * 1e-3) / 1e9
        out["per_op"][name] = {"ms": round(ms, 5), "algorithmic_bytes": nbytes,
                               "algorithmic_GBps": round(gbs, 1),
                               "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
        if name in ("snapshot_segment", "average", "receive_segment", "apply_segment"):
            total += ms
    out["round_segment_ms"] = round(total, 5)
    del theta, Ilist, snap, chunks, acc, deltas
    torch.cuda.empty_cache()
    return out


def time_step_graph(sets, step_fn, steps: int, warmup: int) -> float:
    """ms per step when each input set's step is captured once as a HIP graph
    and replayed (the library launches kernels only: no allocation, no
    memset, so a whole step captures).  The untimed replays let the clocks
    settle again after the idle time of the capture."""
    import torch
    graphs = []
    for s in sets:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step_fn(s)
        graphs.append(g)
    for i in range(max(warmup, len(graphs))):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        graphs[i % len(graphs)].replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del graphs
    return ms


def time_codec_config(cfg, steps: int, warmup: int, dev):
    """The four codec ops of one microbatch on a workload other than the
    headline one.  Input sets rotate over at least 1 GiB (at least two sets)
    so that neither the step nor the per-op timing finds its inputs in the
    256 MB Infinity Cache.  The step is timed with no event inside it; the
    per-op times come from back-to-back calls of one op over the rotating
    sets.  For k % 16 != 0 the basis is the zero-padded copy made once by
    ssn_pad_basis (the library's layout for such ranks); the same step on the
    unpadded basis is reported beside it."""
    import numpy as np
    import torch
    from paper_2607_13332_amd import inputs as I
    from paper_2607_13332_amd import ssn
    N, d, k = cfg.N, cfg.d, cfg.k
    es = 2 if cfg.dtype == "bf16" else 4
    act = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    base = I.codec_inputs_device(cfg, dev, need=("U", "E"))
    U, E = base["U"], base["E"]
    # X, G, Y, G_X and the embedding rows of decompress and compress
    set_bytes = 6 * N * d * es
    nsets = min(24, max(2, -(-(1 << 30) // set_bytes)))
    sets = []
    for j in range(nsets):
        c = I.with_tokens(cfg, N, seed=cfg.seed + 17 * j)
        inp = I.codec_inputs_device(c, dev, need=("ids", "X", "G"))
        inp["Zin"] = I.coords_device(N, k, c.seed + 1, dev)
        inp["GZin"] = I.coords_device(N, k, c.seed + 2, dev)
        inp["Z"] = torch.empty((N, k), dtype=torch.float32, device=dev)
        inp["GZ"] = torch.empty((N, k), dtype=torch.float32, device=dev)
        inp["Y"] = torch.empty((N, d), dtype=act, device=dev)
        inp["GX"] = torch.empty((N, d), dtype=act, device=dev)
        inp["ids_c"] = I.codec_inputs_device(I.with_tokens(cfg, N, seed=c.seed + 7), dev,
                                             need=("ids",))["ids"]
        inp["u"] = int(torch.unique(inp["ids"]).numel())
        inp["u_c"] = int(torch.unique(inp["ids_c"]).numel())
        sets.append(inp)
    ops = ["decompress", "project_grad", "compress", "expand_grad"]
    # the gradient projection takes its range split through a workspace
    # allocated once per basis width (None where the split does not pay)
    wsp = {}

    def ws_for(Ub, split=True):
        w = Ub.shape[1]
        if not split:
            return None
        if w not in wsp:
            wsp[w] = ssn.project_grad_workspace(N, d, k, dev, ldu=w, dtype=act)
        return wsp[w]

    def step(s, Ub, evs=None, split=True):
        if evs:
            evs[0].record()
        ssn.decompress(s["Zin"], s["ids"], E, Ub, out=s["Y"])
        if evs:
            evs[1].record()
        ssn.project_grad(s["G"], Ub, out=s["GZ"], k=k, workspace=ws_for(Ub, split))
        if evs:
            evs[2].record()
        ssn.compress(s["X"], s["ids_c"], E, Ub, out=s["Z"], k=k)
        if evs:
            evs[3].record()
        ssn.expand_grad(s["GZin"], Ub, out=s["GX"])
        if evs:
            evs[4].record()

    def measure(Ub, split=True):
        """(ms per step, per-op mean ms) on basis Ub."""
        for i in range(warmup):
            step(sets[i % nsets], Ub, split=split)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            step(sets[i % nsets], Ub, split=split)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        # per-op times: R back-to-back calls of one op (rotating input sets)
        # queued behind a ~1 ms spin kernel, one event pair around them, so
        # the GPU runs them without waiting for the host between launches (at
        # these sizes a kernel takes about as long as its launch from
        # Python); the time per call includes the dispatch gap between
        # dependent kernels
        R = max(20, nsets)
        calls = {
            "decompress": lambda s: ssn.decompress(s["Zin"], s["ids"], E, Ub, out=s["Y"]),
            "project_grad": lambda s: ssn.project_grad(s["G"], Ub, out=s["GZ"], k=k,
                                                       workspace=ws_for(Ub, split)),
            "compress": lambda s: ssn.compress(s["X"], s["ids_c"], E, Ub, out=s["Z"], k=k),
            "expand_grad": lambda s: ssn.expand_grad(s["GZin"], Ub, out=s["GX"]),
        }
        op_ms = {}
        for op in ops:
            ts = []
            for rep in range(max(3, steps // 10)):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda._sleep(2_000_000)
                e0.record()
                for i in range(R):
                    calls[op](sets[i % nsets])
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) / R)
            op_ms[op] = float(np.median(ts))
        return ms, op_ms

    Ub, ldu, pad_ms = U, k, None
    if k % 16 != 0:
        ldu = 16 * ((k + 15) // 16)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        Ub = ssn.pad_basis(U, ldu)
        e1.record()
        torch.cuda.synchronize()
        pad_ms = e0.elapsed_time(e1)
    ms, op_ms = measure(Ub)
    per_op = {}
    step_bytes = 0
    for op in ops:
        t = op_ms[op]
        byts = float(np.mean([algorithmic_bytes(op, N, d, k, op_u(op, s), es) for s in sets]))
        step_bytes += byts
        per_op[op] = {"ms": round(t, 5), "algorithmic_GBps": round(byts / (t * 1e-3) / 1e9, 1),
                      "frac_hbm_peak": round(byts / (t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    gms = time_step_graph(sets, lambda s: step(s, Ub), steps, warmup)
    # the same step with compress against the projected table P = E U (the
    # NEXT form of section 4.1: E and U are fixed, so P is formed once)
    P = ssn.project_table(E, U)

    def step_projected(s):
        ssn.decompress(s["Zin"], s["ids"], E, Ub, out=s["Y"])
        ssn.project_grad(s["G"], Ub, out=s["GZ"], k=k, workspace=ws_for(Ub))
        ssn.compress_projected(s["X"], s["ids_c"], P, Ub, out=s["Z"])
        ssn.expand_grad(s["GZin"], Ub, out=s["GX"])

    for i in range(warmup):
        step_projected(sets[i % nsets])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step_projected(sets[i % nsets])
    torch.cuda.synchronize()
    pms = (time.perf_counter() - t0) * 1e3 / steps
    basis = f"U [{d}, {k}] stored zero-padded to {ldu} columns (ssn_pad_basis, once per basis)" \
        if ldu != k else f"U [{d}, {k}]"
    out = {"workload": f"N={N} (B={cfg.B} x S={cfg.S}), d={d}, k={k}, V={cfg.V}, {cfg.dtype}, "
                       f"{cfg.ids_dist} ids",
           "basis": basis,
           "input_sets": f"{nsets} rotating sets, {nsets * set_bytes / 2**30:.2f} GiB "
                         "(per-op times: back-to-back calls over the same rotation)",
           "ms_per_step": round(ms, 5), "tokens_per_s": round(N / (ms * 1e-3), 1),
           "step_frac_hbm_peak": round(step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "ms_per_step_hip_graph": round(gms, 5),
           "tokens_per_s_hip_graph": round(N / (gms * 1e-3), 1),
           "per_op": per_op,
           "step_with_projected_compress": {
               "what": "the same step with compress as X U - P[ids], P = E U [V, k] float32 formed once",
               "ms_per_step": round(pms, 5), "tokens_per_s": round(N / (pms * 1e-3), 1)}}
    wsb = wsp.get(Ub.shape[1])
    out["project_grad_entry"] = (
        f"ssn_project_grad_ws: d split into ranges through a {wsb.numel() / 2**20:.1f} MiB workspace "
        "allocated once" if wsb is not None else "ssn_project_grad_ex (no range split at this shape)")
    if wsb is not None:
        # the same step with the gradient projection in one launch, no workspace
        nms, nop = measure(Ub, split=False)
        out["without_range_split"] = {"ms_per_step": round(nms, 5),
                                      "project_grad_ms": round(nop["project_grad"], 5)}
    if pad_ms is not None:
        out["pad_basis_ms"] = round(pad_ms, 5)
        ums, uop = measure(U)
        out["unpadded_basis"] = {
            "what": f"the same step on U [{d}, {k}] as stored (k % 16 != 0: odd-width U rows)",
            "ms_per_step": round(ums, 5), "tokens_per_s": round(N / (ums * 1e-3), 1),
            "per_op_ms": {op: round(v, 5) for op, v in uop.items()}}
    del sets, base, U, E, Ub, P, wsp
    torch.cuda.empty_cache()
    return out


def copy_calibration(mib: int, dev):
    """A plain device copy of known size, three times (scales rocprofv3's
    FETCH_SIZE / WRITE_SIZE counters to bytes)."""
    import torch
    src = torch.empty(mib << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def copy_rate(dev, mib: int = 512, reps: int = 20) -> float:
    """GB/s (bytes read + written) of a plain device copy of `mib` MiB: the
    practical streaming rate that the HBM-bound kernels are compared with."""
    import torch
    src = torch.empty(mib << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2.0 * (mib << 20) / (ms * 1e-3) / 1e9


def run_section(name: str, args, dev):
    from paper_2607_13332_amd import inputs as I
    keep = {int(x) for x in args.sweep_tokens.split(",") if x.strip()}
    names = {x.strip() for x in args.select.split(",") if x.strip()}

    def kept(nm, n):
        return (not keep or n in keep) and (not names or nm in names)

    if name in ("sweep", "paper"):
        cfgs = ([c for c in I.sweep_configs() if c.k == 64] if name == "sweep" else I.paper_configs())
        return {c.name: time_codec_config(c, max(10, args.steps // 2), args.warmup, dev)
                for c in cfgs if kept(c.name, c.N)}
    if name == "f32":
        # float32 storage (activations, embedding, basis) on the matrix cores
        cfgs = [dataclasses.replace(I.STAGE8B, dtype="f32", name="stage8b_f32")] + \
               [dataclasses.replace(c, dtype="f32", name=c.name + "_f32") for c in I.paper_configs()
                if c.B == 1]
        out = {c.name: time_codec_config(c, max(10, args.steps // 2), args.warmup, dev)
               for c in cfgs if kept(c.name, c.N)}
        if not names or "paper8b_mlp_out_f32" in names:
            out["paper8b_mlp_out_f32"] = time_reparam(4096, 18432, 5120, 51, max(10, args.steps // 2), dev,
                                                      dtype="f32")
        return out
    if name == "weights":
        return {wc.name + ("" if dt == "bf16" else "_f32"): time_weights(wc, args.steps, dev, dt)
                for wc in (I.WEIGHTS, I.WEIGHTS_PAPER8B, I.WEIGHTS_PAPER1B) for dt in ("bf16", "f32")
                if not names or wc.name in names}
    if name == "reparam":
        steps = max(10, args.steps // 2)
        shapes = (("paper8b_mlp_out", (4096, 18432, 5120, 51), {}),
                  ("paper8b_mlp_out_padded64", (4096, 18432, 5120, 51), {"pad_to": 64}),
                  ("stage8b_mlp_out", (32768, 14336, 4096, 64), {}))
        return {nm: time_reparam(*shape, steps, dev, **kw) for nm, shape, kw in shapes
                if kept(nm, shape[0])}
    return time_sparta(I.SPARTA_BLOCK8B, args.steps, dev)


def main():
    args = parse_args()
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.copy_calib or 256)
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the codec shards over tokens with no exchange; see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_13332_amd import inputs as I
    from paper_2607_13332_amd import ssn

    ssn.lib()   # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.only:
        if args.copy_calib:
            copy_calibration(args.copy_calib, dev)
        print(json.dumps({"section": args.only, args.only: run_section(args.only, args, dev)}),
              flush=True)
        return
    cfg = I.STAGE8B if args.tokens == 0 else I.with_tokens(I.STAGE8B, args.tokens)
    N, d, k, V = cfg.N, cfg.d, cfg.k, cfg.V

    # ---------------- inputs, resident in HBM ----------------
    base = I.codec_inputs_device(cfg, dev, need=("U", "E"))
    U, E = base["U"], base["E"]
    # X, G, Y, G_X and the embedding rows of decompress and compress
    set_bytes = 6 * N * d * 2
    nsets = min(24, max(2, -(-(1 << 30) // set_bytes)))
    sets = []
    for j in range(nsets):
        c = I.with_tokens(cfg, N, seed=cfg.seed + 17 * j)
        inp = I.codec_inputs_device(c, dev, need=("ids", "X", "G"))
        inp["Zin"] = I.coords_device(N, k, c.seed + 1, dev)
        inp["GZin"] = I.coords_device(N, k, c.seed + 2, dev)
        inp["Z"] = torch.empty((N, k), dtype=torch.float32, device=dev)
        inp["GZ"] = torch.empty((N, k), dtype=torch.float32, device=dev)
        inp["Y"] = torch.empty((N, d), dtype=torch.bfloat16, device=dev)
        inp["GX"] = torch.empty((N, d), dtype=torch.bfloat16, device=dev)
        inp["ids_c"] = I.codec_inputs_device(I.with_tokens(cfg, N, seed=c.seed + 7), dev,
                                             need=("ids",))["ids"]
        inp["u"] = int(torch.unique(inp["ids"]).numel())
        inp["u_c"] = int(torch.unique(inp["ids_c"]).numel())
        sets.append(inp)
    torch.cuda.synchronize()

    ops = ["decompress", "project_grad", "compress", "expand_grad"]

    def step(s, evs=None):
        if evs is not None:
            evs[0].record()
        ssn.decompress(s["Zin"], s["ids"], E, U, out=s["Y"])
        if evs is not None:
            evs[1].record()
        ssn.project_grad(s["G"], U, out=s["GZ"])
        if evs is not None:
            evs[2].record()
        ssn.compress(s["X"], s["ids_c"], E, U, out=s["Z"])
        if evs is not None:
            evs[3].record()
        ssn.expand_grad(s["GZin"], U, out=s["GX"])
        if evs is not None:
            evs[4].record()

    if args.copy_calib:
        copy_calibration(args.copy_calib, dev)

    # untimed: the clock ramp of an idle GPU, then the warmup steps
    t_settle = time.perf_counter() + max(0.0, args.settle_seconds)
    while time.perf_counter() < t_settle:
        for i in range(64):
            step(sets[i % 2])
        torch.cuda.synchronize()
    for i in range(args.warmup):
        step(sets[i % 2])
    torch.cuda.synchronize()

    def op_stats(evs, names):
        out = {}
        for j, op in enumerate(names):
            ts = np.array([e[j].elapsed_time(e[j + 1]) for e in evs])
            out[op] = (float(ts.mean()), np.percentile(ts, [10, 50, 90]))
        return out

    def per_op_entry(op, mean_ms, pct):
        byts = np.mean([algorithmic_bytes(op, N, d, k, op_u(op, s)) for s in sets])
        return {"ms": round(mean_ms, 5),
                "ms_p10_p50_p90": [round(float(x), 5) for x in pct],
                "tokens_per_s": round(N / (mean_ms * 1e-3), 1),
                "algorithmic_GBps": round(byts / (mean_ms * 1e-3) / 1e9, 1),
                "frac_hbm_peak": round(byts / (mean_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                "bytes_per_launch": int(byts)}

    # per-op breakdown: a pass with HIP events around every op (events
    # between kernels cost the step time, so this pass is not the timed one)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(sets[i % 2], events[i])
    torch.cuda.synchronize()
    stats = op_stats(events, ops)
    dom = max(ops, key=lambda o: stats[o][0])

    # ---------------- timed region ----------------
    # the step as a caller runs it; the only events are the pair around the
    # dominant kernel, on the stream it is launched on, for the roofline, on
    # every DOM_EVERY-th step (an event between two kernels idles the GPU for
    # a few microseconds, which a caller's step does not pay)
    DOM_EVERY = 4
    dom_j = ops.index(dom)
    dev_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)]
              for _ in range(0, args.steps, DOM_EVERY)]

    def timed_step(s, ev):
        for j, fn in enumerate((lambda: ssn.decompress(s["Zin"], s["ids"], E, U, out=s["Y"]),
                                lambda: ssn.project_grad(s["G"], U, out=s["GZ"]),
                                lambda: ssn.compress(s["X"], s["ids_c"], E, U, out=s["Z"]),
                                lambda: ssn.expand_grad(s["GZin"], U, out=s["GX"]))):
            if j == dom_j and ev is not None:
                ev[0].record()
                fn()
                ev[1].record()
            else:
                fn()

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        timed_step(sets[i % 2], dev_ev[i // DOM_EVERY] if i % DOM_EVERY == 0 else None)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    dom_ts = np.array([e[0].elapsed_time(e[1]) for e in dev_ev])

    per_op = {op: per_op_entry(op, *stats[op]) for op in ops}
    # HBM bytes measured by the rocprofv3 counters (when taken on these
    # sources) over the same mean durations
    measured = {op: load_traffic(op) for op in ops}
    for op in ops:
        if measured[op] is not None:
            gbs = measured[op] / (stats[op][0] * 1e-3) / 1e9
            per_op[op]["measured_traffic_GBps"] = round(gbs, 1)
            per_op[op]["measured_frac_hbm_peak"] = round(gbs / HBM_PEAK_GBS, 4)
    # the roofline's duration: the dominant kernel inside the timed region
    dom_entry = per_op_entry(dom, float(dom_ts.mean()), np.percentile(dom_ts, [10, 50, 90]))
    achieved = dom_entry["algorithmic_GBps"]
    traffic = load_traffic(dom)
    step_bytes = sum(per_op[o]["bytes_per_launch"] for o in ops)

    result = {
        "metric": "codec tokens/s at d=4096,k=64 bf16 + achieved HBM GB/s as % of peak",
        "value": round(N / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "stage-boundary codec of an 8B-shaped pipeline stage: "
                               "decompress + project_grad + compress + expand_grad per microbatch",
                   "N": N, "B": cfg.B, "S": cfg.S, "d": d, "k": k, "V": V, "ids": cfg.ids_dist,
                   "storage": "bf16", "coords": "fp32", "parallelism": "none (1 GPU)"},
        "step_algorithmic_GBps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "step_frac_hbm_peak": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "step_measured_frac_hbm_peak": (
            None if any(v is None for v in measured.values()) else
            round(sum(measured.values()) / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)),
        "per_op": per_op,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "ms": dom_entry["ms"],
                     "ms_p10_p50_p90": dom_entry["ms_p10_p50_p90"],
                     "bytes_per_launch": dom_entry["bytes_per_launch"],
                     "timed_launches": f"{len(dev_ev)} of the {args.steps} timed steps "
                                       f"(every {DOM_EVERY}th)"},
        "kernel_source_hash": kernel_source_hash(),
    }
    # (not in the counter runs: their copy of known size is the calibration)
    cp_rate = None if args.copy_calib else copy_rate(dev)
    if cp_rate is not None:
        result["hbm_copy_reference"] = {
            "what": "torch device copy of 512 MiB on the same GPU, bytes read + written per second",
            "GBps": round(cp_rate, 1), "frac_hbm_peak": round(cp_rate / HBM_PEAK_GBS, 4),
            "dominant_kernel_frac_of_copy": round(achieved / cp_rate, 4)}

    def time_variant(fn):
        """ms per step with no event inside the step, then per-op stats from
        a pass with events around every op."""
        for i in range(args.warmup):
            fn(sets[i % 2], None)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            fn(sets[i % 2], None)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
        for i in range(args.steps):
            fn(sets[i % 2], evs[i])
        torch.cuda.synchronize()
        return ms, evs

    def rec(evs, j):
        if evs is not None:
            evs[j].record()

    # ---------------- variant: compress against the projected table ----------------
    tev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    tev[0].record()
    P = ssn.project_table(E, U)
    tev[1].record()
    torch.cuda.synchronize()
    P = ssn.project_table(E, U)
    ops2 = ["decompress", "project_grad", "compress_projected", "expand_grad"]

    def step2(s, evs):
        rec(evs, 0)
        ssn.decompress(s["Zin"], s["ids"], E, U, out=s["Y"])
        rec(evs, 1)
        ssn.project_grad(s["G"], U, out=s["GZ"])
        rec(evs, 2)
        ssn.compress_projected(s["X"], s["ids_c"], P, U, out=s["Z"])
        rec(evs, 3)
        ssn.expand_grad(s["GZin"], U, out=s["GX"])
        rec(evs, 4)

    ms2, ev2 = time_variant(step2)
    st2 = op_stats(ev2, ops2)
    cp = per_op_entry("compress_projected", *st2["compress_projected"])
    cp["traffic"] = load_traffic("compress_projected")
    result["variants"] = {
        "compress_projected": cp,
        "table_build": {"what": f"P = E U over all V={V} rows ({V * k * 4 / 1e6:.1f} MB fp32), "
                                "once per basis / embedding change",
                        "ms": round(tev[0].elapsed_time(tev[1]), 5)},
        "step_with_projected_compress": {"ms_per_step": round(ms2, 5),
                                         "tokens_per_s": round(N / (ms2 * 1e-3), 1)},
    }
    # ---------------- variant: coordinates on the wire in bf16 ----------------
    for s_ in sets:
        s_["Zin_b"] = s_["Zin"].to(torch.bfloat16)
        s_["GZin_b"] = s_["GZin"].to(torch.bfloat16)
        s_["Z_b"] = torch.empty((N, k), dtype=torch.bfloat16, device=dev)
        s_["GZ_b"] = torch.empty((N, k), dtype=torch.bfloat16, device=dev)

    def step3(s, evs):
        rec(evs, 0)
        ssn.decompress(s["Zin_b"], s["ids"], E, U, out=s["Y"])
        rec(evs, 1)
        ssn.project_grad(s["G"], U, out=s["GZ_b"], z_dtype=torch.bfloat16)
        rec(evs, 2)
        ssn.compress(s["X"], s["ids_c"], E, U, out=s["Z_b"], z_dtype=torch.bfloat16)
        rec(evs, 3)
        ssn.expand_grad(s["GZin_b"], U, out=s["GX"])
        rec(evs, 4)

    ms3, ev3 = time_variant(step3)
    st3 = op_stats(ev3, ops)
    result["variants"]["step_bf16_coordinates"] = {
        "what": "the same four ops with Z and G_Z in bf16 (half the wire message)",
        "ms_per_step": round(ms3, 5), "tokens_per_s": round(N / (ms3 * 1e-3), 1),
        "per_op_ms": {op: round(st3[op][0], 5) for op in ops}}
    for s_ in sets:
        for key in ("Zin_b", "GZin_b", "Z_b", "GZ_b"):
            del s_[key]

    gms = time_step_graph(sets, step, args.steps, args.warmup)
    result["variants"]["step_hip_graph"] = {
        "what": "the same four ops captured once per input set as a HIP graph and replayed",
        "ms_per_step": round(gms, 5), "tokens_per_s": round(N / (gms * 1e-3), 1),
        "frac_hbm_peak": round(step_bytes / (gms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "measured_frac_hbm_peak": (
            None if any(v is None for v in measured.values()) else
            round(sum(measured.values()) / (gms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4))}
    del P

    # ---------------- weight re-projection (once per optimizer step) ----------------
    if not args.no_weights:
        result["weights"] = time_weights(I.WEIGHTS, args.steps, dev)
        result["weights_f32"] = time_weights(I.WEIGHTS, args.steps, dev, "f32")

    # ---------------- sweep points at k = 64 (Zipf ids) ----------------
    if not args.no_sweep:
        result["sweep_k64"] = {c.name: time_codec_config(c, max(10, args.steps // 2), args.warmup, dev)
                               for c in I.sweep_configs() if c.k == 64}

    # ---------------- the paper's own shapes ----------------
    if not args.no_paper_shapes:
        shapes = {}
        for pc in I.paper_configs():
            shapes[pc.name] = time_codec_config(pc, max(10, args.steps // 2), args.warmup, dev)
        for wc in (I.WEIGHTS_PAPER8B, I.WEIGHTS_PAPER1B):
            shapes[wc.name] = time_weights(wc, args.steps, dev)
        result["paper_shapes"] = shapes

    # ---------------- reparameterized-SSN projections (section 4.1, Eq. (3)) ----------------
    if not args.no_reparam:
        result["reparam"] = run_section("reparam", args, dev)

    # ---------------- sparse averaging with the delta rule (section 4.2) ----------------
    if not args.no_sparta:
        result["sparta"] = run_section("sparta", args, dev)

    # ---------------- CPU baseline: the oracle on a bounded sample ----------------
    if not args.no_cpu_baseline:
        s = sets[0]
        ns = min(N, 2048)
        rows = torch.arange(ns, device=dev)
        sample = {
            "X": I.to_host(s["X"][rows]), "G": I.to_host(s["G"][rows]),
            "Zin": I.to_host(s["Zin"][rows]), "GZin": I.to_host(s["GZin"][rows]),
            "E": I.to_host(E.index_select(0, s["ids"][rows].long())),
            "ids": np.arange(ns, dtype=np.int32), "U": I.to_host(U),
        }
        result["cpu_baseline"] = cpu_baseline(sample, cfg, args.cpu_seconds)

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
