"""HIP graph capture of the whole path: every entry point only enqueues
kernels (no allocation, no memset, no host synchronisation), so a step
captures into one graph.  Each replay, with fresh inputs copied in eagerly
between replays, must equal an eager run on the same inputs bit for bit (the
kernels are deterministic)."""
import numpy as np
import pytest
import torch

from paper_2607_13332_amd import inputs as I
from paper_2607_13332_amd import ssn

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _codec_inputs(N, d, k, V, seed, dtype="bf16"):
    cfg = I.CodecConfig("graph", B=1, S=N, d=d, k=k, V=V, dtype=dtype, seed=seed, structured=False)
    h = I.codec_inputs_device(cfg, DEV)
    h["Zin"] = I.coords_device(N, k, seed + 1, DEV)
    h["GZin"] = I.coords_device(N, k, seed + 2, DEV)
    return h


@pytest.mark.parametrize("N,d,k,dtype", [(4096, 5120, 51, "bf16"), (2048, 4096, 64, "bf16"),
                                         (4096, 5120, 51, "f32"), (20000, 1024, 64, "f32")])
def test_codec_step_replays_match_eager(N, d, k, dtype):
    V = 4096
    print(f"[graph] codec N={N} d={d} k={k} {dtype}", flush=True)
    act = torch.bfloat16 if dtype == "bf16" else torch.float32
    static = _codec_inputs(N, d, k, V, 7000, dtype)
    outs = {"Y": torch.empty((N, d), dtype=act, device=DEV),
            "GZ": torch.empty((N, k), device=DEV), "Z": torch.empty((N, k), device=DEV),
            "GX": torch.empty((N, d), dtype=act, device=DEV)}

    def step(s, o):
        ssn.decompress(s["Zin"], s["ids"], s["E"], s["U"], out=o["Y"])
        ssn.project_grad(s["G"], s["U"], out=o["GZ"])
        ssn.compress(s["X"], s["ids"], s["E"], s["U"], out=o["Z"])
        ssn.expand_grad(s["GZin"], s["U"], out=o["GX"])

    step(static, outs)                       # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(static, outs)
    for rep in range(3):
        fresh = _codec_inputs(N, d, k, V, 7100 + rep, dtype)
        for key in ("X", "G", "E", "U", "ids", "Zin", "GZin"):
            static[key].copy_(fresh[key])
        g.replay()
        got = {key: v.clone() for key, v in outs.items()}
        ref = {key: torch.empty_like(v) for key, v in outs.items()}
        step(static, ref)                    # eager on the same inputs
        torch.cuda.synchronize()
        for key in outs:
            assert torch.equal(got[key], ref[key]), f"replay {rep}: {key} differs from eager"


def test_wire_formats_capture():
    """bf16 coordinates and a zero-padded basis (the _ex entry points) capture
    and replay like the plain step."""
    N, d, k, V, ldu = 4096, 5120, 51, 4096, 64
    print(f"[graph] bf16 coordinates, padded basis N={N} d={d} k={k} ldu={ldu}", flush=True)
    static = _codec_inputs(N, d, k, V, 7200)
    Up = torch.zeros((d, ldu), dtype=torch.bfloat16, device=DEV)
    Zb = static["Zin"].to(torch.bfloat16)
    outs = {"Y": torch.empty((N, d), dtype=torch.bfloat16, device=DEV),
            "GZ": torch.empty((N, k), dtype=torch.bfloat16, device=DEV),
            "Z": torch.empty((N, k), dtype=torch.bfloat16, device=DEV),
            "GX": torch.empty((N, d), dtype=torch.bfloat16, device=DEV),
            "GZw": torch.empty((N, k), device=DEV),
            "GZwb": torch.empty((N, k), dtype=torch.bfloat16, device=DEV)}
    # the range-split projection through the caller's workspace
    ws = ssn.project_grad_workspace(N, d, k, DEV, ldu=ldu)
    assert ws is not None

    def step(o):
        ssn.decompress(Zb, static["ids"], static["E"], Up, out=o["Y"])
        ssn.project_grad(static["G"], Up, out=o["GZ"], z_dtype=torch.bfloat16, k=k)
        ssn.compress(static["X"], static["ids"], static["E"], Up, out=o["Z"], z_dtype=torch.bfloat16, k=k)
        ssn.expand_grad(Zb, Up, out=o["GX"])
        ssn.project_grad(static["G"], Up, out=o["GZw"], k=k, workspace=ws)
        ssn.project_grad(static["G"], Up, out=o["GZwb"], z_dtype=torch.bfloat16, k=k, workspace=ws)

    Up[:, :k] = static["U"]
    step(outs)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(outs)
    for rep in range(3):
        fresh = _codec_inputs(N, d, k, V, 7300 + rep)
        for key in ("X", "G", "E", "ids"):
            static[key].copy_(fresh[key])
        Up[:, :k] = fresh["U"]
        Zb.copy_(fresh["Zin"].to(torch.bfloat16))
        g.replay()
        got = {key: v.clone() for key, v in outs.items()}
        ref = {key: torch.empty_like(v) for key, v in outs.items()}
        step(ref)
        torch.cuda.synchronize()
        for key in outs:
            assert torch.equal(got[key], ref[key]), f"replay {rep}: {key} differs from eager"
        assert torch.equal(got["GZwb"], got["GZw"].to(torch.bfloat16))


@pytest.mark.parametrize("N,din,d,k", [(1024, 2048, 1024, 51), (2048, 16384, 1024, 32)],
                         ids=["d_split_kernels", "row_ranges_and_fused_backward"])
def test_reparam_and_averaging_capture(N, din, d, k):
    """The reparameterized layer (forward + backward with its workspace) and
    a delta-rule round in one graph: the d-split projections with separate
    backward kernels (k = 51), and the row kernel over ranges of din with the
    fused backward pass (k = 32, whole tiles)."""
    g0 = torch.Generator(device=DEV).manual_seed(3)

    def draw():
        return {"H": torch.randn((N, din), generator=g0, device=DEV).to(torch.bfloat16),
                "G": torch.randn((N, d), generator=g0, device=DEV).to(torch.bfloat16),
                "Zp": (0.02 * torch.randn((din, k), generator=g0, device=DEV)).to(torch.bfloat16),
                "theta": torch.randn(100_000, generator=g0, device=DEV),
                "c1": torch.randn(5_000, generator=g0, device=DEV)}

    U = I.to_device(I.store(I.gaussian_orthonormal_basis(d, k, 5), "bf16"), "bf16", DEV)
    st = draw()
    ws = torch.empty((max(4, ssn.reparam_workspace_bytes("bf16", N, din, k)) + 3) // 4, device=DEV)

    def alloc():
        return {"T": torch.empty((N, k), device=DEV),
                "Y": torch.empty((N, d), dtype=torch.bfloat16, device=DEV),
                "GT": torch.empty((N, k), device=DEV),
                "GH": torch.empty((N, din), dtype=torch.bfloat16, device=DEV),
                "GZ": torch.empty((din, k), device=DEV),
                "snap": torch.empty(5_000, device=DEV), "acc": torch.empty(5_000, device=DEV),
                "d0": torch.empty(5_000, device=DEV), "d1": torch.empty(5_000, device=DEV),
                "theta": torch.empty(100_000, device=DEV)}

    def step(s, o):
        ssn.reparam_forward(s["H"], s["Zp"], U, o["T"], o["Y"])
        ssn.reparam_backward(s["H"], s["Zp"], U, s["G"], o["GT"], o["GH"], o["GZ"], ws)
        ssn.sparta_snapshot(s["theta"], first=0, m=100_000, out=o["theta"])   # plain copy
        ssn.sparta_snapshot(o["theta"], first=1_000, m=5_000, out=o["snap"])
        ssn.sparta_average([o["snap"], s["c1"]], [1.0, 3.0], acc=o["acc"], deltas=[o["d0"], o["d1"]])
        ssn.delta_rule(o["theta"], o["acc"], o["snap"], first=1_000)

    outs = alloc()
    step(st, outs)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(st, outs)
    for rep in range(3):
        fresh = draw()
        for key in st:
            st[key].copy_(fresh[key])
        g.replay()
        got = {key: v.clone() for key, v in outs.items()}
        ref = alloc()
        step(st, ref)
        torch.cuda.synchronize()
        for key in outs:
            assert torch.equal(got[key], ref[key]), f"replay {rep}: {key} differs from eager"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_weight_reprojection_capture(dtype):
    """The batched weight re-projection, in place, captured and replayed on
    fresh matrices: each replay equals an eager call on the same matrices."""
    d, k, ns = 2048, 48, (2048, 7168, 1000)
    print(f"[graph] weights d={d} k={k} n={ns} {dtype}", flush=True)
    U = I.to_device(I.store(I.gaussian_orthonormal_basis(d, k, 7400), dtype), dtype, DEV)
    Ws = [I.weights_device(d, n, 7400 + j, DEV, dtype) for j, n in enumerate(ns)]
    ssn.project_weights_batched(Ws, U)        # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ssn.project_weights_batched(Ws, U)
    for rep in range(3):
        fresh = [I.weights_device(d, n, 7500 + 10 * rep + j, DEV, dtype) for j, n in enumerate(ns)]
        for W, F in zip(Ws, fresh):
            W.copy_(F)
        g.replay()
        ref = [F.clone() for F in fresh]
        ssn.project_weights_batched(ref, U)   # eager on the same matrices
        torch.cuda.synchronize()
        for j, (W, R) in enumerate(zip(Ws, ref)):
            assert torch.equal(W, R), f"replay {rep}: matrix {j} differs from eager"
