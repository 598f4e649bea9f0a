"""GPU parity at tensor sizes past 2^31 elements (every kernel's row and
element offsets must be 64-bit), against the float64 oracle on sampled rows
or columns that always include the last ones and the rows around the 2^31
element boundary.

Each case allocates 4-20 GB of device memory (MI355X: 288 GB) and frees it.
"""
import numpy as np
import pytest
import torch

from helpers import (check, mag_compress, mag_decompress, mag_project, mag_reparam_forward,
                     mag_reparam_grad_factor, mag_reparam_grad_input, mag_weights, rel,
                     sample_rows)
from oracle import ssn_oracle as O
from paper_2607_13332_amd import inputs as I
from paper_2607_13332_amd import ssn

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TWO31 = 2 ** 31


def host(t):
    return I.to_host(t)


def boundary_rows(n_rows: int, row_len: int, count: int, seed: int) -> np.ndarray:
    """A seeded sample of rows plus the first rows, the last 256 rows and the
    rows whose elements straddle element 2^31."""
    b = TWO31 // row_len
    extra = [np.arange(4), np.arange(max(0, b - 8), min(n_rows, b + 8)),
             np.arange(max(0, n_rows - 256), n_rows)]
    return np.unique(np.concatenate([sample_rows(n_rows, count, seed)] + extra)).astype(np.int64)


@pytest.mark.timeout(600)
def test_codec_past_2_31_elements():
    """The four codec ops at N = 2^19 + 333 tokens, d = 4096, k = 64: X, G,
    X' and G_X hold 2.15e9 elements each."""
    cfg = I.with_tokens(I.STAGE8B, 2 ** 19 + 333, seed=1090)
    N, d, k = cfg.N, cfg.d, cfg.k
    assert N * d > TWO31
    print(f"[case] codec N={N} d={d} k={k}", flush=True)
    inp = I.codec_inputs_device(cfg, DEV)
    X, ids, E, U, G = inp["X"], inp["ids"], inp["E"], inp["U"], inp["G"]
    Zin = I.coords_device(N, k, cfg.seed, DEV)
    Z, GZ = ssn.compress(X, ids, E, U), ssn.project_grad(G, U)
    Y, GX = ssn.decompress(Zin, ids, E, U), ssn.expand_grad(Zin, U)
    torch.cuda.synchronize()
    rows = boundary_rows(N, d, 512, cfg.seed)
    r = torch.from_numpy(rows).to(DEV)
    Xs, Gs, Zs, Us = host(X[r]), host(G[r]), host(Zin[r]), host(U)
    Es = host(E.index_select(0, ids[r].long()))
    loc = np.arange(len(rows), dtype=np.int32)
    check("large compress", host(Z[r]), O.compress(Xs, loc, Es, Us), "bf16", "f32out",
          mag_compress(Xs, loc, Es, Us))
    check("large decompress", host(Y[r]), O.decompress(Zs, loc, Es, Us), "bf16", "bf16out",
          mag_decompress(Zs, loc, Es, Us))
    check("large project_grad", host(GZ[r]), O.project_grad(Gs, Us), "bf16", "f32out",
          mag_project(Gs, Us))
    check("large expand_grad", host(GX[r]), O.expand_grad(Zs, Us), "bf16", "bf16out",
          mag_decompress(Zs, None, None, Us))
    del inp, X, G, E, Y, GX, Z, GZ, Zin
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("n,dtype", [(2 ** 19 + 8, "bf16"), (2 ** 19 + 1, "bf16"), (2 ** 19 + 4, "f32")])
def test_weight_projection_past_2_31_elements(n, dtype):
    """W [4096, n] with 4096 n > 2^31, re-projected in place: in bf16, n % 8 ==
    0 runs the column-strip kernel and odd n the 64-column panel kernel; in
    float32 (8.6 GB) n % 4 == 0 runs the float32 column-strip kernel."""
    d, k = 4096, 64
    assert d * n > TWO31
    print(f"[case] weights d={d} n={n} k={k} {dtype} family="
          f"{ssn.kernel_family('project_weights', dtype, d, k)}", flush=True)
    U = I.to_device(I.store(I.gaussian_orthonormal_basis(d, k, 1091), dtype), dtype, DEV)
    W = I.weights_device(d, n, 1091, DEV, dtype)
    cols = boundary_rows(n, 1, 256, 1091)
    cols = np.unique(np.concatenate([cols, np.arange(n - 70, n)]))
    c = torch.from_numpy(cols).to(DEV)
    before = host(W[:, c])
    ssn.project_weights(W, U)
    torch.cuda.synchronize()
    Uh = host(U)
    check(f"large weights n={n} {dtype}", host(W[:, c]), O.project_weights(before, Uh), dtype,
          "bf16out" if dtype == "bf16" else "f32out", mag_weights(before, Uh))
    del W, U
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_reparam_layer_past_2_31_elements():
    """Forward and backward of the reparameterized layer with H and dL/dH of
    N din > 2^31 elements (N = 150016, din = 14336, d = 4096, k = 64)."""
    N, din, d, k = 150016, 14336, 4096, 64
    assert N * din > TWO31
    print(f"[case] reparam N={N} din={din} d={d} k={k}", flush=True)
    g = torch.Generator(device=DEV).manual_seed(1092)
    H = torch.randn((N, din), generator=g, device=DEV).to(torch.bfloat16)
    G = torch.randn((N, d), generator=g, device=DEV).to(torch.bfloat16)
    Zp = (0.02 * torch.randn((din, k), generator=g, device=DEV)).to(torch.bfloat16)
    U = I.to_device(I.store(I.gaussian_orthonormal_basis(d, k, 1092), "bf16"), "bf16", DEV)
    T, Y = ssn.reparam_forward(H, Zp, U)
    del T
    GT, GH, GZ = ssn.reparam_backward(H, Zp, U, G)
    torch.cuda.synchronize()
    rows = torch.from_numpy(boundary_rows(N, din, 128, 1092)).to(DEV)
    Hs, Gs, Zh, Uh = host(H[rows]), host(G[rows]), host(Zp), host(U)
    check("large reparam Y", host(Y[rows]), O.reparam_forward(Hs, Zh, Uh), "bf16", "bf16out",
          mag_reparam_forward(Hs, Zh, Uh))
    check("large reparam dL/dH", host(GH[rows]), O.reparam_grad_input(Gs, Zh, Uh), "bf16", "bf16out",
          mag_reparam_grad_input(Gs, Zh, Uh))
    # factor-gradient rows need every token: sampled columns of H, all of G
    cols = torch.from_numpy(np.unique(np.concatenate([sample_rows(din, 24, 3),
                                                      np.arange(din - 8, din)]))).to(DEV)
    Hc, Gall = host(H[:, cols].contiguous()), host(G)
    check("large reparam dL/dZp", host(GZ[cols]), O.reparam_grad_factor(Hc, Gall, Uh), "bf16", "f32out",
          mag_reparam_grad_factor(Hc, Gall, Uh))
    del H, G, Y, GT, GH, GZ
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("form", ["segment", "list"])
def test_averaging_round_past_2_31_parameters(form):
    """Snapshot, weighted average and delta rule on a parameter vector of
    2^31 + 4100 float32 values, at positions past 2^31: the last of 20
    rotating segments, or a sorted list that ends at the last parameter."""
    n = TWO31 + 4100
    print(f"[case] averaging n={n} form={form}", flush=True)
    theta0 = I.sparta_replica_device(n, 1093, DEV)
    if form == "segment":
        first, m = ssn.sparta_segment(n, 19)
        Idev = None
        pos = first + torch.arange(m, device=DEV, dtype=torch.int64)
    else:
        r = np.random.default_rng(1093)
        P = np.unique(np.concatenate([r.integers(0, n, size=1 << 20), [0, TWO31 - 1, TWO31, n - 1]]))
        Idev = torch.from_numpy(P.astype(np.int64)).to(DEV)
        first, m = 0, len(P)
        pos = Idev
    assert int(pos[-1]) == n - 1
    snap = ssn.sparta_snapshot(theta0, I=Idev, first=first, m=m)
    assert torch.equal(snap, theta0[pos])
    chunks = I.sparta_chunks_device(snap, 3, 1093)
    w = [1.0, 0.5, 2.0]
    acc, deltas = ssn.sparta_average(chunks, w)
    sample = torch.from_numpy(np.unique(np.concatenate([
        np.random.default_rng(7).integers(0, m, size=4096), np.arange(m - 64, m)]))).to(DEV)
    cs = [host(ch[sample]) for ch in chunks]
    ref_acc, ref_d = O.sparta_average(cs, w)
    assert rel(host(acc[sample]), ref_acc) <= 2e-6
    for j in range(3):
        assert np.linalg.norm(host(deltas[j][sample]) - ref_d[j]) / np.linalg.norm(ref_acc) <= 2e-6
    theta = theta0
    before_tail = host(theta[pos[sample]])
    ssn.delta_rule(theta, acc, snap, I=Idev, first=first)
    ref = O.delta_rule(before_tail, np.arange(len(before_tail)), host(acc[sample]), host(snap[sample]), 1.0)
    assert rel(host(theta[pos[sample]]), ref) <= 2e-7
    del theta0, theta, snap, chunks, acc, deltas, pos
    torch.cuda.empty_cache()
