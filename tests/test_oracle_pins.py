"""Pins for the float64 oracle, against facts fixed by the paper's definitions
(section 4.1, Eq. (2) and the original-SSN re-projection) and by mathematics:
exact rational brute force, closed forms, invariants and special bases.

Each pin is chosen so that a plausible slip in the oracle -- a dropped or
sign-flipped embedding term, a wrong gather index, a transposed basis, a
missing second factor in the weight projection -- fails at least one test.
"""
import json
import os

import numpy as np
import pytest

from oracle import exact
from oracle import ssn_oracle as O
from paper_2607_13332_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_case(dtype, N=5, d=12, k=3, V=7, n=4, seed=7):
    r = np.random.default_rng(seed)
    U = I.store(I.gaussian_orthonormal_basis(d, k, seed), dtype)
    E = I.store(0.3 * r.standard_normal((V, d)), dtype)
    X = I.store(r.standard_normal((N, d)), dtype)
    G = I.store(r.standard_normal((N, d)), dtype)
    W = I.store(r.standard_normal((d, n)), dtype)
    ids = r.integers(0, V, size=N).astype(np.int32)
    Z = r.standard_normal((N, k)).astype(np.float32)
    return dict(U=U, E=E, X=X, G=G, W=W, ids=ids, Z=Z)


def _rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# ---------------------------------------------------------------- brute force
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_exact_bruteforce_all_ops(dtype):
    c = _rand_case(dtype)
    assert _rel(O.compress(c["X"], c["ids"], c["E"], c["U"]),
                exact.to_float(exact.compress(c["X"], c["ids"], c["E"], c["U"]))) < 1e-14
    assert _rel(O.decompress(c["Z"], c["ids"], c["E"], c["U"]),
                exact.to_float(exact.decompress(c["Z"], c["ids"], c["E"], c["U"]))) < 1e-14
    assert _rel(O.expand_grad(c["Z"], c["U"]),
                exact.to_float(exact.decompress(c["Z"], None, None, c["U"]))) < 1e-14
    assert _rel(O.project_grad(c["G"], c["U"]),
                exact.to_float(exact.project_grad(c["G"], c["U"]))) < 1e-14
    assert _rel(O.project_weights(c["W"], c["U"]),
                exact.to_float(exact.project_weights(c["W"], c["U"]))) < 1e-14


# ---------------------------------------------------------------- closed form
def test_pythagorean_basis_worked_example():
    """d=2, k=1, U=(3/5, 4/5)^T: every value below is computed by hand."""
    U = np.array([[0.6], [0.8]])
    E = np.array([[0.5, 0.5], [2.0, -1.0]])
    X = np.array([[1.0, 2.0], [2.0, -1.0]])
    ids = np.array([0, 1], dtype=np.int32)
    # token 0: (1-0.5)*0.6 + (2-0.5)*0.8 = 0.3 + 1.2 = 1.5 ; token 1: X = E[1] -> 0
    np.testing.assert_allclose(O.compress(X, ids, E, U), [[1.5], [0.0]], atol=1e-15)
    # 0.5 + 1.5*0.6 = 1.4 ; 0.5 + 1.5*0.8 = 1.7
    np.testing.assert_allclose(O.decompress(np.array([[1.5], [0.0]]), ids, E, U),
                               [[1.4, 1.7], [2.0, -1.0]], atol=1e-15)
    # G U = 1*0.6 + 2*0.8 = 2.2 ; expand 2.2 -> (1.32, 1.76)
    np.testing.assert_allclose(O.project_grad(np.array([[1.0, 2.0]]), U), [[2.2]], atol=1e-15)
    np.testing.assert_allclose(O.expand_grad(np.array([[2.2]]), U), [[1.32, 1.76]], atol=1e-15)
    # W = e_1 (one column): U^T W = 0.6 -> U*0.6 = (0.36, 0.48)
    np.testing.assert_allclose(O.project_weights(np.array([[1.0], [0.0]]), U), [[0.36], [0.48]],
                               atol=1e-15)


def test_structured_activation_recovers_coordinates():
    """X = E[ids] + Z0 U^T (+ noise orthogonal to span U) compresses to Z0."""
    d, k, V, N = 96, 8, 50, 40
    r = np.random.default_rng(3)
    U = I.gaussian_orthonormal_basis(d, k, 11)
    E = 0.02 * r.standard_normal((V, d))
    ids = r.integers(0, V, size=N).astype(np.int32)
    Z0 = r.standard_normal((N, k))
    X = np.array(E[ids])
    for c in range(k):                       # column-by-column superposition
        X += np.outer(Z0[:, c], U[:, c])
    np.testing.assert_allclose(O.compress(X, ids, E, U), Z0, atol=1e-12)
    # noise in the orthogonal complement (from a complete QR) is invisible
    q, _ = np.linalg.qr(np.concatenate([U, r.standard_normal((d, d - k))], axis=1))
    comp = q[:, k:]
    eta = r.standard_normal((N, d - k)) @ comp.T
    np.testing.assert_allclose(O.compress(X + eta, ids, E, U), Z0, atol=1e-11)
    # generic noise moves Z by at most ||eta|| (U has orthonormal columns)
    eta2 = 1e-3 * r.standard_normal((N, d))
    dz = O.compress(X + eta2, ids, E, U) - Z0
    assert np.linalg.norm(dz) <= np.linalg.norm(eta2) * (1 + 1e-12)


def test_roundtrip_and_identities():
    d, k, V, N = 64, 6, 20, 33
    r = np.random.default_rng(5)
    U = I.gaussian_orthonormal_basis(d, k, 2)
    E = r.standard_normal((V, d)).astype(np.float32)
    ids = r.integers(0, V, size=N).astype(np.int32)
    Z = r.standard_normal((N, k))
    # compress(decompress(Z)) == Z
    np.testing.assert_allclose(O.compress(O.decompress(Z, ids, E, U), ids, E, U), Z, atol=1e-12)
    # decompress(0) is exactly the gathered embedding rows
    assert np.array_equal(O.decompress(np.zeros((N, k)), ids, E, U), E[ids].astype(np.float64))
    # compress(E[ids]) is exactly zero
    assert np.array_equal(O.compress(E[ids], ids, E, U), np.zeros((N, k)))
    # the sender expansion is the adjoint of the gradient projection
    G = r.standard_normal((N, d))
    H = r.standard_normal((N, k))
    lhs = np.sum(O.project_grad(G, U) * H)
    rhs = np.sum(G * O.expand_grad(H, U))
    assert abs(lhs - rhs) <= 1e-12 * abs(lhs)


def test_linearity_and_cross_op_consistency():
    c = _rand_case("f32", N=17, d=40, k=5, V=9)
    r = np.random.default_rng(9)
    G1, G2 = r.standard_normal((2, 17, 40))
    a, b = 1.75, -0.5
    np.testing.assert_allclose(O.project_grad(a * G1 + b * G2, c["U"]),
                               a * O.project_grad(G1, c["U"]) + b * O.project_grad(G2, c["U"]),
                               atol=1e-12)
    # compress = project_grad(X) - project_grad(E[ids])
    np.testing.assert_allclose(O.compress(c["X"], c["ids"], c["E"], c["U"]),
                               O.project_grad(c["X"], c["U"]) - O.project_grad(c["E"][c["ids"]], c["U"]),
                               atol=1e-12)


# ---------------------------------------------------------------- special bases
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_selection_basis_is_exact(dtype):
    d, k, V, N, n = 32, 5, 11, 19, 7
    r = np.random.default_rng(13)
    Uf = I.selection_basis(d, k, 4)
    cols = np.argmax(Uf, axis=0)
    U = I.store(Uf, dtype)
    E = I.store(r.standard_normal((V, d)), dtype)
    X = I.store(r.standard_normal((N, d)), dtype)
    ids = r.integers(0, V, size=N).astype(np.int32)
    Xd, Ed = O.f64(X), O.f64(E)
    assert np.array_equal(O.compress(X, ids, E, U), (Xd - Ed[ids])[:, cols])
    assert np.array_equal(O.project_grad(X, U), Xd[:, cols])
    Z = r.standard_normal((N, k)).astype(np.float32)
    ref = Ed[ids].copy()
    ref[:, cols] += Z
    assert np.array_equal(O.decompress(Z, ids, E, U), ref)
    W = I.store(r.standard_normal((d, n)), dtype)
    PW = np.zeros((d, n))
    PW[cols] = O.f64(W)[cols]
    assert np.array_equal(O.project_weights(W, U), PW)


@pytest.mark.parametrize("d,k", [(256, 8), (4096, 64)])
def test_hadamard_basis_exactly_orthonormal(d, k):
    U = I.store(I.hadamard_basis(d, k, 1), "bf16")
    U64 = O.f64(U)
    assert np.array_equal(U64.T @ U64, np.eye(k))
    r = np.random.default_rng(1)
    Z = r.standard_normal((16, k))
    ids = np.zeros(16, dtype=np.int32)
    E = np.zeros((1, d), dtype=np.float32)
    np.testing.assert_allclose(O.compress(O.decompress(Z, ids, E, U), ids, E, U), Z, atol=1e-12)


# ---------------------------------------------------------------- weights
def test_weight_projection_properties():
    d, k, n = 48, 7, 10
    r = np.random.default_rng(21)
    U = I.gaussian_orthonormal_basis(d, k, 6)
    W1, W2 = r.standard_normal((2, d, n))
    P1 = O.project_weights(W1, U)
    # idempotent
    np.testing.assert_allclose(O.project_weights(P1, U), P1, atol=1e-12)
    # self-adjoint
    assert abs(np.sum(P1 * W2) - np.sum(W1 * O.project_weights(W2, U))) < 1e-10
    # Pythagoras: ||W||^2 = ||PW||^2 + ||W - PW||^2
    assert abs(np.sum(W1 ** 2) - np.sum(P1 ** 2) - np.sum((W1 - P1) ** 2)) < 1e-9
    # rank <= k and columns inside span(U)
    s = np.linalg.svd(P1, compute_uv=False)
    assert np.all(s[k:] < 1e-12 * s[0])
    # a matrix already in the subspace is unchanged; its complement is removed
    A = r.standard_normal((k, n))
    Win = sum(np.outer(U[:, c], A[c]) for c in range(k))
    np.testing.assert_allclose(O.project_weights(Win, U), Win, atol=1e-12)
    q, _ = np.linalg.qr(np.concatenate([U, r.standard_normal((d, d - k))], axis=1))
    Wout = q[:, k:] @ r.standard_normal((d - k, n))
    assert np.linalg.norm(O.project_weights(Wout, U)) < 1e-12 * np.linalg.norm(Wout)


def test_bf16_widening_is_exact():
    bits = np.array([0x0000, 0x3F80, 0xBF80, 0x4049, 0x0001, 0x7F7F], dtype=np.uint16)
    vals = O.f64(bits)
    assert vals[0] == 0.0 and vals[1] == 1.0 and vals[2] == -1.0
    assert vals[3] == 3.140625                       # 0x4049 = 1.5703125 * 2
    assert vals[4] == 2.0 ** -133                     # smallest bf16 subnormal
    assert vals[5] == (2 - 2 ** -7) * 2.0 ** 127      # largest finite bf16


# ---------------------------------------------------------------- paper figures
def test_paper_wire_figures():
    """Printed message sizes of the stage boundary (fixtures cite the passage)."""
    with open(os.path.join(GOLDEN, "paper_figures.json")) as f:
        fig = json.load(f)
    b = fig["uncompressed_boundary_mbit"]
    bits = O.boundary_bits(b["tokens"], b["d"], 32)
    assert round(bits / 1e6) == b["value"]
    c8 = fig["compression_8b"]
    assert c8["d"] / c8["rate"] == pytest.approx(c8["wire_width"])
    c1 = fig["compression_1b"]
    assert round(c1["d"] / c1["rank"]) == c1["rate"]
    # the codec message is 1/rate of the uncompressed one (activations in FP32)
    assert O.boundary_bits(b["tokens"], c8["wire_width"], 32) == pytest.approx(bits / c8["rate"])


# ---------------------------------------------------------------- reparameterized SSN
def test_reparam_forward_equals_the_formed_weight():
    """Eq. (3): the factorized layer computes the same function as H W with
    W = Zp U^T formed explicitly (exact rational brute force)."""
    r = np.random.default_rng(3)
    N, din, d, k = 4, 6, 5, 2
    H = I.store(r.standard_normal((N, din)), "bf16")
    Zp = I.store(r.standard_normal((din, k)), "bf16")
    U = I.store(I.gaussian_orthonormal_basis(d, k, 3), "bf16")
    ref = exact.to_float(exact.reparam_forward(H, Zp, U))
    assert _rel(O.reparam_forward(H, Zp, U), ref) < 1e-14


def test_reparam_gradients_by_exact_perturbation():
    """L = <G, Y> is linear in H and in Zp, so a perturbation by t in one
    entry changes L by exactly t times that entry of the gradient (exact
    rational arithmetic, forward function only)."""
    from fractions import Fraction
    r = np.random.default_rng(11)
    N, din, d, k = 3, 5, 4, 2
    H = r.standard_normal((N, din)).astype(np.float32)
    Zp = r.standard_normal((din, k)).astype(np.float32)
    U = I.gaussian_orthonormal_basis(d, k, 11).astype(np.float32)
    G = r.standard_normal((N, d)).astype(np.float32)
    Gf = exact._frac(G)
    L0 = exact.bilinear(Gf, exact.reparam_forward(H, Zp, U))
    gZ = O.reparam_grad_factor(H, G, U)
    gH = O.reparam_grad_input(G, Zp, U)
    t = 0.5
    for (i, j) in [(0, 0), (din - 1, k - 1), (2, 1)]:
        Zq = Zp.copy()
        Zq[i, j] += np.float32(t)
        dL = exact.bilinear(Gf, exact.reparam_forward(H, Zq, U)) - L0
        step = Fraction(float(Zq[i, j])) - Fraction(float(Zp[i, j]))
        assert abs(float(dL / step) - gZ[i, j]) <= 1e-12 * max(1.0, abs(gZ[i, j]))
    for (i, j) in [(0, 0), (N - 1, din - 1), (1, 3)]:
        Hq = H.copy()
        Hq[i, j] += np.float32(t)
        dL = exact.bilinear(Gf, exact.reparam_forward(Hq, Zp, U)) - L0
        step = Fraction(float(Hq[i, j])) - Fraction(float(H[i, j]))
        assert abs(float(dL / step) - gH[i, j]) <= 1e-12 * max(1.0, abs(gH[i, j]))


def test_reparam_rows_stay_in_the_subspace_and_embedding_round_trips():
    """Every row of the layer output lies in span(U): compressing it (E = 0)
    recovers H Zp exactly in exact arithmetic; the factored embedding looked
    up by id and compressed returns the factor rows E[ids]."""
    r = np.random.default_rng(5)
    N, din, d, k, V = 6, 7, 16, 3, 9
    U = I.hadamard_basis(d, k, 5)                     # exactly orthonormal
    H = r.standard_normal((N, din))
    Zp = r.standard_normal((din, k))
    Y = O.reparam_forward(H, Zp, U)
    zeros = np.zeros((1, d))
    ids0 = np.zeros(N, dtype=np.int32)
    assert _rel(O.compress(Y, ids0, zeros, U), H @ Zp) < 1e-13
    Ef = r.standard_normal((V, k))
    ids = r.integers(0, V, size=N).astype(np.int32)
    X0 = O.factored_embedding(Ef, ids, U)
    assert _rel(O.compress(X0, ids0, zeros, U), Ef[ids]) < 1e-13
    # the factor gradient is the weight gradient projected onto U
    G = r.standard_normal((N, d))
    assert _rel(O.reparam_grad_factor(H, G, U), (H.T @ G) @ U) < 1e-13


# ---------------------------------------------------------------- sparse averaging, delta rule
def test_delta_rule_consensus_and_retained_progress():
    """Eq. (sparta) / Eq. (delta_rule): replicas that did not move during the
    round end on the average; replicas that moved keep their local update on
    top of the consensus shift; coordinates outside P never change."""
    r = np.random.default_rng(9)
    n, R = 200, 4
    P = O.sparta_indices(n, 10, I=r.choice(n, 10, replace=False))
    thetas = [r.standard_normal(n) for _ in range(R)]
    snaps = [O.sparta_snapshot(t, P) for t in thetas]
    avg, deltas = O.sparta_average(snaps, [1.0] * R)
    assert np.allclose(avg, np.mean([t[P] for t in thetas], axis=0), rtol=0, atol=1e-15)
    for j in range(R):
        # no local progress: the replica lands on the average exactly (up to rounding)
        out = O.delta_rule(thetas[j], P, avg, snaps[j])
        assert np.allclose(out[P], avg, atol=1e-15)
        mask = np.ones(n, bool)
        mask[P] = False
        assert np.array_equal(out[mask], thetas[j][mask])
        # local progress made during the round is kept
        moved = thetas[j] + 0.25
        out2 = O.delta_rule(moved, P, avg, snaps[j])
        assert np.allclose(out2[P] - avg, moved[P] - snaps[j], atol=1e-14)
        # the reducer's return is the same correction
        assert np.allclose(snaps[j] + deltas[j], avg, atol=1e-15)
    # lam scales the correction (AsyncMesh form); lam = 0 leaves theta alone
    assert np.array_equal(O.delta_rule(thetas[0], P, avg, snaps[0], 0.0), thetas[0])


def test_sparta_weighted_average_and_segments():
    """Weighted mean by hand, zero-weight senders add nothing (the averaging
    algorithm lets a sender with weight 0 absorb the average), the weighted
    deltas sum to zero, and 20 rotating segments tile the vector."""
    c = [np.array([1.0, 2.0]), np.array([3.0, 6.0]), np.array([100.0, -7.0])]
    acc, deltas = O.sparta_average(c, [1.0, 3.0, 0.0])
    assert np.allclose(acc, [(1 + 9) / 4, (2 + 18) / 4])
    assert np.allclose(deltas[2], acc - c[2])
    assert np.allclose(sum(w * dl for w, dl in zip([1.0, 3.0, 0.0], deltas)), 0.0)
    n, segs = 1000, 20
    cover = np.concatenate([O.sparta_indices(n, n // segs, first=j * (n // segs)) for j in range(segs)])
    assert np.array_equal(np.sort(cover), np.arange(n))



def test_sparta_segment_schedule_by_hand():
    """Segments of n = 10 in S = 4 by hand: [0,2) [2,5) [5,7) [7,10); the
    schedule repeats every S rounds; for any n the segments tile [0, n)
    in order with sizes that differ by at most one."""
    assert [O.sparta_segment(10, r, 4) for r in range(4)] == [(0, 2), (2, 3), (5, 2), (7, 3)]
    assert O.sparta_segment(10, 5, 4) == O.sparta_segment(10, 1, 4)
    for n, S in [(1000, 20), (7, 20), (0, 3), (320_000_003, 20)]:
        segs = [O.sparta_segment(n, r, S) for r in range(S)]
        ends = [f + m for f, m in segs]
        assert segs[0][0] == 0 and ends[-1] == n
        assert all(segs[j + 1][0] == ends[j] for j in range(S - 1))
        sizes = [m for _, m in segs]
        assert max(sizes) - min(sizes) <= 1
    with pytest.raises(ValueError):
        O.sparta_segment(10, -1, 4)


# ---------------------------------------------------------------- parity metric
def test_rel_frobenius_by_hand():
    """The parity metric on values worked by hand: ||got - ref|| / ||ref||
    with ref = diag(3, 4) (norm 5), the argument order matters, bf16 bit
    patterns are widened before the difference, and a zero reference takes
    the absolute bar ||got|| / ||inputs|| (exactly 0 or inf without one)."""
    ref = np.array([[3.0, 0.0], [0.0, 4.0]])
    got = np.array([[3.0, 1.0], [0.0, 4.0]])
    assert O.rel_frobenius(got, ref) == pytest.approx(1.0 / 5.0, rel=1e-15)
    # swapped: the difference has norm 1 and the new reference sqrt(26)
    assert O.rel_frobenius(ref, got) == pytest.approx(1.0 / np.sqrt(26.0), rel=1e-15)
    # a 3-4-5 error: ||(0.3, 0.4)|| = 0.5 against ||(6, 8)|| = 10
    assert O.rel_frobenius(np.array([6.3, 8.4]), np.array([6.0, 8.0])) == pytest.approx(0.05, rel=1e-13)
    # bf16 0x3F80 is 1.0; against 1 + 2^-7 the error is 2^-7 / (1 + 2^-7)
    b = np.array([0x3F80], dtype=np.uint16)
    assert O.rel_frobenius(b, np.array([1.0 + 2 ** -7])) == pytest.approx(2 ** -7 / (1 + 2 ** -7), rel=1e-15)
    assert O.rel_frobenius(b, np.array([1.0])) == 0.0
    # zero reference: ||(3, 4)|| = 5 against inputs of norm 50 -> 0.1
    z = np.zeros(2)
    assert O.rel_frobenius(np.array([3.0, 4.0]), z, scale=50.0) == pytest.approx(0.1, rel=1e-15)
    assert O.rel_frobenius(np.zeros(2), z) == 0.0
    assert O.rel_frobenius(np.array([0.0, 1e-30]), z) == float("inf")
    with pytest.raises(ValueError):
        O.rel_frobenius(np.zeros(3), np.zeros(2))


# ---------------------------------------------------------------- bandwidth estimate
def _body_stage_trainable_params(m, rank):
    """Trainable parameters of one body stage of the reparameterized model
    (section 5.2 model card; section 4.1: the attention and MLP output
    projections are trained as factors of din x k, every other projection is
    full): per layer Wq d x (heads * hd), Wk and Wv d x (kv * hd), the output
    factor (heads * hd) x k, gate and up d x ffn, the down factor ffn x k.
    Normalisation scales (a few thousand values) are left out."""
    d, hd = m["d"], m["head_dim"]
    ffn = int(np.ceil(m["ffn_multiplier"] * (8 * d / 3) / m["ffn_round"]) * m["ffn_round"])
    attn = d * m["heads"] * hd + 2 * d * m["kv_heads"] * hd + m["heads"] * hd * rank
    mlp = 2 * d * ffn + ffn * rank
    return m["body_layers"] * (attn + mlp)


def test_bandwidth_floor_matches_the_paper():
    """Section 3.5.2: about 113 Mbit/s (BF16 all-reduce) and 186 Mbit/s (FP32)
    per contributor, from a_f = a_b = 3, FP32 activations of 4096 tokens at
    the compressed width d / 100 = 51.2, and 5 % of a body stage's trainable
    parameters every 10 s.  Both figures are reproduced to 1 Mbit/s."""
    with open(os.path.join(GOLDEN, "paper_figures.json")) as f:
        fig = json.load(f)
    m, bw, c8 = fig["model_8b"], fig["bandwidth_floor"], fig["compression_8b"]
    params = _body_stage_trainable_params(m, fig["rank_8b"]["rank"])
    assert 900e6 < params < 915e6          # 4 x 226.6M
    payload = m["sparse_share"] * params
    for bits, want in ((16, bw["mbit_per_s_bf16"]), (32, bw["mbit_per_s_fp32"])):
        got = O.bandwidth_floor_bits_per_s(bw["a_f"], bw["a_b"], m["seq_len"], c8["wire_width"],
                                           bits, payload, bw["ar_time_s"]) / 1e6
        assert abs(got - want) <= 1.0, (bits, got, want)
    # the activation share alone: 32 x 6 x 4096 x 51.2 bits/s = 40.3 Mbit/s
    act = O.bandwidth_floor_bits_per_s(3, 3, 4096, 51.2, 16, 0.0, 10.0)
    assert act == pytest.approx(40_265_318.4, rel=1e-12)
