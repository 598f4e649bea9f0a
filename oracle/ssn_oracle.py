"""Plain float64 CPU oracle for the subspace-network (SSN) stage-boundary codec.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the
HIP library and its Python binding) never calls it, and the two share no code.

What the codec computes (paper section 4.1, "Pipeline-Parallel Communication
with Reparameterized SSNs"):

* Eq. (1) writes the residual stream after layer l as the embedding plus a sum
  of attention/MLP output-projection contributions.  When every projection's
  rows lie in span(U_k), U_k (d x k) orthonormal, the stream minus the fixed
  embedding lies in that subspace.
* Eq. (2): a stage subtracts the fixed token embedding (T_fixed, called E
  here; Pluralis-8B uses rotary positions, so there is no additive positional
  term) and sends the k coordinates (X - E[ids]) U_k per token.
* The receiver rebuilds the activation with U_k^T: X' = E[ids] + Z U_k^T.
* Gradients cross the boundary through the same projection: the gradient
  arriving at the receiver's input is sent back as G U_k, and the sender
  expands it to G_Z U_k^T (chain rule through Eq. (2)).
* The original SSN keeps full-width output projections and, after every
  optimizer step, projects them back into the subspace.  With PyTorch's
  [out = d, in = n] weight layout the constrained index is the row index, so
  the projection is W <- U (U^T W).

Every function converts the stored inputs exactly to float64 (bf16 bits are
widened by a shift, fp32 -> f64 is exact), evaluates the definition with
numpy's float64 matmul as the only library primitive, and returns the
unrounded float64 result.  Rows are processed in blocks of at most
``ROW_BLOCK`` tokens so the V x d embedding table is never widened whole.

Parity pins for every function live in tests/test_oracle_pins.py (exact
rational brute force, closed forms and invariants fixed by the definitions).
"""
from __future__ import annotations

import numpy as np

ROW_BLOCK = 4096


def f64(a) -> np.ndarray:
    """Exact float64 view of a stored array.

    uint16 arrays are bfloat16 bit patterns (the top half of an IEEE binary32);
    float32/float64 arrays are taken as they are.
    """
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if a.dtype in (np.float32, np.float64):
        return a.astype(np.float64)
    raise TypeError(f"unsupported stored dtype {a.dtype}")


def compress(X, ids, E, U) -> np.ndarray:
    """Eq. (2): Z = (X - E[ids]) U, one row per token.  X [N,d], ids [N],
    E [V,d], U [d,k]  ->  Z [N,k] float64."""
    X = np.asarray(X)
    ids = np.asarray(ids)
    U64 = f64(U)
    N = X.shape[0]
    Z = np.empty((N, U64.shape[1]), dtype=np.float64)
    for r0 in range(0, N, ROW_BLOCK):
        r1 = min(N, r0 + ROW_BLOCK)
        D = f64(X[r0:r1]) - f64(np.asarray(E)[ids[r0:r1]])
        Z[r0:r1] = D @ U64
    return Z


def decompress(Z, ids, E, U) -> np.ndarray:
    """Receiver side of Eq. (2): X' = E[ids] + Z U^T.  With E and ids both
    None this is the sender-side gradient expansion G_Z U^T."""
    Z64 = f64(Z)
    U64 = f64(U)
    N = Z64.shape[0]
    out = np.empty((N, U64.shape[0]), dtype=np.float64)
    for r0 in range(0, N, ROW_BLOCK):
        r1 = min(N, r0 + ROW_BLOCK)
        out[r0:r1] = Z64[r0:r1] @ U64.T
        if E is not None:
            out[r0:r1] += f64(np.asarray(E)[np.asarray(ids)[r0:r1]])
    return out


def project_grad(G, U) -> np.ndarray:
    """Backward compression: G_Z = G U.  G [N,d] -> [N,k] float64."""
    G = np.asarray(G)
    U64 = f64(U)
    N = G.shape[0]
    out = np.empty((N, U64.shape[1]), dtype=np.float64)
    for r0 in range(0, N, ROW_BLOCK):
        r1 = min(N, r0 + ROW_BLOCK)
        out[r0:r1] = f64(G[r0:r1]) @ U64
    return out


def expand_grad(GZ, U) -> np.ndarray:
    """Sender-side gradient expansion G_Z U^T (decompress without E)."""
    return decompress(GZ, None, None, U)


def project_weights(W, U) -> np.ndarray:
    """Original-SSN re-projection W <- U (U^T W) for W [d, n] ([out, in])."""
    U64 = f64(U)
    W64 = f64(W)
    T = U64.T @ W64
    return U64 @ T


# --------------------------------------------------------------------------
# Reparameterized SSN (section 4.1, Eq. (3)).  An output projection W [din, d]
# (row-vector convention of Eq. (1): a layer adds H W to the residual stream,
# H [N, din]) is stored as its factor Zp [din, k] with W = Zp U^T, so every
# row of W lies in span(U).  The layer never forms W:
#   forward            Y = (H Zp) U^T                          [N, d]
#   input gradient     dL/dH = dL/dY W^T = (dL/dY U) Zp^T       [N, din]
#   factor gradient    dL/dZp = (dL/dW) U = H^T (dL/dY U)       [din, k]
# and the trainable embedding is factored the same way, T_S = E U^T, looked up
# by token id: X0 = E[ids] U^T with E [V, k].
# --------------------------------------------------------------------------
def reparam_forward(H, Zp, U) -> np.ndarray:
    """Y = (H Zp) U^T, row blocks of H."""
    H = np.asarray(H)
    Zp64, U64 = f64(Zp), f64(U)
    N = H.shape[0]
    out = np.empty((N, U64.shape[0]), dtype=np.float64)
    for r0 in range(0, N, ROW_BLOCK):
        r1 = min(N, r0 + ROW_BLOCK)
        out[r0:r1] = (f64(H[r0:r1]) @ Zp64) @ U64.T
    return out


def reparam_grad_input(G, Zp, U) -> np.ndarray:
    """dL/dH = (G U) Zp^T for G = dL/dY [N, d]."""
    G = np.asarray(G)
    Zp64, U64 = f64(Zp), f64(U)
    N = G.shape[0]
    out = np.empty((N, Zp64.shape[0]), dtype=np.float64)
    for r0 in range(0, N, ROW_BLOCK):
        r1 = min(N, r0 + ROW_BLOCK)
        out[r0:r1] = (f64(G[r0:r1]) @ U64) @ Zp64.T
    return out


def reparam_grad_factor(H, G, U) -> np.ndarray:
    """dL/dZp = H^T (G U) [din, k], summed over row blocks of the tokens."""
    H, G = np.asarray(H), np.asarray(G)
    U64 = f64(U)
    out = np.zeros((H.shape[1], U64.shape[1]), dtype=np.float64)
    for r0 in range(0, H.shape[0], ROW_BLOCK):
        r1 = min(H.shape[0], r0 + ROW_BLOCK)
        out += f64(H[r0:r1]).T @ (f64(G[r0:r1]) @ U64)
    return out


def factored_embedding(E, ids, U) -> np.ndarray:
    """X0 = E[ids] U^T for the factored embedding table E [V, k]."""
    return decompress(np.asarray(E)[np.asarray(ids)], None, None, U)


# --------------------------------------------------------------------------
# Sparse weight averaging with the delta rule (section 4.2, Eq. (sparta) and
# Eq. (delta_rule); the asynchronous sparse weight-averaging algorithm of
# section 3.3.1).  Each round
# selects an index set P of the float32 master weights theta (a rotating
# segment, or any shared index set); every replica snapshots theta[P]; a
# reducer averages the replicas' snapshots with weights w_i and returns each
# sender the difference average - snapshot; the replica, whose weights have
# moved on meanwhile, adds lambda times (average - snapshot) to them
# (lambda = 1 in the paper).
# --------------------------------------------------------------------------
def sparta_indices(n: int, m: int, I=None, first: int = 0) -> np.ndarray:
    """The round's index set: the list I, or the segment [first, first + m)."""
    if I is not None:
        return np.asarray(I, dtype=np.int64)
    return np.arange(first, first + m, dtype=np.int64)


def sparta_segment(n: int, r: int, segments: int = 20):
    """(first, m) of the segment averaged in round r.  The run shares a 1/20
    share of the parameters per round and consecutive rounds cover every
    parameter once per 20 rounds (sections 3.3.1 and 5.2); read here as
    `segments` contiguous segments, segment s = [floor(s n / S), floor((s+1) n / S)),
    visited in order, round r taking segment r mod S."""
    if n < 0 or r < 0 or segments < 1:
        raise ValueError("n >= 0, r >= 0 and segments >= 1")
    s = r % segments
    lo = (s * n) // segments
    hi = ((s + 1) * n) // segments
    return lo, hi - lo


def sparta_snapshot(theta, idx) -> np.ndarray:
    """snap = theta[P]."""
    return f64(theta)[np.asarray(idx, dtype=np.int64)]


def sparta_average(chunks, weights):
    """acc = sum_i w_i c_i / sum_i w_i; delta_i = acc - c_i (what the reducer
    returns to sender i)."""
    C = np.stack([f64(c) for c in chunks])
    w = np.asarray(weights, dtype=np.float64)
    acc = (w[:, None] * C).sum(axis=0) / w.sum()
    return acc, [acc - C[i] for i in range(C.shape[0])]


def delta_rule(theta, idx, avg, snap, lam: float = 1.0) -> np.ndarray:
    """theta[P] <- theta[P] + lam (avg - snap); other entries unchanged."""
    out = f64(theta).copy()
    idx = np.asarray(idx, dtype=np.int64)
    out[idx] = out[idx] + lam * (f64(avg) - f64(snap))
    return out


def rel_frobenius(got, ref, scale=None) -> float:
    """The parity metric: ||got - ref||_F / ||ref||_F in float64, got widened
    exactly from its stored dtype (bf16 bit patterns included).

    When the reference is all zero there is no relative error to take; the
    bar is then an absolute one, ||got||_F <= tol * ||inputs||_F, so this
    returns ||got||_F / scale with `scale` the Frobenius norm of the inputs
    that produced the output.  Without a scale a zero reference is met only
    by an exactly zero output (0.0), anything else is infinitely far (inf).
    """
    g = f64(got) if np.asarray(got).dtype == np.uint16 else np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if g.shape != r.shape:
        raise ValueError(f"shape mismatch {g.shape} vs {r.shape}")
    den = np.linalg.norm(r)
    if den > 0.0:
        return float(np.linalg.norm(g - r) / den)
    num = np.linalg.norm(g)
    if scale is not None and scale > 0.0:
        return float(num / scale)
    return 0.0 if num == 0.0 else float("inf")


# --------------------------------------------------------------------------
# Wire sizes of a stage boundary (section 4.1 and the bandwidth estimate of
# section 3.5).  Activations cross the wire in FP32.
# --------------------------------------------------------------------------
def boundary_bits(n_tokens: int, width: float, bits_per_value: int = 32) -> float:
    """Bits of one boundary message carrying `width` values per token."""
    return float(n_tokens) * float(width) * bits_per_value


def bandwidth_floor_bits_per_s(a_f: float, a_b: float, seq_len: int, width: float,
                               ar_bits: int, ar_payload_params: float, ar_time_s: float) -> float:
    """Per-contributor bandwidth estimate of section 3.5.2 (estimated
    communication): a_f forward and a_b backward activation payloads per
    second, each seq_len x width values in FP32, plus one all-reduce of
    `ar_payload_params` values of `ar_bits` bits every `ar_time_s` seconds
    (with SPARTA the payload is the sparse share of the stage's parameters)."""
    return 32.0 * (a_f + a_b) * seq_len * width + ar_bits * ar_payload_params / ar_time_s
