"""Shared helpers for the GPU parity tests (test code; may use the oracle)."""
from __future__ import annotations

import numpy as np

from oracle import ssn_oracle as O
from paper_2607_13332_amd import inputs as I

# Parity bars: relative Frobenius error against the float64 oracle.
TOL = {"f32": 1e-5, "bf16": 2e-2}

# Tighter bounds the kernels' own arithmetic guarantees (fp32 accumulation;
# bf16 outputs rounded once, ~2^-9/sqrt(3) relative); they catch regressions
# that the parity bar alone would let through (e.g. dropping the lo half of Z).
DESIGN = {("f32", "f32out"): 3e-6, ("bf16", "f32out"): 2e-5, ("bf16", "bf16out"): 2.5e-3,
          ("f32", "f32out_dec"): 3e-6}

# Unit roundoff of the fp32 accumulation (2^-24 for round to nearest, taken
# as 2^-23 so that any faithful rounding of the hardware is covered) and the
# residual of a float32 operand split into bf16 hi + lo parts (|x - hi - lo|
# <= 2^-16 |x| for round-to-nearest or truncating splits).
U_F32 = 2.0 ** -23
SPLIT = 2.0 ** -16


def rel(got, ref) -> float:
    return O.rel_frobenius(got, ref)


def absval(a) -> np.ndarray:
    """|a| of a stored array, in the stored format (bf16 bit patterns keep
    their magnitude bits), so that the oracle widens it like the original."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return a & np.uint16(0x7FFF)
    return np.abs(a)


def ulp(x, out_bf16: bool) -> np.ndarray:
    """Spacing of the output format at |x| (bf16: 8 significant bits, fp32:
    24), floored at the smallest normal spacing."""
    m = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), 2.0 ** -126)
    _, e = np.frexp(m)                       # m = f 2^e with f in [0.5, 1)
    return np.ldexp(1.0, e - 1 - (7 if out_bf16 else 23))


def elementwise_bound(ref, mag, L: int, split: bool, out_bf16: bool) -> np.ndarray:
    """Per-element error bound of a kernel output against the float64 oracle.

    Every output is a sum of L products accumulated in fp32 (one or two
    chained contractions of total length L), rounded once to the output
    format.  With M the same map applied to the absolute values of the inputs
    (so M bounds the sum of |terms|), the accumulated value differs from the
    exact one by at most L u M (u = fp32 unit roundoff), plus SPLIT M where a
    float32 operand enters the matrix cores as bf16 hi + lo; the final
    rounding adds at most half an output ulp of the accumulated value, which
    is at most one ulp of the exact value.  Twice the accumulation term keeps
    the bound safe when that value sits at a binade edge."""
    acc = (L * U_F32 + (SPLIT if split else 0.0)) * np.asarray(mag, dtype=np.float64)
    return ulp(ref, out_bf16) + 2.0 * acc


def check_elementwise(name, got, ref, mag, L: int, split: bool, out_bf16: bool):
    g = O.f64(got) if np.asarray(got).dtype == np.uint16 else np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    bound = elementwise_bound(r, mag, L, split, out_bf16)
    ratio = np.abs(g - r)
    ratio /= bound
    worst = int(np.argmax(ratio))
    q = float(ratio.flat[worst])
    assert q <= 1.0, (f"{name}: element {np.unravel_index(worst, r.shape)} got {g.flat[worst]!r} "
                      f"ref {r.flat[worst]!r} bound {bound.flat[worst]:.3e}")
    return q


def structured_inputs(cfg, basis="gaussian"):
    """Host inputs for a structured workload: X = E[ids] + Z0 U^T + eta,
    composed in float64 by the oracle with the stored E and U, rounded once."""
    h = I.codec_inputs_host(cfg, basis=basis)
    if cfg.structured:
        x = O.decompress(h["Z0"], h["ids"], h["E"], h["U"]) + h["eta"]
        h["X"] = I.store(x, cfg.dtype)
    return h


def rand_coords(N: int, k: int, seed: int) -> np.ndarray:
    """Seeded float32 coordinates used as decompress / expansion inputs."""
    return np.random.default_rng(seed).standard_normal((N, k)).astype(np.float32)


def sample_rows(N: int, count: int, seed: int) -> np.ndarray:
    """Seeded sorted row sample that always includes the first and last rows."""
    r = np.random.default_rng(seed)
    pick = r.choice(N, size=min(count, N), replace=False)
    return np.unique(np.concatenate([pick, [0, N - 1]])).astype(np.int64)


# Magnitudes M of each op: the oracle's own map on |inputs| (see
# elementwise_bound), with the contraction length L and whether a float32
# operand is split into bf16 hi + lo on the matrix cores.
def mag_compress(X, ids, E, U):
    aU = absval(U)
    return (O.project_grad(absval(X), aU) + O.project_grad(absval(np.asarray(E)[np.asarray(ids)]), aU),
            U.shape[0], False)


def mag_project(G, U):
    return O.project_grad(absval(G), absval(U)), U.shape[0], False


def mag_decompress(Z, ids, E, U):
    return (O.decompress(absval(Z), ids, None if E is None else absval(E), absval(U)),
            U.shape[1], True)


def mag_weights(W, U):
    return O.project_weights(absval(W), absval(U)), U.shape[0] + U.shape[1], True


def mag_reparam_T(H, Zp):
    return mag_project(H, Zp)


def mag_reparam_forward(H, Zp, U):
    return O.reparam_forward(absval(H), absval(Zp), absval(U)), Zp.shape[0] + U.shape[1], True


def mag_reparam_grad_input(G, Zp, U):
    return O.reparam_grad_input(absval(G), absval(Zp), absval(U)), U.shape[0] + U.shape[1], True


def mag_reparam_grad_factor(H, G, U):
    return O.reparam_grad_factor(absval(H), absval(G), absval(U)), U.shape[0] + H.shape[0], True


def check(name, got, ref, dtype, kind, mag=None):
    """Relative Frobenius error against the parity bar and the design bound;
    with `mag` = (M, L, split) also every element against its own bound
    (helpers.elementwise_bound), so that one wrong element cannot hide in
    the norm of a large output."""
    err = rel(got, ref)
    q = None
    if mag is not None:
        M, L, split = mag
        q = check_elementwise(name, got, ref, M, L, split, out_bf16=(kind == "bf16out"))
    print(f"[parity] {name}: rel={err:.3e}" + ("" if q is None else f" max|err|/bound={q:.3f}"),
          flush=True)
    assert err <= TOL[dtype], f"{name}: rel {err:.3e} above the parity bar {TOL[dtype]}"
    assert err <= DESIGN[(dtype, kind)], f"{name}: rel {err:.3e} above design bound"
    return err
