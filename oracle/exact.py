"""Exact rational brute force for the SSN codec on tiny inputs.

TEST INFRASTRUCTURE ONLY (same rule as ssn_oracle.py).  Every stored bf16 or
fp32 value is a dyadic rational, so converting it to ``fractions.Fraction`` is
exact, and every sum and product below is exact.  These loops evaluate the
definitions of section 4.1 one scalar at a time, with no library primitive, and
pin the float64 oracle on inputs small enough for pure Python.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from .ssn_oracle import f64


def _frac(a):
    """Stored array -> nested lists of exact Fractions."""
    return np.vectorize(lambda v: Fraction(float(v)), otypes=[object])(f64(a))


def compress(X, ids, E, U):
    Xf, Ef, Uf = _frac(X), _frac(E), _frac(U)
    N, d = Xf.shape
    k = Uf.shape[1]
    Z = np.empty((N, k), dtype=object)
    for i in range(N):
        row = int(ids[i])
        for c in range(k):
            acc = Fraction(0)
            for j in range(d):
                acc += (Xf[i, j] - Ef[row, j]) * Uf[j, c]
            Z[i, c] = acc
    return Z


def decompress(Z, ids, E, U):
    Zf, Uf = _frac(Z), _frac(U)
    Ef = None if E is None else _frac(E)
    N, k = Zf.shape
    d = Uf.shape[0]
    out = np.empty((N, d), dtype=object)
    for i in range(N):
        for j in range(d):
            acc = Fraction(0) if Ef is None else Ef[int(ids[i]), j]
            for c in range(k):
                acc += Zf[i, c] * Uf[j, c]
            out[i, j] = acc
    return out


def project_grad(G, U):
    Gf, Uf = _frac(G), _frac(U)
    N, d = Gf.shape
    k = Uf.shape[1]
    out = np.empty((N, k), dtype=object)
    for i in range(N):
        for c in range(k):
            acc = Fraction(0)
            for j in range(d):
                acc += Gf[i, j] * Uf[j, c]
            out[i, c] = acc
    return out


def project_weights(W, U):
    Wf, Uf = _frac(W), _frac(U)
    d, n = Wf.shape
    k = Uf.shape[1]
    out = np.empty((d, n), dtype=object)
    for col in range(n):
        t = []
        for c in range(k):
            acc = Fraction(0)
            for j in range(d):
                acc += Uf[j, c] * Wf[j, col]
            t.append(acc)
        for j in range(d):
            acc = Fraction(0)
            for c in range(k):
                acc += Uf[j, c] * t[c]
            out[j, col] = acc
    return out


def _matmul(A, B):
    """Exact product of two Fraction matrices (nested loops)."""
    n, m = A.shape
    p = B.shape[1]
    out = np.empty((n, p), dtype=object)
    for i in range(n):
        for j in range(p):
            acc = Fraction(0)
            for t in range(m):
                acc += A[i, t] * B[t, j]
            out[i, j] = acc
    return out


def reparam_forward(H, Zp, U):
    """Y = H W with the weight formed explicitly, W = Zp U^T (the function the
    factorization must reproduce)."""
    W = _matmul(_frac(Zp), _frac(U).T)
    return _matmul(_frac(H), W)


def bilinear(G, Y):
    """<G, Y> = sum of elementwise products (a loss that is linear in Y)."""
    acc = Fraction(0)
    for g, y in zip(np.asarray(G, dtype=object).ravel(), np.asarray(Y, dtype=object).ravel()):
        acc += g * y
    return acc


def to_float(a) -> np.ndarray:
    return np.vectorize(float, otypes=[np.float64])(a)
