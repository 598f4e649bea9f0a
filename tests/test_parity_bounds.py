"""CPU checks of the per-element parity bound used by the GPU tests
(helpers.elementwise_bound): results computed the way the kernels compute
them -- fp32 accumulation, a float32 operand split into bf16 hi + lo, one
rounding to the output format -- stay inside it, and a single wrong element,
or a dropped lo half, does not."""
import numpy as np
import pytest

from helpers import check_elementwise, mag_compress, mag_decompress, mag_weights
from oracle import ssn_oracle as O
from paper_2607_13332_amd import inputs as I


def _f32_dot_rows(A, B):
    """A [n, L] @ B [L, m] accumulated sequentially in float32 (products of
    bf16 values are exact in float32; fp32 inputs round each FMA once)."""
    A32 = np.asarray(A, dtype=np.float64)
    B32 = np.asarray(B, dtype=np.float64)
    acc = np.zeros((A32.shape[0], B32.shape[1]), dtype=np.float32)
    for j in range(A32.shape[1]):
        acc = (acc.astype(np.float64) + np.outer(A32[:, j], B32[j])).astype(np.float32)
    return acc


def _split_bf16(x32):
    hi = O.f64(I.store(x32, "bf16"))
    lo = O.f64(I.store(np.asarray(x32, dtype=np.float64) - hi, "bf16"))
    return hi, lo


def _case(seed=3, N=48, d=256, k=16, V=20):
    r = np.random.default_rng(seed)
    U = I.store(I.gaussian_orthonormal_basis(d, k, seed), "bf16")
    E = I.store(0.02 * r.standard_normal((V, d)), "bf16")
    X = I.store(r.standard_normal((N, d)), "bf16")
    ids = r.integers(0, V, size=N).astype(np.int32)
    Z = r.standard_normal((N, k)).astype(np.float32)
    return X, ids, E, U, Z


def test_fp32_accumulated_compress_is_inside_the_bound():
    X, ids, E, U, _ = _case()
    got = (_f32_dot_rows(O.f64(X), O.f64(U)).astype(np.float64)
           - _f32_dot_rows(O.f64(E)[ids], O.f64(U)).astype(np.float64)).astype(np.float32)
    M, L, split = mag_compress(X, ids, E, U)
    q = check_elementwise("sim compress", got, O.compress(X, ids, E, U), M, L, split, out_bf16=False)
    assert q < 1.0


def test_split_and_rounded_decompress_is_inside_the_bound():
    X, ids, E, U, Z = _case()
    hi, lo = _split_bf16(Z)
    acc = (_f32_dot_rows(hi, O.f64(U).T).astype(np.float64)
           + _f32_dot_rows(lo, O.f64(U).T).astype(np.float64)).astype(np.float32)
    got = I.store(acc.astype(np.float64) + O.f64(E)[ids], "bf16")
    ref = O.decompress(Z, ids, E, U)
    M, L, split = mag_decompress(Z, ids, E, U)
    assert check_elementwise("sim decompress", got, ref, M, L, split, out_bf16=True) <= 1.0
    # the same without the lo half of Z: outside the bound
    bad = I.store(_f32_dot_rows(hi, O.f64(U).T).astype(np.float64) + O.f64(E)[ids], "bf16")
    with pytest.raises(AssertionError):
        check_elementwise("sim decompress, lo dropped", bad, ref, M, L, split, out_bf16=True)


@pytest.mark.parametrize("where", [(0, 0), (17, 5), (47, 15)])
def test_one_wrong_element_is_caught(where):
    X, ids, E, U, _ = _case()
    ref = O.compress(X, ids, E, U)
    got = ref.astype(np.float32)
    M, L, split = mag_compress(X, ids, E, U)
    check_elementwise("exact", got, ref, M, L, split, out_bf16=False)
    bad = got.copy()
    bad[where] = 0.0 if abs(bad[where]) > 0.05 else 1.0     # a lane that stored nothing useful
    with pytest.raises(AssertionError):
        check_elementwise("one wrong element", bad, ref, M, L, split, out_bf16=False)
    # the whole-output Frobenius metric alone barely moves
    assert O.rel_frobenius(bad, ref) < 0.2


def test_weight_projection_bound_and_a_swapped_column():
    r = np.random.default_rng(5)
    d, n, k = 128, 40, 8
    U = I.store(I.gaussian_orthonormal_basis(d, k, 5), "bf16")
    W = I.store(0.02 * r.standard_normal((d, n)), "bf16")
    T = _f32_dot_rows(O.f64(U).T, O.f64(W))
    hi, lo = _split_bf16(T)
    acc = (_f32_dot_rows(O.f64(U), hi).astype(np.float64)
           + _f32_dot_rows(O.f64(U), lo).astype(np.float64))
    got = I.store(acc, "bf16")
    ref = O.project_weights(W, U)
    M, L, split = mag_weights(W, U)
    assert check_elementwise("sim weights", got, ref, M, L, split, out_bf16=True) <= 1.0
    bad = got.copy()
    bad[:, [3, 4]] = bad[:, [4, 3]]
    with pytest.raises(AssertionError):
        check_elementwise("swapped columns", bad, ref, M, L, split, out_bf16=True)
