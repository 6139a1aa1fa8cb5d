"""Pins of the oracle's triangular matrix multiplication (trmm, Section 7.1:
a square lower-triangular matrix times a dense matrix, the reduction over k
being a variable loop of extent i + 1).  Checked against numpy's dense product
with np.tril, the reference BLAS routine dtrmm (scipy), closed forms (identity,
all-ones triangle = running sums of B's rows), brute force on tiny inputs, and
the promise that entries above the diagonal are never read (NaN there changes
nothing)."""
import numpy as np
import pytest
import scipy.linalg.blas as blas

import oracle
from tests.test_oracle_numerics import BF16, F32, half_ulp, store, val


def _ops(rng, n, m, dtype, scale=1.0):
    return store(rng.standard_normal((n, n)) * scale, dtype), store(rng.standard_normal((n, m)) * scale, dtype)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("n,m", [(1, 1), (5, 3), (17, 40), (64, 8), (100, 37)])
def test_matches_numpy_tril(dtype, n, m):
    rng = np.random.default_rng(n * 100 + m)
    L, B = _ops(rng, n, m, dtype)
    C = val(oracle.trmm(dtype, n, m, L, B), dtype)
    ref = np.tril(val(L, dtype)) @ val(B, dtype)
    assert np.all(np.abs(C - ref) <= half_ulp(ref, dtype) * (1 + 1e-9) + 1e-300)


def test_matches_reference_blas_dtrmm():
    rng = np.random.default_rng(7)
    n, m = 45, 23
    L, B = _ops(rng, n, m, F32)
    Ld, Bd = val(L, F32), val(B, F32)
    ref = blas.dtrmm(1.0, np.asfortranarray(Ld), np.asfortranarray(Bd), lower=1)
    C = val(oracle.trmm(F32, n, m, L, B), F32)
    assert np.all(np.abs(C - ref) <= half_ulp(ref, F32) * (1 + 1e-9) + 1e-300)


def test_upper_triangle_is_never_read():
    rng = np.random.default_rng(8)
    n, m = 30, 12
    L, B = _ops(rng, n, m, F32)
    Lnan = L.copy()
    Lnan[np.triu_indices(n, 1)] = np.nan
    Lzero = L.copy()
    Lzero[np.triu_indices(n, 1)] = 0
    a = oracle.trmm(F32, n, m, Lnan, B)
    assert np.all(np.isfinite(a)) and np.array_equal(a, oracle.trmm(F32, n, m, Lzero, B))


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_closed_forms(dtype):
    rng = np.random.default_rng(9)
    n, m = 40, 9
    B = store(rng.integers(-4, 5, size=(n, m)).astype(np.float64), dtype)
    # identity: C = B exactly
    assert np.array_equal(oracle.trmm(dtype, n, m, store(np.eye(n), dtype), B), B)
    # all ones on and below the diagonal: row i of C is the sum of B's rows 0..i
    ones = store(np.ones((n, n)), dtype)
    C = val(oracle.trmm(dtype, n, m, ones, B), dtype)
    assert np.array_equal(C, np.cumsum(val(B, dtype), axis=0))   # small integers: exact in both formats


def test_brute_force_and_leading_dimensions():
    rng = np.random.default_rng(10)
    n, m, ldl, ldb = 6, 4, 9, 7
    Lw = store(rng.standard_normal((n, ldl)), F32)
    Bw = store(rng.standard_normal((n, ldb)), F32)
    C = val(oracle.trmm(F32, n, m, Lw, Bw, ldl=ldl, ldb=ldb), F32)
    Lv, Bv = val(Lw, F32), val(Bw, F32)
    for i in range(n):
        for j in range(m):
            exact = sum(Lv[i, k] * Bv[k, j] for k in range(i + 1))
            assert abs(C[i, j] - exact) <= half_ulp(np.array(exact), F32) * (1 + 1e-9) + 1e-300


def test_empty_shapes():
    assert oracle.trmm(F32, 0, 5, np.zeros(0, np.float32), np.zeros(0, np.float32)).shape == (0, 5)
    assert oracle.trmm(F32, 3, 0, np.ones(9, np.float32), np.zeros(0, np.float32), ldb=1).shape == (3, 0)


def test_selected_rows_equal_the_full_product():
    rng = np.random.default_rng(11)
    n, m = 70, 19
    L, B = _ops(rng, n, m, BF16)
    full = oracle.trmm(BF16, n, m, L, B)
    rows = [0, 1, 33, 69, 33]
    assert np.array_equal(oracle.trmm_rows(BF16, n, m, L, B, rows), full[rows])
