"""Pins of the oracle's variable-sized batched GEMM (vgemm, Section 7.1): packed
storage offsets, largest-first order and tile prefix against hand-worked values and
numpy; the products against numpy per problem and against the fully padded batched
GEMM the paper compares with (pad every problem to the largest sizes, one dense
batched matmul, crop)."""
import numpy as np
import pytest

import oracle
from tests.test_oracle_numerics import BF16, F32, half_ulp, store, val


def test_offsets_hand_worked():
    # (m, n, k) = (512, 640, 768) and (1408, 512, 512); 128 x 256 output tiles
    off = oracle.vgemm_offsets([[512, 640, 768], [1408, 512, 512]])
    assert off.a_off.tolist() == [0, 512 * 768, 512 * 768 + 1408 * 512]
    assert off.b_off.tolist() == [0, 640 * 768, 640 * 768 + 512 * 512]
    assert off.c_off.tolist() == [0, 512 * 640, 512 * 640 + 1408 * 512]
    assert off.order.tolist() == [1, 0]                    # 369e6 > 252e6 multiply-adds
    assert off.tile_off.tolist() == [0, 11 * 2, 11 * 2 + 4 * 3]


@pytest.mark.parametrize("B", [0, 1, 7, 64])
def test_offsets_match_numpy(B):
    rng = np.random.default_rng(B)
    dims = rng.integers(4, 12, size=(B, 3)) * 128
    dims[::5, 2] = dims[::5, 2] // 2          # some ties and repeated work values
    off = oracle.vgemm_offsets(dims)
    d = dims.astype(np.int64)
    assert (off.a_off == np.concatenate([[0], np.cumsum(d[:, 0] * d[:, 2])])).all()
    assert (off.b_off == np.concatenate([[0], np.cumsum(d[:, 1] * d[:, 2])])).all()
    assert (off.c_off == np.concatenate([[0], np.cumsum(d[:, 0] * d[:, 1])])).all()
    work = d[:, 0] * d[:, 1] * d[:, 2]
    assert (off.order == np.argsort(-work, kind="stable")).all()
    tiles = [-(-int(d[b, 0]) // 128) * -(-int(d[b, 1]) // 256) for b in off.order]
    assert (off.tile_off == np.concatenate([[0], np.cumsum(tiles, dtype=np.int64)])).all()


def test_negative_size_rejected():
    with pytest.raises(ValueError):
        oracle.vgemm_offsets([[128, -1, 128]])


def _batch(rng, dims, dtype, scale=1.0):
    d = np.asarray(dims, np.int64).reshape(-1, 3)
    a = store(rng.standard_normal(int((d[:, 0] * d[:, 2]).sum())) * scale, dtype)
    b = store(rng.standard_normal(int((d[:, 1] * d[:, 2]).sum())) * scale, dtype)
    return a, b


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_products_match_numpy(dtype):
    rng = np.random.default_rng(3)
    dims = [[5, 7, 3], [1, 1, 1], [12, 4, 9], [0, 3, 2], [6, 0, 4], [3, 5, 0]]   # non-square, empty and k = 0
    a, b = _batch(rng, dims, dtype)
    c = val(oracle.vgemm(dtype, dims, a, b), dtype)
    A, Bv = val(a, dtype), val(b, dtype)
    ao = bo = co = 0
    for m, n, k in dims:
        ref = A[ao:ao + m * k].reshape(m, k) @ Bv[bo:bo + n * k].reshape(n, k).T
        got = c[co:co + m * n].reshape(m, n)
        assert np.all(np.abs(got - ref) <= half_ulp(ref, dtype) * (1 + 1e-9) + 1e-300)
        ao, bo, co = ao + m * k, bo + n * k, co + m * n


def test_equals_fully_padded_batched_gemm():
    # the paper's baseline: pad every problem to the largest (m, n, k) with zeros
    rng = np.random.default_rng(4)
    dims = rng.integers(1, 5, size=(9, 3)) * 8
    a, b = _batch(rng, dims, F32)
    c = val(oracle.vgemm(F32, dims, a, b), F32)
    M, N, K = dims.max(axis=0)
    Ap = np.zeros((len(dims), M, K))
    Bp = np.zeros((len(dims), N, K))
    A, Bv = val(a, F32), val(b, F32)
    ao = bo = 0
    for p, (m, n, k) in enumerate(dims):
        Ap[p, :m, :k] = A[ao:ao + m * k].reshape(m, k)
        Bp[p, :n, :k] = Bv[bo:bo + n * k].reshape(n, k)
        ao, bo = ao + m * k, bo + n * k
    Cp = np.matmul(Ap, Bp.transpose(0, 2, 1))
    co = 0
    for p, (m, n, k) in enumerate(dims):
        assert np.allclose(c[co:co + m * n].reshape(m, n), Cp[p, :m, :n], rtol=1e-6, atol=1e-6)
        co += m * n
