"""GPU parity of the triangular matrix multiplication (trmm, Section 7.1):
C = tril(L) B against the oracle element by element on ragged sizes (partial
tiles in every dimension, padded leading dimensions, NaN stored above L's
diagonal), and on sampled rows of the benchmark's 8192 x 8192 product in the
launch configuration the benchmark times."""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import bf16_close, close, dev, host
from workloads import make_trmm_operands

pytestmark = pytest.mark.gpu


def _padded(a, width, dtype):
    """Storage array a [rows, w] placed in the first w columns of a [rows, width] array
    whose other entries are NaN (so a read past a row's end would show)."""
    rows, w = a.shape
    fill = np.float32(np.nan) if dtype == "f32" else np.uint16(0x7fc0)
    out = np.full((rows, width), fill, dtype=a.dtype)
    out[:, :w] = a
    return out


def _run(L, B, n, m, dtype, ldl, ldb, ldc):
    import paper_2110_10221_amd as rag

    Ld = dev(_padded(L, ldl, dtype), dtype)
    Bd = dev(_padded(B, ldb, dtype), dtype)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    Cw = torch.full((n, ldc), float("nan"), dtype=tdt, device="cuda")
    rag.ragged_trmm(Ld[:, :n], Bd[:, :m], Cw[:, :m])
    torch.cuda.synchronize()
    got = host(Cw, dtype)
    if ldc > m:   # columns past m untouched
        assert np.all(np.isnan(got[:, m:].astype(np.float32) if dtype == "f32" else
                               (got[:, m:].astype(np.uint32) << 16).view(np.float32)))
    return np.ascontiguousarray(got[:, :m])


@pytest.mark.parametrize("n,m,pad", [(1, 8, 0), (8, 8, 8), (64, 256, 0), (100, 40, 8), (128, 256, 8),
                                     (129, 264, 0), (300, 520, 16), (520, 136, 8), (700, 8, 0)])
def test_bf16_matches_oracle(n, m, pad):
    rng = np.random.default_rng(n * 7 + m)
    L, B = make_trmm_operands(n, m, rng, "bf16")
    print(f"trmm bf16 n={n} m={m} pad={pad}", flush=True)
    got = _run(L, B, n, m, "bf16", n + (-n % 8) + pad, m + pad, m + pad)
    ref = oracle.trmm("bf16", n, m, L, B)
    ok, worst = bf16_close(got, ref)
    assert ok, worst


@pytest.mark.parametrize("n,m", [(1, 1), (7, 5), (65, 63), (200, 257), (129, 3)])
def test_f32_matches_oracle(n, m):
    rng = np.random.default_rng(n + 100 * m)
    L, B = make_trmm_operands(n, m, rng, "f32")
    print(f"trmm f32 n={n} m={m}", flush=True)
    got = _run(L, B, n, m, "f32", n + 3, m + 1, m + 2)
    assert close(got, oracle.trmm("f32", n, m, L, B), "f32", m)


def test_identity_and_empty():
    import paper_2110_10221_amd as rag

    n, m = 256, 64
    rng = np.random.default_rng(3)
    _, B = make_trmm_operands(n, m, rng, "bf16")
    eye = torch.eye(n, dtype=torch.bfloat16, device="cuda")
    Bd = dev(B, "bf16").view(n, m)
    C = torch.empty_like(Bd)
    rag.ragged_trmm(eye, Bd, C)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), Bd.view(torch.int16))
    z = torch.empty(0, 64, dtype=torch.bfloat16, device="cuda")
    rag.ragged_trmm(torch.empty(0, 0, dtype=torch.bfloat16, device="cuda"), z, z)


def test_host_errors():
    import paper_2110_10221_amd as rag

    L = torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda")
    B = torch.zeros(64, 12, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(rag.RaggedError, match="RAG_ERR_SHAPE"):
        rag.ragged_trmm(L, B, torch.empty_like(B))                       # bf16 needs m % 8 == 0
    B = torch.zeros(64, 16, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(rag.RaggedError, match="RAG_ERR_ARG"):
        rag.ragged_trmm(L, B, B)                                         # C overlaps B


def test_benchmark_size_sampled_rows():
    # the benchmark's 8192 x 8192 bf16 product, NaN above L's diagonal; rows at tile
    # edges and at random checked against the oracle row by row
    import paper_2110_10221_amd as rag

    n = m = 8192
    rng = np.random.default_rng(8192)
    L, B = make_trmm_operands(n, m, rng, "bf16")
    print("trmm bf16 n=m=8192", flush=True)
    Ld, Bd = dev(L, "bf16").view(n, n), dev(B, "bf16").view(n, m)
    C = torch.empty(n, m, dtype=torch.bfloat16, device="cuda")
    rag.ragged_trmm(Ld, Bd, C)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, 127, 128, 4095, 8064, n - 1], rng.integers(0, n, 4)]))
    got = host(C, "bf16")[rows]
    ref = oracle.trmm_rows("bf16", n, m, L, B, rows)
    ok, worst = bf16_close(got, ref)
    assert ok, worst
