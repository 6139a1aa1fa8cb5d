"""GPU parity of the variable-sized batched GEMM (vgemm, Section 7.1): the plan
(packed offsets, largest-first order, tile prefix and tile list) bit-exact
against the oracle's, the products against the oracle's vgemm element by element
on small ragged batches, and sampled rows of the paper-sized batch (every size a
multiple of 128 in [512, 1408]) in the launch configuration the benchmark times."""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import bf16_close, canary_buffer, canary_intact, close, dev, host
from workloads import draw_vgemm_dims, make_vgemm_operands

pytestmark = pytest.mark.gpu

TM, TN = oracle.VGEMM_TILE_M, oracle.VGEMM_TILE_N


def _plan(dims, tile_cap=None):
    import paper_2110_10221_amd as rag

    d = np.ascontiguousarray(np.asarray(dims, np.int32).reshape(-1, 3))
    plan = rag.VgemmPlan(torch.from_numpy(d).cuda(), tile_cap=tile_cap, host_dims=d)
    rag.vgemm_offsets(plan)
    return plan


def _expected_items(dims, off):
    items = []
    for p in off.order:
        m, n, _ = (int(v) for v in dims[p])
        tm = -(-m // TM)
        for idx in range(tm * -(-n // TN)):
            items.append((p, idx % tm, idx // tm, 0))
    return np.array(items, np.int32).reshape(-1, 4)


@pytest.mark.parametrize("B", [1, 7, 64, 300, 1500])
def test_plan_matches_oracle(B):
    rng = np.random.default_rng(B)
    dims = rng.integers(0, 12, size=(B, 3)).astype(np.int32) * 128
    dims[::3] = rng.integers(1, 2000, size=dims[::3].shape)   # ragged edges, zero sizes, ties
    dims[1::7] = dims[0]
    print(f"vgemm plan B={B}", flush=True)
    plan = _plan(dims)
    off = oracle.vgemm_offsets(dims)
    torch.cuda.synchronize()
    assert not plan.data_errors()
    for name in ("a_off", "b_off", "c_off", "order", "tile_off"):
        assert np.array_equal(getattr(plan, name).cpu().numpy(), getattr(off, name)), name
    n = int(off.tile_off[-1])
    assert plan.n_tiles() == n
    got = plan.tile_items.cpu().numpy()[:4 * n].reshape(-1, 4)
    assert np.array_equal(got, _expected_items(dims, off))


def test_plan_flags():
    import paper_2110_10221_amd as rag

    plan = _plan([[128, -1, 64], [64, 64, 64]], tile_cap=4)
    assert "negative size" in plan.data_errors()
    plan = _plan([[128, 70000, 64]], tile_cap=600)
    assert any("RAG_VGEMM_MAX_DIM" in e for e in plan.data_errors())
    dims = [[300, 600, 64], [128, 256, 64]]          # 3 * 3 + 1 tiles
    plan = _plan(dims, tile_cap=9)
    assert "tile_cap exceeded" in plan.data_errors() and plan.n_tiles() == 0
    # a plan with a data error writes nothing
    a = torch.zeros(300 * 64 + 128 * 64, dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(600 * 64 + 256 * 64, dtype=torch.bfloat16, device="cuda")
    whole, c = canary_buffer(300 * 600 + 128 * 256, "bf16")
    rag.ragged_vgemm(plan, a, b, c)
    torch.cuda.synchronize()
    assert torch.isnan(whole.float()).all()
    assert _plan(dims, tile_cap=10).data_errors() == []


def _run(dims, a, b, dtype, tile_cap=None):
    import paper_2110_10221_amd as rag

    plan = _plan(dims, tile_cap)
    n_c = int(oracle.vgemm_offsets(dims).c_off[-1])
    whole, c = canary_buffer(n_c, dtype)
    rag.ragged_vgemm(plan, dev(a, dtype), dev(b, dtype), c)
    torch.cuda.synchronize()
    assert not plan.data_errors()
    assert canary_intact(whole, n_c)
    return host(c, dtype)


def _check_products(got, dims, a, b, dtype):
    ref = oracle.vgemm(dtype, dims, a, b)
    co = 0
    for m, n, _ in np.asarray(dims, np.int64):
        g, o = got[co:co + m * n], ref[co:co + m * n]
        assert close(g, o, dtype, int(n) if n else None), (m, n, bf16_close(g, o) if dtype == "bf16" else None)
        co += m * n


BF16_CASES = [
    [[1, 8, 64]],                                                   # one row, one 8-wide column block
    [[127, 248, 128], [129, 264, 64], [300, 520, 640], [256, 256, 192]],   # ragged tile edges
    [[5, 16, 64], [0, 64, 64], [64, 0, 128], [40, 40, 0], [513, 776, 256]],  # empty problems, k = 0
    [[128 * i, 256 * j, 64 * (i + j)] for i in range(1, 4) for j in range(1, 3)],  # exact tiles
]


@pytest.mark.parametrize("case", range(len(BF16_CASES)))
def test_bf16_products(case):
    dims = np.array(BF16_CASES[case], np.int32)
    rng = np.random.default_rng(40 + case)
    a, b = make_vgemm_operands(dims, rng, "bf16")
    print(f"vgemm bf16 dims={dims.tolist()}", flush=True)
    _check_products(_run(dims, a, b, "bf16"), dims, a, b, "bf16")


@pytest.mark.parametrize("dims", [
    [[1, 1, 1], [7, 5, 3], [65, 63, 17]],
    [[130, 300, 33], [0, 4, 4], [9, 0, 9], [12, 31, 0], [200, 257, 100]],
])
def test_f32_products_any_shape(dims):
    dims = np.array(dims, np.int32)
    rng = np.random.default_rng(int(dims.sum()))
    a, b = make_vgemm_operands(dims, rng, "f32")
    print(f"vgemm f32 dims={dims.tolist()}", flush=True)
    _check_products(_run(dims, a, b, "f32"), dims, a, b, "f32")


def test_loose_tile_cap():
    # a capacity far above the tile count (idle workgroups) changes nothing
    dims = np.array([[200, 264, 128], [64, 512, 64]], np.int32)
    rng = np.random.default_rng(5)
    a, b = make_vgemm_operands(dims, rng, "bf16")
    exact = _run(dims, a, b, "bf16")
    loose = _run(dims, a, b, "bf16", tile_cap=5000)
    assert np.array_equal(exact, loose)


def test_bf16_shape_rule_and_operand_capacity():
    import paper_2110_10221_amd as rag

    dims = np.array([[64, 12, 64]], np.int32)              # n % 8 != 0: bf16 refuses, fp32 accepts
    plan = _plan(dims)
    a = torch.ones(64 * 64, dtype=torch.bfloat16, device="cuda")
    b = torch.ones(12 * 64, dtype=torch.bfloat16, device="cuda")
    whole, c = canary_buffer(64 * 12, "bf16")
    rag.ragged_vgemm(plan, a, b, c)
    torch.cuda.synchronize()
    assert any("bf16" in e for e in plan.data_errors())
    assert torch.isnan(whole.float()).all()
    plan = _plan(dims)
    c32 = torch.empty(64 * 12, dtype=torch.float32, device="cuda")
    rag.ragged_vgemm(plan, a.float(), b.float(), c32)
    torch.cuda.synchronize()
    assert not plan.data_errors() and torch.all(c32 == 64)
    # operands smaller than the packed batch
    plan = _plan(dims)
    whole, c32 = canary_buffer(64 * 12 - 1, "f32")
    rag.ragged_vgemm(plan, a.float(), b.float(), c32)
    torch.cuda.synchronize()
    assert "operand buffer too small" in plan.data_errors()
    assert torch.isnan(whole).all()


def test_host_errors():
    import paper_2110_10221_amd as rag

    plan = _plan([[64, 64, 64]])
    x = torch.zeros(64 * 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(rag.RaggedError, match="RAG_ERR_SHAPE"):
        rag.ragged_vgemm(plan, x[1:], x, torch.empty_like(x))       # misaligned bf16 operand
    with pytest.raises(rag.RaggedError, match="RAG_ERR_ARG"):
        rag.ragged_vgemm(plan, x, x, x)                              # c overlaps a
    y = torch.empty_like(x)
    assert rag.library().ragged_vgemm(plan.ref(), x.data_ptr(), x.numel(), x.data_ptr(), x.numel(), y.data_ptr(),
                                      y.numel(), 7, None) == -2           # RAG_ERR_DTYPE
    big = rag.VgemmPlan(plan.dims, tile_cap=1)
    big.c.tile_cap = rag.RAG_VGEMM_MAX_TILES + 1          # rejected on the host before any launch
    with pytest.raises(rag.RaggedError, match="RAG_ERR_CAPACITY"):
        rag.vgemm_offsets(big)


@pytest.mark.parametrize("B", [64, 128])
def test_paper_batch_sampled(B):
    # the benchmark's batch (sizes uniform over the multiples of 128 in [512, 1408])
    # in the benchmark's launch configuration; outputs checked on sampled rows of
    # sampled problems (largest, smallest, median work) against the oracle
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(B)
    dims = draw_vgemm_dims(B, rng)
    a, b = make_vgemm_operands(dims, rng, "bf16")
    print(f"vgemm paper batch B={B}", flush=True)
    off = oracle.vgemm_offsets(dims)
    plan = _plan(dims)
    c = torch.empty(int(off.c_off[-1]), dtype=torch.bfloat16, device="cuda")
    rag.ragged_vgemm(plan, dev(a, "bf16"), dev(b, "bf16"), c)
    torch.cuda.synchronize()
    assert not plan.data_errors()
    got = host(c, "bf16")
    for p in sorted({int(off.order[0]), int(off.order[-1]), int(off.order[B // 2])}):
        m, n, k = (int(v) for v in dims[p])
        rows = np.unique(np.concatenate([[0, 1, TM - 1, TM, m - 1], rng.integers(0, m, 3)]))
        A = a[off.a_off[p]:off.a_off[p + 1]].reshape(m, k)[rows]
        Bp = b[off.b_off[p]:off.b_off[p + 1]]
        ref = oracle.vgemm("bf16", [[len(rows), n, k]], A.reshape(-1), Bp)
        g = got[off.c_off[p]:off.c_off[p + 1]].reshape(m, n)[rows].reshape(-1)
        ok, worst = bf16_close(g, ref)
        assert ok, (p, worst)
