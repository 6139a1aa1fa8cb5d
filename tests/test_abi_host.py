"""Host-side checks of the C interface (no GPU needed, nothing is launched).

The library must load, export every function include/ragged.h declares, and
reject bad arguments on the host before any HIP call.  The validation cases use
fake device addresses that are never dereferenced: each case is built to fail
validation.  They are skipped where a GPU is present, so a mistake in a case can
never launch a kernel on fake pointers.
"""
import ctypes
import os
import re

import pytest
import torch

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ragged.h")
LIB = os.path.join(ROOT, "paper_2110_10221_amd", "libragged.so")

needs_lib = pytest.mark.skipif(not os.path.exists(LIB), reason="libragged.so not built")
no_gpu = pytest.mark.skipif(torch.cuda.is_available(), reason="fake-pointer validation cases run only without a GPU")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^(?:const\s+char\s*\*|rag_status)\s+(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_interface():
    names = declared_functions()
    for n in ("ragged_offsets", "ragged_qkt", "ragged_softmax", "ragged_attn_v", "ragged_attention",
              "packed_linear", "packed_layernorm", "encoder_layer", "encoder_layer_workspace",
              "ragged_plan_capacity", "ragged_status_string", "ragged_last_error"):
        assert n in names


@needs_lib
def test_library_exports_every_declared_function():
    lib = ctypes.CDLL(LIB)
    for n in declared_functions():
        assert hasattr(lib, n), n


@needs_lib
def test_package_imports_and_plan_struct_matches_header():
    import paper_2110_10221_amd as rag

    # 4 int32 + 2 int64 + 10 pointers, no padding on LP64
    assert ctypes.sizeof(rag.RagPlan) == 4 * 4 + 2 * 8 + 10 * 8
    assert ctypes.sizeof(rag.RagLayerWeights) == 12 * 8


@needs_lib
@pytest.mark.parametrize("seed", range(5))
def test_plan_capacity_bounds_the_work_lists(seed):
    import numpy as np

    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 200))
    H = int(rng.integers(1, 17))
    L = rng.integers(0, 700, size=B).astype(np.int32)
    q, a = rag.ragged_plan_capacity(B, int(L.sum()), int(L.max()), H)
    p = oracle.offsets(L, H)
    assert len(p.qkt_items) <= q and len(p.av_items) <= a


FAKE = 0x7f0000000000  # never dereferenced


def _plan(rag, **over):
    f = dict(batch=4, total_tokens=232, max_len=128, heads=2, qkt_cap=100, av_cap=100,
             lengths=FAKE, tok_off=FAKE + 0x1000, att_off=FAKE + 0x2000, order=FAKE + 0x3000,
             tok_seq=FAKE + 0x4000, qkt_item_off=FAKE + 0x5000, av_item_off=FAKE + 0x6000,
             qkt_items=FAKE + 0x7000, av_items=FAKE + 0x8000, status=FAKE + 0x9000)
    f.update(over)
    return rag.RagPlan(**f)


@needs_lib
@no_gpu
def test_host_validation_rejects_bad_arguments():
    import paper_2110_10221_amd as rag

    lib = rag.library()
    P = ctypes.c_void_p
    ERR_ARG, ERR_DTYPE, ERR_SHAPE, ERR_CAP, ERR_WS = -1, -2, -3, -4, -5
    s = None  # default stream; never reached

    assert lib.ragged_offsets(None, s) == ERR_ARG
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, batch=0)), s) == ERR_ARG
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, batch=70000)), s) == ERR_ARG
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, heads=0)), s) == ERR_ARG
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, qkt_cap=2 ** 31)), s) == ERR_CAP
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, status=0)), s) == ERR_ARG
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, qkt_items=FAKE + 4)), s) == ERR_ARG  # misaligned
    assert lib.ragged_offsets(ctypes.byref(_plan(rag, max_len=2 ** 30)), s) == ERR_SHAPE   # offset overflow

    plan = ctypes.byref(_plan(rag))
    q = P(FAKE + 0x10000)
    # ragged_qkt(plan, q, ldq, k, ldk, head_dim, scale, scores, cap, dtype, stream)
    lib.ragged_qkt.argtypes = [P, P, ctypes.c_int32, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, P,
                               ctypes.c_int64, ctypes.c_int32, P]
    assert lib.ragged_qkt(plan, q, 128, q, 128, 32, 0.125, q, 10, 1, s) == ERR_SHAPE     # head_dim
    assert lib.ragged_qkt(plan, q, 100, q, 128, 64, 0.125, q, 10, 1, s) == ERR_SHAPE     # ld < H*dh
    assert lib.ragged_qkt(plan, q, 132, q, 132, 64, 0.125, q, 10, 1, s) == ERR_SHAPE     # ld*2 % 16
    assert lib.ragged_qkt(plan, P(FAKE + 2), 128, q, 128, 64, 0.125, q, 10, 1, s) == ERR_SHAPE  # misaligned
    assert lib.ragged_qkt(plan, q, 128, q, 128, 64, 0.125, q, 10, 7, s) == ERR_DTYPE
    assert lib.ragged_qkt(plan, None, 128, q, 128, 64, 0.125, q, 10, 1, s) == ERR_ARG
    assert lib.ragged_qkt(plan, q, 128, q, 128, 64, 0.125, None, 10, 1, s) == ERR_ARG
    assert lib.ragged_qkt(plan, q, 128, q, 128, 64, 0.125, q, -1, 1, s) == ERR_ARG
    assert lib.ragged_qkt(plan, q, 128, q, 128, 64, float("nan"), q, 10, 1, s) == ERR_ARG   # scale not finite
    assert lib.ragged_qkt(plan, q, 128, q, 128, 64, float("inf"), q, 10, 1, s) == ERR_ARG

    lib.ragged_attention.argtypes = [P, P, ctypes.c_int32, P, ctypes.c_int32, P, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_float, P, ctypes.c_int32, ctypes.c_int32, P]
    assert lib.ragged_attention(plan, q, 128, q, 128, q, 128, 64, 0.1, q, 128, 0, s) == ERR_DTYPE  # bf16 only
    assert lib.ragged_attention(plan, q, 128, q, 128, q, 128, 64, float("nan"), q, 128, 1, s) == ERR_ARG
    assert b"scale" in lib.ragged_last_error()

    # packed_linear(x, ldx, w, bias, res, ldr, act, y, ldy, T, K, N, dtype, stream)
    lib.packed_linear.argtypes = [P, ctypes.c_int32, P, P, P, ctypes.c_int32, ctypes.c_int32, P, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P]
    x, w, y = P(FAKE), P(FAKE + 0x100000), P(FAKE + 0x200000)
    assert lib.packed_linear(x, 512, w, None, None, 0, 0, y, 512, 10, 500, 512, 1, s) == ERR_SHAPE   # K % 64
    assert lib.packed_linear(x, 512, w, None, None, 0, 0, y, 512, 10, 512, 500, 1, s) == ERR_SHAPE   # N % 64
    assert lib.packed_linear(x, 512, w, None, None, 0, 5, y, 512, 10, 512, 512, 1, s) == ERR_ARG     # act
    assert lib.packed_linear(x, 512, w, None, None, 0, 0, y, 512, -1, 512, 512, 1, s) == ERR_ARG     # T
    assert lib.packed_linear(x, 512, w, None, None, 0, 0, x, 512, 10, 512, 512, 1, s) == ERR_ARG     # y == x
    assert lib.packed_linear(x, 512, w, None, P(FAKE + 0x200008), 512, 0, y, 512, 10, 512, 512, 1, s) == ERR_SHAPE
    assert lib.packed_linear(x, 512, w, None, y, 256, 0, y, 512, 10, 512, 512, 1, s) == ERR_SHAPE   # ldr < N
    assert lib.packed_linear(x, 512, w, P(FAKE + 2), None, 0, 0, y, 512, 10, 512, 512, 1, s) == ERR_SHAPE  # bias

    lib.packed_layernorm.argtypes = [P, ctypes.c_int32, P, P, ctypes.c_float, P, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_int32, P]
    assert lib.packed_layernorm(x, 512, w, w, 1e-5, y, 512, 10, 500, 1, s) == ERR_SHAPE    # d % 8
    assert lib.packed_layernorm(x, 8192, w, w, 1e-5, y, 8192, 10, 8192, 1, s) == ERR_SHAPE  # d > 4096
    assert lib.packed_layernorm(x, 512, None, w, 1e-5, y, 512, 10, 512, 1, s) == ERR_ARG

    n = ctypes.c_size_t()
    lib.encoder_layer_workspace.argtypes = [ctypes.c_int32] * 7 + [ctypes.POINTER(ctypes.c_size_t)]
    assert lib.encoder_layer_workspace(232, 128, 128, 2, 256, 1, 0, ctypes.byref(n)) == 0
    fused = n.value
    assert lib.encoder_layer_workspace(232, 128, 128, 2, 256, 1, 1, ctypes.byref(n)) == 0
    assert n.value >= fused + 2 * 232 * 128 * 2
    weights = rag.RagLayerWeights(*([FAKE + 0x400000] * 12))
    lib.encoder_layer.argtypes = [P, P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_float, ctypes.c_int32, ctypes.c_int32, P, P, ctypes.c_size_t,
                                  ctypes.c_int32, P, P]
    ws = P(FAKE + 0x800000)
    assert lib.encoder_layer(plan, x, y, 128, 2, 64, 256, 1e-5, 1, 0, ctypes.byref(weights), ws, fused - 1, 1, s,
                             None) == ERR_WS
    assert lib.encoder_layer(plan, x, y, 256, 2, 64, 256, 1e-5, 1, 0, ctypes.byref(weights), ws, fused, 1, s,
                             None) == ERR_SHAPE   # d_model != heads * head_dim
    assert lib.encoder_layer(plan, x, y, 128, 4, 64, 256, 1e-5, 1, 0, ctypes.byref(weights), ws, fused, 1, s,
                             None) == ERR_SHAPE   # heads differ from the plan
    assert lib.encoder_layer(plan, x, y, 128, 2, 64, 256, 1e-5, 1, 8, ctypes.byref(weights), ws, fused, 1, s,
                             None) == ERR_ARG     # unknown flag
    assert lib.encoder_layer(plan, x, x, 128, 2, 64, 256, 1e-5, 1, 0, ctypes.byref(weights), ws, fused, 1, s,
                             None) == ERR_ARG     # x and y overlap
    assert b"overlap" in lib.ragged_last_error()
    lib.ragged_status_string.restype = ctypes.c_char_p
    assert lib.ragged_status_string(-5) == b"RAG_ERR_WORKSPACE"


def _vplan(rag, **over):
    f = dict(batch=3, tile_cap=40, dims=FAKE, a_off=FAKE + 0x1000, b_off=FAKE + 0x2000, c_off=FAKE + 0x3000,
             order=FAKE + 0x4000, tile_off=FAKE + 0x5000, tile_items=FAKE + 0x6000, status=FAKE + 0x7000)
    f.update(over)
    return rag.RagVgemmPlan(**f)


@needs_lib
def test_vgemm_plan_struct_and_capacity():
    import numpy as np
    import paper_2110_10221_amd as rag

    # int32 batch (padded to 8) + int64 tile_cap + 8 pointers
    assert ctypes.sizeof(rag.RagVgemmPlan) == 8 + 8 + 8 * 8
    rng = np.random.default_rng(0)
    dims = rng.integers(0, 3000, size=(50, 3)).astype(np.int32)
    cap = rag.vgemm_plan_capacity(50, int(dims[:, 0].max()), int(dims[:, 1].max()))
    assert int(oracle.vgemm_offsets(dims).tile_off[-1]) <= cap
    assert rag.vgemm_plan_capacity(2, 129, 256) == 2 * 2 * 1
    with pytest.raises(rag.RaggedError, match="RAG_ERR_ARG"):
        rag.vgemm_plan_capacity(0, 128, 128)


@needs_lib
def test_vgemm_tile_count_matches_the_oracle_prefix():
    import numpy as np
    import paper_2110_10221_amd as rag

    for seed in range(4):
        rng = np.random.default_rng(seed)
        dims = rng.integers(0, 3000, size=(int(rng.integers(1, 80)), 3)).astype(np.int32)
        dims[::7, 2] = 0  # k = 0 problems still own output tiles
        assert rag.vgemm_tile_count(dims) == int(oracle.vgemm_offsets(dims).tile_off[-1])
    assert rag.vgemm_tile_count([[128, 256, 64], [129, 257, 64], [0, 512, 64]]) == 1 + 4 + 0
    with pytest.raises(rag.RaggedError, match="RAG_ERR_ARG"):
        rag.vgemm_tile_count([[128, -1, 64]])
    with pytest.raises(rag.RaggedError, match="RAG_ERR_ARG"):
        rag.vgemm_tile_count([[rag.RAG_VGEMM_MAX_DIM + 1, 1, 1]])
    with pytest.raises(rag.RaggedError, match="RAG_ERR_ARG"):
        rag.vgemm_tile_count(np.zeros((0, 3), np.int32))


@needs_lib
def test_plan_rejects_non_contiguous_lengths():
    import paper_2110_10221_amd as rag

    L = torch.tensor([3, 5, 7, 9], dtype=torch.int32)
    with pytest.raises(ValueError, match="contiguous"):
        rag.Plan(L[::2], 10, 7, 2)
    with pytest.raises(ValueError, match="contiguous"):
        rag.Plan(torch.tensor([4], dtype=torch.int32).expand(8), 32, 4, 2)


@needs_lib
@no_gpu
def test_vgemm_host_validation():
    import paper_2110_10221_amd as rag

    lib = rag.library()
    P = ctypes.c_void_p
    ERR_ARG, ERR_DTYPE, ERR_SHAPE, ERR_CAP = -1, -2, -3, -4
    s = None
    off = lib.vgemm_offsets
    assert off(None, s) == ERR_ARG
    assert off(ctypes.byref(_vplan(rag, batch=0)), s) == ERR_ARG
    assert off(ctypes.byref(_vplan(rag, batch=4097)), s) == ERR_ARG
    assert off(ctypes.byref(_vplan(rag, tile_cap=-1)), s) == ERR_ARG
    assert off(ctypes.byref(_vplan(rag, tile_cap=(1 << 30) + 1)), s) == ERR_CAP
    assert off(ctypes.byref(_vplan(rag, order=0)), s) == ERR_ARG
    assert off(ctypes.byref(_vplan(rag, tile_items=FAKE + 8)), s) == ERR_ARG    # not 16-byte aligned
    assert off(ctypes.byref(_vplan(rag, a_off=FAKE + 4)), s) == ERR_ARG         # int64 array misaligned
    plan = ctypes.byref(_vplan(rag))
    a, b, c = P(FAKE + 0x100000), P(FAKE + 0x200000), P(FAKE + 0x300000)
    vg = lib.ragged_vgemm
    vg.argtypes = [P, P, ctypes.c_int64, P, ctypes.c_int64, P, ctypes.c_int64, ctypes.c_int32, P]
    assert vg(plan, a, 10, b, 10, c, 10, 5, s) == ERR_DTYPE
    assert vg(plan, None, 10, b, 10, c, 10, 1, s) == ERR_ARG
    assert vg(plan, a, -1, b, 10, c, 10, 1, s) == ERR_ARG
    assert vg(plan, P(FAKE + 0x100008), 10, b, 10, c, 10, 1, s) == ERR_SHAPE      # bf16 needs 16-byte alignment
    assert vg(plan, a, 10, b, 10, P(FAKE + 0x100010), 10, 1, s) == ERR_ARG        # c overlaps a
    assert vg(plan, a, 10, b, 10, P(FAKE + 0x200000 + 36), 100, 0, s) == ERR_ARG  # c overlaps b (fp32)


@needs_lib
@no_gpu
def test_trmm_host_validation():
    import paper_2110_10221_amd as rag

    lib = rag.library()
    P = ctypes.c_void_p
    ERR_ARG, ERR_DTYPE, ERR_SHAPE = -1, -2, -3
    tr = lib.ragged_trmm
    tr.argtypes = [P, ctypes.c_int32, P, ctypes.c_int32, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_int32, P]
    l, b, c = P(FAKE), P(FAKE + 0x10000000), P(FAKE + 0x20000000)
    s = None
    assert tr(l, 64, b, 64, c, 64, 64, 64, 4, s) == ERR_DTYPE
    assert tr(l, 64, b, 64, c, 64, -1, 64, 1, s) == ERR_ARG
    assert tr(l, 64, b, 64, c, 64, 0, 64, 1, s) == 0            # empty: nothing to do, nothing launched
    assert tr(l, 64, b, 64, c, 64, 64, 0, 1, s) == 0
    assert tr(l, 32, b, 64, c, 64, 64, 64, 1, s) == ERR_SHAPE    # ldl < n
    assert tr(l, 64, b, 60, c, 64, 64, 64, 1, s) == ERR_SHAPE    # ldb < m
    assert tr(l, 64, b, 72, c, 72, 64, 68, 1, s) == ERR_SHAPE    # bf16: m % 8
    assert tr(l, 68, b, 64, c, 64, 64, 64, 1, s) == ERR_SHAPE    # bf16: ld keeps rows 16-byte aligned
    assert tr(P(FAKE + 8), 64, b, 64, c, 64, 64, 64, 1, s) == ERR_SHAPE   # misaligned bf16 operand
    assert tr(None, 64, b, 64, c, 64, 64, 64, 1, s) == ERR_ARG
    assert tr(l, 64, b, 64, P(FAKE + 0x10000000 + 64), 64, 64, 64, 1, s) == ERR_ARG   # C overlaps B
    assert tr(l, 64, b, 64, P(FAKE + 4096), 64, 64, 64, 1, s) == ERR_ARG             # C overlaps L
    assert tr(l, 1 << 23, b, 64, c, 64, 64, 64, 1, s) == ERR_SHAPE                    # ldl too large for bf16
    assert b"ldl" in lib.ragged_last_error()
