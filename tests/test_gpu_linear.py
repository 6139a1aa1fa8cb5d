"""GPU parity of the token-wise operators against the oracle: packed_linear
(every epilogue, ragged token counts, the layer's shapes) and packed_layernorm."""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import canary_buffer, canary_intact, close, dev, host
from workloads import random_storage

pytestmark = pytest.mark.gpu

ACTS = [oracle.ACT_NONE, oracle.ACT_GELU_ERF, oracle.ACT_GELU_TANH]


def _linear(dtype, T, K, N, act, with_bias, with_res, seed=0, in_place=False, rows=None):
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(seed)
    x = random_storage(rng, (T, K), dtype)
    w = random_storage(rng, (N, K), dtype, 0.05)
    b = random_storage(rng, (N,), dtype, 0.5) if with_bias else None
    r = random_storage(rng, (T, N), dtype) if with_res else None
    print(f"linear {dtype} T={T} K={K} N={N} act={act} bias={with_bias} res={with_res}", flush=True)
    whole, y = canary_buffer(T * N, dtype)
    y = y.view(T, N)
    rd = dev(r, dtype) if with_res else None
    if in_place:
        y.copy_(rd)
        rd = y
    rag.packed_linear(dev(x, dtype), dev(w, dtype), y, dev(b, dtype) if with_bias else None, rd, act)
    torch.cuda.synchronize()
    assert canary_intact(whole, T * N)
    got = host(y, dtype)
    if rows is not None:  # the oracle computes sampled rows only
        x, r, got = x[rows], (r[rows] if with_res else None), got[rows]
    ref = oracle.linear(dtype, x, w, b, r, act)
    return got, ref


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("with_bias,with_res", [(True, True), (True, False), (False, True), (False, False)])
def test_epilogues(dtype, act, with_bias, with_res):
    got, ref = _linear(dtype, 300, 128, 320, act, with_bias, with_res)
    assert close(got, ref, dtype, 320)


@pytest.mark.parametrize("T", [1, 17, 255, 256, 257, 1000])
@pytest.mark.parametrize("K,N", [(64, 64), (512, 1536), (192, 768), (2048, 512)])
def test_ragged_token_counts(T, K, N):
    got, ref = _linear("bf16", T, K, N, oracle.ACT_NONE, True, False, seed=T + K)
    assert close(got, ref, "bf16")


@pytest.mark.parametrize("T,K,N,act,res", [(2236, 2048, 512, oracle.ACT_NONE, True),
                                           (2236, 512, 2048, oracle.ACT_GELU_ERF, False),
                                           (1001, 1024, 320, oracle.ACT_NONE, True),
                                           (5000, 256, 1024, oracle.ACT_NONE, True),
                                           (4096, 256, 2048, oracle.ACT_GELU_TANH, True)])
def test_f32_small_and_large_launches(T, K, N, act, res):
    # fp32 on the matrix cores, 64 x 64 tiles where they leave the busiest CU less
    # work (the batch-32 lognormal FF2 and FF1 shapes, 1001 x 320 with a ragged tail of
    # tokens and features, 5000 tokens: 320 tiles of 128 x 128 on 256 CUs), 128 x 128
    # tiles otherwise (4096 x 2048: 512 tiles, two full rounds); sampled rows
    rows = np.r_[0:16, T // 2:T // 2 + 16, T - 16:T]
    got, ref = _linear("f32", T, K, N, act, True, res, seed=T + K, rows=rows)
    assert close(got, ref, "f32", N)


def test_in_place_residual():
    got, ref = _linear("bf16", 200, 256, 256, oracle.ACT_NONE, True, True, in_place=True)
    assert close(got, ref, "bf16")


def test_empty_batch_is_a_no_op():
    import paper_2110_10221_amd as rag

    x = torch.empty(0, 128, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(64, 128, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(0, 64, dtype=torch.bfloat16, device="cuda")
    rag.packed_linear(x, w, y)
    torch.cuda.synchronize()


@pytest.mark.parametrize("T", [2048, 2049, 3001])
@pytest.mark.parametrize("K,N", [(128, 2112), (192, 3072)])
def test_wide_outputs_ragged_tails(T, K, N):
    # wide outputs with a plain epilogue: ragged token and feature tails over many tiles
    got, ref = _linear("bf16", T, K, N, oracle.ACT_NONE, True, False, seed=T + N)
    assert close(got, ref, "bf16")


@pytest.mark.parametrize("K,N,act,res", [(1024, 3072, 0, False), (1024, 1024, 0, True), (1024, 4096, 1, False),
                                         (4096, 1024, 0, True)])
def test_layer_shapes_full_token_count_sampled_rows(K, N, act, res):
    # the four GEMMs of a d_model 1024 / FFN 4096 layer at 35475 tokens (batch 128,
    # lengths uniform in [32, 512]); the oracle checks 96 sampled rows
    T = 35475
    rows = np.r_[0:32, T // 2:T // 2 + 32, T - 32:T]
    got, ref = _linear("bf16", T, K, N, act, True, res, seed=N, rows=rows)
    assert close(got, ref, "bf16")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T,d", [(1, 64), (37, 512), (1000, 1024), (5, 4096), (3, 72)])
def test_layernorm(dtype, T, d):
    import paper_2110_10221_amd as rag

    if dtype == "f32" and d % 4:
        pytest.skip("fp32 rows are read in 16-byte chunks")
    rng = np.random.default_rng(T * d)
    x = random_storage(rng, (T, d), dtype, 2.0)
    g = random_storage(rng, (d,), dtype, 0.3)
    b = random_storage(rng, (d,), dtype, 0.3)
    whole, y = canary_buffer(T * d, dtype)
    rag.packed_layernorm(dev(x, dtype), dev(g, dtype), dev(b, dtype), y.view(T, d), 1e-5)
    torch.cuda.synchronize()
    assert canary_intact(whole, T * d)
    assert close(host(y, dtype).reshape(T, d), oracle.layernorm(dtype, x, g, b, 1e-5), dtype, d)


def test_layernorm_in_place():
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(9)
    x = random_storage(rng, (64, 512), "bf16")
    g, b = random_storage(rng, (512,), "bf16"), random_storage(rng, (512,), "bf16")
    xd = dev(x, "bf16")
    rag.packed_layernorm(xd, dev(g, "bf16"), dev(b, "bf16"), xd, 1e-5)
    torch.cuda.synchronize()
    assert close(host(xd, "bf16"), oracle.layernorm("bf16", x, g, b, 1e-5), "bf16")
