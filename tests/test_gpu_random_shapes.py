"""Seeded random ragged batches against the oracle: the prelude bit-exact, the
attention operators (separate and fused) and small encoder layers within their
tolerances.  Each test walks its seeds in order and stops at the first failing
one, whose seed and shape the assertion names."""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import bf16_row_close, dev, host, scores_close, close, values
from tests.test_gpu_attention import _fused, _fused_close, _oracle_chain, _run_unfused
from tests.test_gpu_layer import _gpu_layer, _small_weights
from tests.test_gpu_offsets import _check_equal, _gpu_plan
from workloads import random_storage

pytestmark = pytest.mark.gpu

N_SEEDS = 12


def _draw(seed, max_batch=40, max_len=600):
    """Lengths with zeros, ones, tile edges and long rows mixed in; 1-4 heads."""
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, max_batch + 1))
    kind = rng.integers(0, 4, size=B)
    L = np.where(kind == 0, rng.integers(0, 3, size=B),
                 np.where(kind == 1, rng.choice([63, 64, 65, 127, 128, 129, 255, 256, 257], size=B),
                          rng.integers(1, max_len + 1, size=B))).astype(np.int32)
    if L.sum() == 0:
        L[0] = 1
    H = int(rng.integers(1, 5))
    return rng, L, H


def test_random_offsets():
    for seed in range(N_SEEDS):
        _, L, H = _draw(seed, max_batch=300, max_len=1500)
        print(f"seed {seed}: offsets B={len(L)} H={H}", flush=True)
        plan = _gpu_plan(L, H)
        try:
            _check_equal(plan, L, H)
        except AssertionError as e:
            raise AssertionError(f"seed {seed}, lengths {L.tolist()}, H {H}") from e


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_random_attention_operators(dtype):
    for seed in range(N_SEEDS):
        rng, L, H = _draw(seed)
        T = int(L.sum())
        print(f"seed {seed}: {dtype} operators B={len(L)} T={T} H={H}", flush=True)
        q, k, v = (random_storage(rng, (T, H * 64), dtype, 0.5) for _ in range(3))
        S, P, O = _run_unfused(L, H, q, k, v, dtype, 0.125)
        tag = f"seed {seed}, lengths {L.tolist()}, H {H}"
        assert scores_close(S, oracle.qkt(dtype, L, H, 64, q, H * 64, k, H * 64, 0.125), L, H, dtype), "QK^T " + tag
        assert scores_close(P, oracle.softmax(dtype, L, H, S), L, H, dtype), "softmax " + tag
        assert close(O, oracle.attn_v(dtype, L, H, 64, P, v, H * 64), dtype, H * 64), "Attn.V " + tag


def test_random_fused_attention():
    for seed in range(N_SEEDS):
        rng, L, H = _draw(seed)
        T = int(L.sum())
        print(f"seed {seed}: fused B={len(L)} T={T} H={H}", flush=True)
        q, k = (random_storage(rng, (T, H * 64), "bf16", float(rng.choice([0.5, 2.0]))) for _ in range(2))
        v = random_storage(rng, (T, H * 64), "bf16", 1.0)
        got = _fused(L, H, q, k, v, 0.125)
        try:
            _fused_close(got, L, H, q, k, v, 0.125)
        except AssertionError as e:
            raise AssertionError(f"seed {seed}, lengths {L.tolist()}, H {H}") from e


def test_random_layers():
    import paper_2110_10221_amd as rag

    flag_choices = [0, rag.RAG_LAYER_BUILD_PLAN, rag.RAG_LAYER_UNFUSED_ATTENTION,
                    rag.RAG_LAYER_BUILD_PLAN | rag.RAG_LAYER_CAUSAL]
    for seed in range(N_SEEDS):
        rng, L, H = _draw(seed, max_batch=12, max_len=300)
        T = int(L.sum())
        d, dff = H * 64, 64 * int(rng.integers(2, 9))
        flags = flag_choices[seed % len(flag_choices)]
        print(f"seed {seed}: layer B={len(L)} T={T} H={H} d_ff={dff} flags={flags}", flush=True)
        x = random_storage(rng, (T, d), "bf16")
        w = _small_weights(rng, d, dff, "bf16")
        if flags & rag.RAG_LAYER_BUILD_PLAN:
            # the layer builds its plan: a fresh plan, no ragged_offsets before
            plan = rag.Plan(torch.from_numpy(L).cuda(), T, int(max(L.max(), 1)), H)
            ws = torch.empty(rag.encoder_layer_workspace(T, int(max(L.max(), 1)), d, H, dff, rag.RAG_BF16, flags),
                             dtype=torch.uint8, device="cuda")
            y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
            rag.encoder_layer(plan, dev(x, "bf16"), y, {n: dev(a, "bf16") for n, a in w.items()}, dff, ws,
                              flags=flags)
            torch.cuda.synchronize()
            assert not plan.data_errors()
            got = host(y, "bf16").reshape(T, d)
        else:
            got = _gpu_layer(L, x, w, d, H, dff, "bf16", flags)
        ref = oracle.encoder_layer("bf16", L, x, w, d, H, dff, causal=bool(flags & rag.RAG_LAYER_CAUSAL))
        ok, worst = bf16_row_close(got, ref, d)
        assert ok, (f"seed {seed}, lengths {L.tolist()}, H {H}, d_ff {dff}, flags {flags}", worst)
