"""encoder_layer_noalloc (the layer with the library's fixed device scratch array
as its workspace) against encoder_layer with a caller workspace: the same
kernels on the same inputs, so the outputs must be bit-identical.  Two calls in
a row, the second on a smaller batch (the scratch array keeps the first call's
contents), and a layer too large for the array is refused before launching."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from tests.helpers import bf16_row_close, canary_buffer, canary_intact, dev, host
from workloads import BIAS_NAMES, LN_NAMES, WEIGHT_NAMES, make_workload, random_storage

pytestmark = pytest.mark.gpu


def _weights(rng, d, dff):
    w = {}
    for n, shape in (("w_qkv", (3 * d, d)), ("w_o", (d, d)), ("w_ff1", (dff, d)), ("w_ff2", (d, dff))):
        w[n] = random_storage(rng, shape, "bf16", 0.05)
    for n, m in (("b_qkv", 3 * d), ("b_o", d), ("b_ff1", dff), ("b_ff2", d)):
        w[n] = random_storage(rng, (m,), "bf16", 0.05)
    for n in LN_NAMES:
        w[n] = random_storage(rng, (d,), "bf16", 0.1)
    return w


def _both(L, x, w, d, H, dff, flags):
    """(encoder_layer output, encoder_layer_noalloc output) as bf16 storage."""
    import paper_2110_10221_amd as rag

    L = np.asarray(L, np.int32)
    T, mx = int(L.sum()), int(L.max())
    lens = torch.from_numpy(L).cuda()
    wd = {n: dev(a, "bf16") for n, a in w.items()}
    xd = dev(x, "bf16")
    outs = []
    for noalloc in (False, True):
        plan = rag.Plan(lens, T, mx, H)
        if not flags & rag.RAG_LAYER_BUILD_PLAN:
            rag.ragged_offsets(plan)
        whole, y = canary_buffer(T * d, "bf16")
        if noalloc:
            rag.encoder_layer_noalloc(plan, xd, y.view(T, d), wd, dff, flags=flags)
        else:
            ws = torch.empty(rag.encoder_layer_workspace(T, mx, d, H, dff, rag.RAG_BF16, flags), dtype=torch.uint8,
                             device="cuda")
            rag.encoder_layer(plan, xd, y.view(T, d), wd, dff, ws, flags=flags)
        torch.cuda.synchronize()
        assert not plan.data_errors(), plan.data_errors()
        assert canary_intact(whole, T * d)
        outs.append(host(y, "bf16").reshape(T, d))
    return outs


def test_noalloc_matches_encoder_layer_twice_second_smaller():
    import paper_2110_10221_amd as rag

    # first call: the batch-32 d512 layer (lognormal lengths), building its plan
    wl = make_workload(3, seed=2, random_ln=True)
    cfg = wl.cfg
    w = {n: wl.tensors[n] for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    print(f"noalloc call 1: B={cfg.batch} T={wl.total_tokens} d={cfg.d_model}", flush=True)
    ref, got = _both(wl.lengths, wl.tensors["x"], w, cfg.d_model, cfg.heads, cfg.d_ff, rag.RAG_LAYER_BUILD_PLAN)
    assert np.array_equal(got, ref)
    # second call: a smaller batch and width, unfused attention (score buffer in the scratch too)
    rng = np.random.default_rng(7)
    L = np.array([5, 70, 33, 0, 129], np.int32)
    d, H, dff = 128, 2, 256
    x = random_storage(rng, (int(L.sum()), d), "bf16")
    w = _weights(rng, d, dff)
    print(f"noalloc call 2: B={len(L)} T={int(L.sum())} d={d}", flush=True)
    ref, got = _both(L, x, w, d, H, dff, rag.RAG_LAYER_UNFUSED_ATTENTION)
    assert np.array_equal(got, ref)
    ok, worst = bf16_row_close(got, oracle.encoder_layer("bf16", L, x, w, d, H, dff), d)
    assert ok, worst


def test_noalloc_refuses_a_layer_larger_than_its_scratch():
    import paper_2110_10221_amd as rag

    # the batch-128 d1024 layer needs ~436 MB of workspace, above the fixed array
    L = np.full(128, 277, np.int32)
    T, d, H, dff = int(L.sum()), 1024, 16, 4096
    assert rag.encoder_layer_workspace(T, 277, d, H, dff) > rag.RAG_NOALLOC_SCRATCH_BYTES
    plan = rag.Plan(torch.from_numpy(L).cuda(), T, 277, H)
    w = {n: torch.zeros(s, dtype=torch.bfloat16, device="cuda")
         for n, s in (("w_qkv", (3 * d, d)), ("b_qkv", (3 * d,)), ("w_o", (d, d)), ("b_o", (d,)), ("ln1_g", (d,)),
                      ("ln1_b", (d,)), ("w_ff1", (dff, d)), ("b_ff1", (dff,)), ("w_ff2", (d, dff)), ("b_ff2", (d,)),
                      ("ln2_g", (d,)), ("ln2_b", (d,)))}
    x = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    whole, y = canary_buffer(T * d, "bf16")
    with pytest.raises(rag.RaggedError, match="RAG_ERR_WORKSPACE"):
        rag.encoder_layer_noalloc(plan, x, y.view(T, d), w, dff, flags=rag.RAG_LAYER_BUILD_PLAN)
    torch.cuda.synchronize()
    assert torch.isnan(whole.float()).all()  # nothing was launched
