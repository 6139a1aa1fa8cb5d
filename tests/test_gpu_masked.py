"""GPU parity of masked (causal) attention: the causal operators, the fused causal
kernel and the causal layer against the oracle's masked definitions."""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import (BF16_ATOL, BF16_RTOL, bf16_row_close, canary_buffer, canary_intact, close, dev, host,
                           rising_keys, scores_close, values)
from tests.test_gpu_layer import _gpu_layer, _small_weights
from workloads import BIAS_NAMES, LN_NAMES, WEIGHT_NAMES, make_workload, random_storage

pytestmark = pytest.mark.gpu


def _plan(L, H):
    import paper_2110_10221_amd as rag

    L = np.asarray(L, np.int32)
    plan = rag.Plan(torch.from_numpy(L).cuda(), int(L.sum()), int(max(L.max(), 1)), H)
    rag.ragged_offsets(plan)
    return plan


def _upper(L, H):
    """Boolean mask of the entries j > i of every [L_b, H, L_b] score block, flattened."""
    parts = []
    for n in L:
        n = int(n)
        up = np.arange(n)[None, :] > np.arange(n)[:, None]
        parts.append(np.broadcast_to(up[:, None, :], (n, H, n)).reshape(-1))
    return np.concatenate(parts) if parts else np.zeros(0, bool)


def _lower_only(buf_bits, up, dtype):
    """Check the untouched upper triangle (still the NaN canary) and zero it like the oracle."""
    vals = values(buf_bits, dtype)
    assert np.all(np.isnan(vals[up])), "masked entries were written"
    assert np.all(np.isfinite(vals[~up]))
    out = np.array(buf_bits, copy=True)
    out[up] = 0
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("L", [[1, 15, 16, 17, 63, 64, 65, 127, 129, 200], [0, 7, 0, 300, 2], [513, 40], [64] * 3])
@pytest.mark.parametrize("H", [1, 3])
def test_causal_operators(dtype, L, H):
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(sum(L) * 5 + H)
    L = np.array(L, np.int32)
    T, d = int(L.sum()), H * 64
    q, k, v = (random_storage(rng, (T, d), dtype, 0.5) for _ in range(3))
    n = oracle.score_elems(L, H)
    plan = _plan(L, H)
    print(f"causal ops {dtype} L={L.tolist()} H={H}", flush=True)
    s_whole, S = canary_buffer(n, dtype)
    p_whole, P = canary_buffer(n, dtype)
    o_whole, O = canary_buffer(T * d, dtype)
    rag.ragged_qkt_causal(plan, dev(q, dtype), dev(k, dtype), S, 0.125)
    rag.ragged_softmax_causal(plan, S, P)
    rag.ragged_attn_v_causal(plan, P, dev(v, dtype), O.view(T, d))
    torch.cuda.synchronize()
    assert not plan.data_errors()
    assert canary_intact(s_whole, n) and canary_intact(p_whole, n) and canary_intact(o_whole, T * d)
    up = _upper(L, H)
    Sg, Pg = _lower_only(host(S, dtype), up, dtype), _lower_only(host(P, dtype), up, dtype)
    Og = host(O, dtype).reshape(T, d)
    So = oracle.qkt(dtype, L, H, 64, q, d, k, d, 0.125, causal=True)
    assert scores_close(Sg, So, L, H, dtype), "QK^T"
    assert scores_close(Pg, oracle.softmax(dtype, L, H, Sg, causal=True), L, H, dtype), "softmax"
    assert close(Og, oracle.attn_v(dtype, L, H, 64, Pg, v, d, causal=True), dtype, d), "Attn.V"


def test_causal_softmax_in_place():
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(31)
    L, H = np.array([9, 100, 700], np.int32), 2
    n = oracle.score_elems(L, H)
    S = dev(random_storage(rng, (n,), "bf16", 3.0), "bf16")
    plan = _plan(L, H)
    P = torch.full_like(S, float("nan"))
    rag.ragged_softmax_causal(plan, S, P)
    S2 = S.clone()
    rag.ragged_softmax_causal(plan, S2)
    torch.cuda.synchronize()
    up = torch.from_numpy(_upper(L, H)).cuda()
    assert torch.equal(P[~up].view(torch.int16), S2[~up].view(torch.int16))
    assert torch.equal(S2[up].view(torch.int16), S[up].view(torch.int16))  # in place: masked entries untouched


def _fused_causal(L, H, q, k, v, scale):
    import paper_2110_10221_amd as rag

    T, d = int(np.sum(L)), H * 64
    plan = _plan(L, H)
    o_whole, O = canary_buffer(T * d, "bf16")
    rag.ragged_attention_causal(plan, dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), O.view(T, d), scale)
    torch.cuda.synchronize()
    assert not plan.data_errors()
    assert canary_intact(o_whole, T * d)
    return host(O, "bf16").reshape(T, d)


def _fused_causal_close(got_bits, L, H, q, k, v, scale):
    """As for the unmasked fused kernel: the reference is exact masked attention (the
    oracle's masked chain in fp32 on the same bf16 inputs) and the bf16 bound is
    taken relative to sum_{j<=i} p_ij |v_j| (the oracle's masked Attn.V of |V|)."""
    d = H * 64
    q32, k32, v32 = (values(a, "bf16").astype(np.float32) for a in (q, k, v))
    P = oracle.softmax("f32", L, H, oracle.qkt("f32", L, H, 64, q32, d, k32, d, scale, causal=True), causal=True)
    ref = np.asarray(oracle.attn_v("f32", L, H, 64, P, v32, d, causal=True), np.float64).reshape(-1)
    mag = np.asarray(oracle.attn_v("f32", L, H, 64, P, np.abs(v32), d, causal=True), np.float64).reshape(-1)
    err = np.abs(values(got_bits, "bf16").reshape(-1) - ref)
    excess = err - (BF16_ATOL + BF16_RTOL * mag)
    assert np.all(np.isfinite(err)) and excess.max(initial=0.0) <= 0, excess.max()
    if err.size:
        assert err.mean() <= 4e-3 * mag.mean(), (err.mean(), mag.mean())


@pytest.mark.parametrize("L", [[1, 15, 16, 17, 63, 64, 65, 127, 129, 200], [0, 7, 0, 300, 2], [512] * 3,
                               [8, 64, 9, 384, 511], [33] * 7])
@pytest.mark.parametrize("H", [1, 4])
@pytest.mark.parametrize("qk_scale", [0.5, 4.0])
def test_fused_causal_attention(L, H, qk_scale):
    rng = np.random.default_rng(sum(L) + 3 * H)
    L = np.array(L, np.int32)
    T = int(L.sum())
    print(f"fused causal L={L.tolist()} H={H} qk_scale={qk_scale}", flush=True)
    q, k = (random_storage(rng, (T, H * 64), "bf16", qk_scale) for _ in range(2))
    v = random_storage(rng, (T, H * 64), "bf16", 1.0)
    _fused_causal_close(_fused_causal(L, H, q, k, v, 1 / 8), L, H, q, k, v, 1 / 8)


@pytest.mark.parametrize("H", [16, 3])
def test_fused_causal_every_block_count(H):
    # every count of 32-query blocks per sequence (see the unmasked test) and zero lengths
    from tests.test_gpu_attention import BLOCKS_L

    rng = np.random.default_rng(100 + H)
    L = np.array(BLOCKS_L, np.int32)
    T = int(L.sum())
    print(f"fused causal block counts H={H}", flush=True)
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    _fused_causal_close(_fused_causal(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


def test_fused_causal_reference_raised_every_chunk():
    # scores rising by 16 nats per chunk of 32 keys: each row raises its reference
    # at every chunk up to its own (the diagonal chunk masked past the query)
    L = np.array([700, 512, 33, 64, 95, 1], np.int32)
    H = 2
    print("fused causal rising scores", flush=True)
    q, k, v = rising_keys(L, H, 16.0, seed=3)
    _fused_causal_close(_fused_causal(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


def test_fused_causal_large_batch():
    rng = np.random.default_rng(1101)
    L = rng.integers(0, 41, size=1100).astype(np.int32)
    L[[3, 700]] = [300, 512]
    H, T = 2, int(L.sum())
    print(f"fused causal B=1100 T={T}", flush=True)
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    _fused_causal_close(_fused_causal(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


def test_fused_causal_first_rows_and_prefix():
    # each sequence's first output row is V's first row (up to bf16 rounding of an exact copy),
    # and truncating every sequence to its first m tokens leaves rows < m unchanged
    rng = np.random.default_rng(33)
    L, H = np.array([70, 1, 200], np.int32), 2
    T = int(L.sum())
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    got = _fused_causal(L, H, q, k, v, 0.125)
    st = np.concatenate([[0], np.cumsum(L)])
    for b in range(len(L)):
        assert np.array_equal(got[st[b]], v[st[b]])
    m = np.minimum(L, 40)
    idx = np.concatenate([np.arange(st[b], st[b] + m[b]) for b in range(len(L))])
    got_m = _fused_causal(m, H, q[idx], k[idx], v[idx], 0.125)
    assert np.array_equal(got_m, got[idx])


@pytest.mark.parametrize("L", [[600, 3], [1100, 0, 77, 513]])
def test_fused_causal_long_rows(L):
    # rows longer than 512 keys stream through the same LDS stages
    rng = np.random.default_rng(sum(L))
    L, H = np.array(L, np.int32), 2
    T = int(L.sum())
    print(f"fused causal long L={L.tolist()}", flush=True)
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    _fused_causal_close(_fused_causal(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


@pytest.mark.parametrize("dtype,flags", [("bf16", 2), ("bf16", 3), ("f32", 2)])
@pytest.mark.parametrize("L", [[5, 70, 33, 1], [0, 64, 0, 129], [200, 17, 64, 3, 99]])
def test_causal_layer_small(dtype, flags, L):
    import paper_2110_10221_amd as rag

    assert flags & rag.RAG_LAYER_CAUSAL
    rng = np.random.default_rng(sum(L) + flags)
    L = np.array(L, np.int32)
    d, H, dff = 128, 2, 256
    w = _small_weights(rng, d, dff, dtype)
    x = random_storage(rng, (int(L.sum()), d), dtype)
    print(f"causal layer {dtype} flags={flags} L={L.tolist()}", flush=True)
    got = _gpu_layer(L, x, w, d, H, dff, dtype, flags)
    ref = oracle.encoder_layer(dtype, L, x, w, d, H, dff, causal=True)
    if dtype == "bf16":
        ok, worst = bf16_row_close(got, ref, d)
        assert ok, worst
    else:
        assert close(got, ref, "f32", d)


def test_causal_layer_lognormal_batch_sampled():
    # bf16 layer, batch 32, lognormal lengths (median 60, max 512), d_model 512, 8 heads, FFN 2048, masked
    wl = make_workload(3, seed=0, random_ln=True)
    cfg = wl.cfg
    w = {n: wl.tensors[n] for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    got = _gpu_layer(wl.lengths, wl.tensors["x"], w, cfg.d_model, cfg.heads, cfg.d_ff, "bf16", 2)
    L = wl.lengths
    st = np.concatenate([[0], np.cumsum(L)])
    order = np.argsort(-L, kind="stable")
    for b in sorted({int(order[0]), int(order[-1]), int(order[len(L) // 2])}):
        print(f"  oracle sequence {b} (L={L[b]})", flush=True)
        ref = oracle.encoder_layer("bf16", L[b:b + 1], wl.tensors["x"][st[b]:st[b + 1]], w, cfg.d_model, cfg.heads,
                                   cfg.d_ff, causal=True)
        ok, worst = bf16_row_close(got[st[b]:st[b + 1]], ref, cfg.d_model)
        assert ok, (b, worst)
