"""GPU parity of the ragged attention operators against the oracle:
ragged_qkt, ragged_softmax, ragged_attn_v (fp32 and bf16) and the fused
ragged_attention (bf16), on the SDPA configurations and on ragged shapes that
exercise every tile edge, with NaN guard regions around every output."""
import math

import numpy as np
import pytest
import torch

import oracle
from tests.helpers import (BF16_ATOL, BF16_RTOL, bf16_close, canary_buffer, canary_intact, close, dev, host,
                           rising_keys, scores_close, values)
from workloads import make_workload, random_storage

pytestmark = pytest.mark.gpu


def _plan(L, H):
    import paper_2110_10221_amd as rag

    L = np.asarray(L, np.int32)
    plan = rag.Plan(torch.from_numpy(L).cuda(), int(L.sum()), int(max(L.max(), 1)), H)
    rag.ragged_offsets(plan)
    return plan


def _run_unfused(L, H, q, k, v, dtype, scale, ld=None):
    import paper_2110_10221_amd as rag

    T = int(np.sum(L))
    d = H * 64
    n = oracle.score_elems(L, H)
    plan = _plan(L, H)
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    if ld is not None:  # Q, K, V as column blocks of one [T, ld] buffer
        buf = torch.zeros(T, ld, dtype=qd.dtype, device="cuda")
        buf[:, :d], buf[:, d:2 * d], buf[:, 2 * d:3 * d] = qd, kd, vd
        qd, kd, vd = buf[:, :d], buf[:, d:2 * d], buf[:, 2 * d:3 * d]
    s_whole, S = canary_buffer(n, dtype)
    p_whole, P = canary_buffer(n, dtype)
    o_whole, O = canary_buffer(T * d, dtype)
    rag.ragged_qkt(plan, qd, kd, S, scale)
    rag.ragged_softmax(plan, S, P)
    rag.ragged_attn_v(plan, P, vd, O.view(T, d))
    torch.cuda.synchronize()
    assert not plan.data_errors(), plan.data_errors()
    assert canary_intact(s_whole, n) and canary_intact(p_whole, n) and canary_intact(o_whole, T * d)
    return host(S, dtype), host(P, dtype), host(O, dtype).reshape(T, d)


def _oracle_chain(L, H, q, k, v, dtype, scale):
    d = H * 64
    S = oracle.qkt(dtype, L, H, 64, q, d, k, d, scale)
    P = oracle.softmax(dtype, L, H, S)
    O = oracle.attn_v(dtype, L, H, 64, P, v, d)
    return S, P, O


def _check_ops(L, H, q, k, v, dtype, scale, ld=None, chain=True):
    """Each operator against the oracle on the same input; with `chain`, also the
    GPU chain against the oracle chain.  (softmax turns an absolute score error e
    into a relative probability error e, so in fp32 the chain comparison only
    holds while |S| * 2^-24 stays well under 1e-5.)"""
    S, P, O = _run_unfused(L, H, q, k, v, dtype, scale, ld)
    So, Po, Oo = _oracle_chain(L, H, q, k, v, dtype, scale)
    assert scores_close(S, So, L, H, dtype), "QK^T"
    assert scores_close(P, oracle.softmax(dtype, L, H, S), L, H, dtype), "softmax"
    assert close(O, oracle.attn_v(dtype, L, H, 64, P, v, H * 64), dtype, H * 64), "Attn.V"
    if chain:
        assert scores_close(P, Po, L, H, dtype), "softmax (chain)"
        assert close(O, Oo, dtype, H * 64), "Attn.V (chain)"


def test_config1_fp32():
    wl = make_workload(1, seed=0)
    print("config 1", wl.lengths.tolist(), flush=True)
    _check_ops(wl.lengths, wl.cfg.heads, wl.tensors["q"], wl.tensors["k"], wl.tensors["v"], "f32", 0.125)


def test_config2_bf16():
    wl = make_workload(2, seed=0)
    print("config 2 T =", wl.total_tokens, flush=True)
    _check_ops(wl.lengths, wl.cfg.heads, wl.tensors["q"], wl.tensors["k"], wl.tensors["v"], "bf16", 0.125)


def test_unfused_operators_batch128_sampled_sequences():
    # the batch-128, 16-head shape: the plan holds about 9.7k (sequence, 64-query,
    # head) items, enough for the operators to group several heads per work item
    # (and QK^T to prefetch the next head's Q block); every operator's output of
    # a spread of whole sequences against the oracle run on that sequence alone
    wl = make_workload(4, seed=0)
    L, H = wl.lengths, wl.cfg.heads
    d = H * 64
    rng = np.random.default_rng(4)
    T = wl.total_tokens
    q, k, v = (random_storage(rng, (T, d), "bf16", 1.0) for _ in range(3))
    print(f"unfused operators B={len(L)} T={T}", flush=True)
    S, P, O = _run_unfused(L, H, q, k, v, "bf16", 0.125)
    tok = np.concatenate([[0], np.cumsum(L)])
    att = H * np.concatenate([[0], np.cumsum(L.astype(np.int64) ** 2)])
    order = np.argsort(-L, kind="stable")
    picks = sorted(set(np.linspace(0, len(L) - 1, 5).round().astype(int).tolist()) | {int(order[0]), int(order[-1])})
    for b in picks:
        Lb = L[b:b + 1]
        qb, kb, vb = (a[tok[b]:tok[b + 1]] for a in (q, k, v))
        Sb, Pb = S[att[b]:att[b + 1]], P[att[b]:att[b + 1]]
        assert scores_close(Sb, oracle.qkt("bf16", Lb, H, 64, qb, d, kb, d, 0.125), Lb, H, "bf16"), ("QK^T", b)
        assert scores_close(Pb, oracle.softmax("bf16", Lb, H, Sb), Lb, H, "bf16"), ("softmax", b)
        assert close(O[tok[b]:tok[b + 1]], oracle.attn_v("bf16", Lb, H, 64, Pb, vb, d), "bf16", d), ("Attn.V", b)


RAGGED = [
    [1, 15, 16, 17, 63, 64, 65, 127, 129, 200],
    [0, 7, 0, 300, 2],
    [513, 40],       # a row longer than the register path of the softmax
    [64] * 5,
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("L", RAGGED)
@pytest.mark.parametrize("H", [1, 3])
def test_ragged_shapes(dtype, L, H):
    rng = np.random.default_rng(sum(L) * 7 + H)
    T = sum(L)
    q, k, v = (random_storage(rng, (T, H * 64), dtype, 0.5) for _ in range(3))
    _check_ops(np.array(L, np.int32), H, q, k, v, dtype, 1 / 8)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_large_scores_and_strided_qkv(dtype):
    # N(0, 4^2) inputs with scale 1: peaked rows exercise the max subtraction;
    # Q, K, V are column blocks of one [T, 3d + 64] buffer
    rng = np.random.default_rng(3)
    L, H = np.array([33, 90, 5], np.int32), 2
    T = int(L.sum())
    q, k, v = (random_storage(rng, (T, H * 64), dtype, 4.0 if i < 2 else 1.0) for i in range(3))
    _check_ops(L, H, q, k, v, dtype, 1.0, ld=3 * H * 64 + 64, chain=dtype == "bf16")


def test_softmax_in_place_matches_out_of_place():
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(4)
    L, H = np.array([9, 100, 700], np.int32), 2
    n = oracle.score_elems(L, H)
    S = dev(random_storage(rng, (n,), "bf16", 3.0), "bf16")
    plan = _plan(L, H)
    P = torch.empty_like(S)
    rag.ragged_softmax(plan, S, P)
    S2 = S.clone()
    rag.ragged_softmax(plan, S2)
    torch.cuda.synchronize()
    assert torch.equal(P.view(torch.int16), S2.view(torch.int16))


def _fused(L, H, q, k, v, scale):
    import paper_2110_10221_amd as rag

    T = int(np.sum(L))
    d = H * 64
    plan = _plan(L, H)
    o_whole, O = canary_buffer(T * d, "bf16")
    rag.ragged_attention(plan, dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), O.view(T, d), scale)
    torch.cuda.synchronize()
    assert not plan.data_errors()
    assert canary_intact(o_whole, T * d)
    return host(O, "bf16").reshape(T, d)


@pytest.mark.parametrize("L", RAGGED + [[512] * 3, [8, 64, 9, 384, 511], [700, 1030, 3, 64, 0, 1537]])
@pytest.mark.parametrize("H", [1, 4])
@pytest.mark.parametrize("qk_scale", [0.5, 4.0])
def test_fused_attention(L, H, qk_scale):
    rng = np.random.default_rng(sum(L) + H)
    L = np.array(L, np.int32)
    T = int(L.sum())
    print(f"fused L={L.tolist()} H={H} qk_scale={qk_scale}", flush=True)
    q, k = (random_storage(rng, (T, H * 64), "bf16", qk_scale) for _ in range(2))
    v = random_storage(rng, (T, H * 64), "bf16", 1.0)
    got = _fused(L, H, q, k, v, 1 / 8)
    _fused_close(got, L, H, q, k, v, 1 / 8)


def _fused_close(got_bits, L, H, q, k, v, scale):
    """The fused kernel stores neither scores nor probabilities, so its reference is
    exact attention (the oracle chain in fp32 on the same bf16 inputs).  Its own
    roundings (bf16 exponentials, bf16 output) perturb each output by a fraction
    of sum_j p_j |v_j|, the scale of the weighted sum, which the oracle's Attn.V of
    |V| gives; the bf16 bound is taken relative to that, per element, and the mean
    error must stay near the rounding level."""
    d = H * 64
    q32, k32, v32 = (values(a, "bf16").astype(np.float32) for a in (q, k, v))
    P = oracle.softmax("f32", L, H, oracle.qkt("f32", L, H, 64, q32, d, k32, d, scale))
    ref = np.asarray(oracle.attn_v("f32", L, H, 64, P, v32, d), np.float64)
    mag = np.asarray(oracle.attn_v("f32", L, H, 64, P, np.abs(v32), d), np.float64)
    err = np.abs(values(got_bits, "bf16").reshape(-1) - ref.reshape(-1))
    mag = mag.reshape(-1)
    excess = err - (BF16_ATOL + BF16_RTOL * mag)
    assert np.all(np.isfinite(err)) and excess.max(initial=0.0) <= 0, excess.max()
    if err.size:
        assert err.mean() <= 4e-3 * mag.mean(), (err.mean(), mag.mean())


# every count of 32-query blocks per sequence, 1..16 (lengths 1, 33, ..., 481, 512),
# with zero lengths between
BLOCKS_L = [1, 33, 0, 65, 97, 129, 161, 193, 225, 257, 289, 321, 353, 385, 417, 449, 481, 512, 32, 0, 96, 7]


@pytest.mark.parametrize("H", [16, 3])
def test_fused_attention_every_block_count(H):
    rng = np.random.default_rng(H)
    L = np.array(BLOCKS_L, np.int32)
    T = int(L.sum())
    print(f"fused block counts H={H}", flush=True)
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    _fused_close(_fused(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


@pytest.mark.parametrize("step", [16.0, 40.0])
def test_fused_attention_reference_raised_every_chunk(step):
    # scores rising by `step` nats per chunk of 32 keys: every later chunk of every
    # row passes the kernel's exponential-sum cap, so each one recomputes its
    # scores, raises the row's reference and rescales the running sums
    L = np.array([700, 512, 33, 64, 95, 1], np.int32)
    H = 2
    print(f"fused rising scores step={step}", flush=True)
    q, k, v = rising_keys(L, H, step, seed=int(step))
    _fused_close(_fused(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


def test_fused_attention_large_batch():
    # 1100 short sequences and two long ones: 2200 (sequence, head) pairs walked by the persistent grid
    rng = np.random.default_rng(1100)
    L = rng.integers(0, 41, size=1100).astype(np.int32)
    L[[3, 700]] = [300, 512]
    H, T = 2, int(L.sum())
    print(f"fused B=1100 T={T}", flush=True)
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    _fused_close(_fused(L, H, q, k, v, 0.125), L, H, q, k, v, 0.125)


def test_fused_attention_sdpa_workload():
    # bf16 ragged attention, batch 32, 8 heads, lengths uniform in [16, 512]
    wl = make_workload(2, seed=0)
    L, H = wl.lengths, wl.cfg.heads
    got = _fused(L, H, wl.tensors["q"], wl.tensors["k"], wl.tensors["v"], 0.125)
    _fused_close(got, L, H, wl.tensors["q"], wl.tensors["k"], wl.tensors["v"], 0.125)


def test_fused_attention_rejects_rows_beyond_32bit_offsets():
    # max_len * ld * 2 bytes must stay below 2^31: a plan promising 2^24-token rows
    # of leading dimension 64 is refused on the host before anything launches
    import paper_2110_10221_amd as rag

    L, H = np.array([3, 5], np.int32), 1
    plan = rag.Plan(torch.from_numpy(L).cuda(), int(L.sum()), 1 << 24, H)
    z = torch.zeros(int(L.sum()), 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(rag.RaggedError, match="RAG_ERR_SHAPE"):
        rag.ragged_attention(plan, z, z, z, torch.empty_like(z), 0.125)


def test_fused_attention_negative_scale():
    rng = np.random.default_rng(11)
    L = np.array([5, 33, 130], np.int32)
    T, H = int(L.sum()), 2
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    got = _fused(L, H, q, k, v, -0.2)
    _fused_close(got, L, H, q, k, v, -0.2)


@pytest.mark.parametrize("scale", [0.0, -0.0])
def test_fused_attention_zero_scale_is_uniform(scale):
    # a zero scale makes every score 0 and the softmax uniform over the row's
    # keys; lengths that leave the last 32-key chunk partial, masked keys included
    rng = np.random.default_rng(12)
    L = np.array([1, 5, 33, 70, 130], np.int32)
    T, H = int(L.sum()), 2
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    got = _fused(L, H, q, k, v, scale)
    assert np.all(np.isfinite(values(got, "bf16")))
    _fused_close(got, L, H, q, k, v, scale)
    # the oracle chain gives the mean of each sequence's V rows, elementwise
    st = np.concatenate([[0], np.cumsum(L)])
    vv = values(v, "bf16").reshape(T, H * 64)
    mean = np.concatenate([np.repeat(vv[st[b]:st[b + 1]].mean(0, keepdims=True), L[b], 0) for b in range(len(L))])
    g = values(got, "bf16").reshape(T, H * 64)
    assert np.abs(g - mean).max() <= 1e-3 + 2e-2 * np.abs(vv).max()


def test_unfused_attention_zero_scale_matches_oracle():
    rng = np.random.default_rng(13)
    L, H = np.array([3, 64, 100], np.int32), 2
    T = int(L.sum())
    q, k, v = (random_storage(rng, (T, H * 64), "bf16", 1.0) for _ in range(3))
    _check_ops(L, H, q, k, v, "bf16", 0.0)


def test_score_buffer_too_small_is_reported_not_written():
    import paper_2110_10221_amd as rag

    rng = np.random.default_rng(5)
    L, H = np.array([40, 50], np.int32), 2
    T = int(L.sum())
    q = dev(random_storage(rng, (T, 128), "bf16"), "bf16")
    n = oracle.score_elems(L, H)
    whole, S = canary_buffer(n - 1, "bf16")
    plan = _plan(L, H)
    rag.ragged_qkt(plan, q, q, S, 0.125)
    torch.cuda.synchronize()
    assert plan.status[0].item() & 32
    assert torch.isnan(whole.float()).all()


def test_determinism_and_sequence_permutation():
    rng = np.random.default_rng(6)
    L, H = np.array([70, 3, 129], np.int32), 2
    T = int(L.sum())
    q, k, v = (random_storage(rng, (T, 128), "bf16") for _ in range(3))
    a = _fused(L, H, q, k, v, 0.125)
    b = _fused(L, H, q, k, v, 0.125)
    assert (a == b).all()
    perm = [2, 0, 1]
    st = np.concatenate([[0], np.cumsum(L)])
    cat = lambda x: np.concatenate([x[st[i]:st[i + 1]] for i in perm])
    c = _fused(L[perm], H, cat(q), cat(k), cat(v), 0.125)
    assert (c == cat(a)).all()
    S1, P1, O1 = _run_unfused(L, H, q, k, v, "bf16", 0.125)
    S2, P2, O2 = _run_unfused(L, H, q, k, v, "bf16", 0.125)
    assert (S1 == S2).all() and (P1 == P2).all() and (O1 == O2).all()
