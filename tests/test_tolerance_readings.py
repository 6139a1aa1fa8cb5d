"""CPU evidence for the two bf16 tolerance readings the GPU parity tests use.

Neither test touches the GPU path; both compare the oracle with arithmetic
written here independently of it.

* Composed layer (reading of the bf16 tolerance for the whole layer): an
  independent fp32 pipeline (numpy float32 products, torch's bf16 rounding at
  every interface tensor, the same composition of the nine operators) is as
  correct as the GPU path, yet it misses the element-wise bound
  |g - o| <= 1e-3 + 2e-2 |o| on outputs that LayerNorm leaves near zero: a
  one-ulp rounding flip upstream (fp32 against fp64 accumulation landing on
  different sides of a bf16 rounding boundary) reaches them as an absolute
  error.  It meets the row-scaled bound |g - o| <= 1e-3 + 2e-2 max_row |o|
  with a wide margin, and its mean error is tiny.
* Fused attention (reading of its rounding): an emulation of the fused
  kernel's arithmetic (fp32 scores, online softmax whose reference is the
  first chunk's maximum, raised only when a chunk's exponentials sum past
  2^16, bf16 unnormalised exponentials as the P.V operand, one division by
  the fp32 row sum at the end) against exact
  attention (the oracle chain in fp32 on the same bf16 inputs) meets
  |g - o| <= 1e-3 + 2e-2 sum_j p_j |v_j| and a mean error of at most 4e-3 of
  the mean magnitude, while the element-wise bound against the bf16 oracle
  chain (which rounds scores and probabilities) does not hold.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import (BF16_ATOL, BF16_RTOL, ELEM_PASS_MIN, ROW_MEAN_TOL, bf16_row_close, bf16_row_stats, rising_keys,
                           values)
from workloads import BIAS_NAMES, LN_NAMES, WEIGHT_NAMES, bf16_bits_to_f32, make_workload, random_storage


def _rd(x):
    """float32 -> bfloat16 (round to nearest even, torch) -> float32."""
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).float().numpy()


def _layer_fp32(x_bits, w_bits, d, H, dff, eps=1e-5, fused=False):
    """The nine-operator post-LN layer for ONE sequence in float32 with bf16 storage;
    with `fused`, attention takes the fused kernel's arithmetic (_fused_emulation)."""
    v = lambda a: bf16_bits_to_f32(a).astype(np.float32)
    X = v(x_bits)
    W = {k: v(a) for k, a in w_bits.items()}
    n, dh = X.shape[0], d // H
    qkv = _rd(X @ W["w_qkv"].T + W["b_qkv"])
    O = np.zeros((n, d), np.float32)
    if fused:
        bits = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        O = _rd(_fused_emulation(np.array([n]), H, bits(qkv[:, :d]), bits(qkv[:, d:2 * d]), bits(qkv[:, 2 * d:]),
                                 1.0 / np.sqrt(dh)))
    for h in range(H if not fused else 0):
        q = qkv[:, h * dh:(h + 1) * dh]
        k = qkv[:, d + h * dh:d + (h + 1) * dh]
        vv = qkv[:, 2 * d + h * dh:2 * d + (h + 1) * dh]
        S = _rd((q @ k.T) * np.float32(1.0 / np.sqrt(dh)))
        e = np.exp(S - S.max(1, keepdims=True))
        P = _rd(e / e.sum(1, keepdims=True))
        O[:, h * dh:(h + 1) * dh] = _rd(P @ vv)

    def ln(y, g, b):
        m = y.mean(1, keepdims=True)
        var = ((y - m) ** 2).mean(1, keepdims=True)
        return _rd(g * ((y - m) / np.sqrt(var + np.float32(eps))) + b)

    Y1 = _rd(O @ W["w_o"].T + W["b_o"] + X)
    H1 = ln(Y1, W["ln1_g"], W["ln1_b"])
    z = H1 @ W["w_ff1"].T + W["b_ff1"]
    F = _rd(0.5 * z * (1.0 + torch.special.erf(torch.from_numpy(z / np.float32(np.sqrt(2.0)))).numpy()))
    Y2 = _rd(F @ W["w_ff2"].T + W["b_ff2"] + H1)
    return ln(Y2, W["ln2_g"], W["ln2_b"])


@pytest.mark.parametrize("cid", [3, 5])
def test_independent_fp32_layer_meets_the_row_scaled_bound(cid):
    wl = make_workload(cid, seed=0, random_ln=True)
    cfg = wl.cfg
    L = wl.lengths
    st = np.concatenate([[0], np.cumsum(L)])
    w = {n: wl.tensors[n] for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    order = np.argsort(-L, kind="stable")
    elem_worst = -np.inf
    for b in (int(order[0]), int(order[len(L) // 2]), int(order[-1])):
        xs = wl.tensors["x"][st[b]:st[b + 1]]
        ref_bits = oracle.encoder_layer("bf16", L[b:b + 1], xs, w, cfg.d_model, cfg.heads, cfg.d_ff)
        got = _layer_fp32(xs, w, cfg.d_model, cfg.heads, cfg.d_ff)
        got_bits = torch.from_numpy(got).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        ok, worst = bf16_row_close(got_bits, ref_bits, cfg.d_model)
        assert ok and worst < -1e-2, (b, worst)  # a wide margin
        ref = values(ref_bits, "bf16").reshape(-1, cfg.d_model)
        err = np.abs(got.astype(np.float64) - ref)
        rowmax = np.abs(ref).max(1, keepdims=True)
        assert (err / rowmax).mean(1).max() <= 1e-3
        elem_worst = max(elem_worst, float((err - (BF16_ATOL + BF16_RTOL * np.abs(ref))).max()))
    if cid == 5:
        # the longest sequence of the skewed batch misses the element-wise bound
        assert elem_worst > 0, elem_worst


def _fused_emulation(L, H, q, k, v, scale, cap=65536.0, stats=None):
    """The fused kernel's arithmetic: per (sequence, head), blocks of 32 query rows
    (one wave) walk the keys 32 at a time.  The first chunk sets each row's
    reference m to its maximum z = s * |scale| * log2(e); later chunks take
    e = exp2(z - m) and, if any row's sum over either half of the chunk's keys
    (the 16 keys one lane holds: key k with bit 2 of k equal to the lane half)
    exceeds `cap`, the whole block raises m to max(m, chunk maximum), rescales
    its running sums and outputs and recomputes e (counted in stats["raises"])."""
    T, d = int(np.sum(L)), H * 64
    qf, kf, vf = (bf16_bits_to_f32(a).reshape(T, d).astype(np.float32) for a in (q, k, v))
    out = np.zeros((T, d), np.float32)
    zs = np.float32(abs(scale) * 1.4426950408889634)
    sign = np.float32(-1.0 if scale < 0 else 1.0)
    half = (np.arange(32) >> 2) & 1
    t0 = 0
    for n in L:
        n = int(n)
        for h in range(H):
            K = kf[t0:t0 + n, h * 64:(h + 1) * 64]
            V = vf[t0:t0 + n, h * 64:(h + 1) * 64]
            for r0 in range(0, n, 32):
                Q = qf[t0 + r0:t0 + min(n, r0 + 32), h * 64:(h + 1) * 64] * sign
                m = np.full(Q.shape[0], -np.inf, np.float32)
                lsum = np.zeros(Q.shape[0], np.float32)
                o = np.zeros((Q.shape[0], 64), np.float32)
                for c in range(0, n, 32):
                    s = (Q @ K[c:c + 32].T).astype(np.float32)  # [rows, keys of the chunk]
                    z = s * zs
                    if c == 0:
                        m = z.max(1)
                    e = np.exp2(z - m[:, None]).astype(np.float32)
                    if c > 0:
                        hk = half[:s.shape[1]]
                        ps = np.stack([e[:, hk == 0].sum(1), e[:, hk == 1].sum(1)], 1)
                        if not (ps <= cap).all():
                            if stats is not None:
                                stats["raises"] = stats.get("raises", 0) + 1
                            mn = np.maximum(m, z.max(1))
                            alpha = np.exp2(m - mn).astype(np.float32)
                            lsum *= alpha
                            o *= alpha[:, None]
                            m = mn
                            e = np.exp2(z - m[:, None]).astype(np.float32)
                    lsum += e.sum(1, dtype=np.float32)
                    o += _rd(e) @ V[c:c + 32]
                out[t0 + r0:t0 + r0 + Q.shape[0], h * 64:(h + 1) * 64] = o / lsum[:, None]
        t0 += n
    return out


CASES = [([1, 15, 16, 17, 63, 64, 65, 127, 129, 200], 1, 0.5), ([1, 15, 16, 17, 63, 64, 65, 127, 129, 200], 4, 4.0),
         ([0, 7, 0, 300, 2], 4, 0.5), ([8, 64, 9, 384, 511], 1, 4.0), ([700, 40, 3], 2, 1.0)]


@pytest.mark.parametrize("Ls,H,qscale", CASES)
def test_fused_rounding_emulation_meets_the_fused_bound(Ls, H, qscale):
    L = np.array(Ls, np.int32)
    T, d = int(L.sum()), H * 64
    rng = np.random.default_rng(T + H)
    q, k = (random_storage(rng, (T, d), "bf16", qscale) for _ in range(2))
    v = random_storage(rng, (T, d), "bf16", 1.0)
    scale = 0.125
    got = _rd(_fused_emulation(L, H, q, k, v, scale)).astype(np.float64)  # the kernel stores bf16
    q32, k32, v32 = (bf16_bits_to_f32(a).reshape(T, d).astype(np.float32) for a in (q, k, v))
    P = oracle.softmax("f32", L, H, oracle.qkt("f32", L, H, 64, q32, d, k32, d, scale))
    exact = np.asarray(oracle.attn_v("f32", L, H, 64, P, v32, d), np.float64).reshape(T, d)
    mag = np.asarray(oracle.attn_v("f32", L, H, 64, P, np.abs(v32), d), np.float64).reshape(T, d)
    err = np.abs(got - exact)
    assert (err - (BF16_ATOL + BF16_RTOL * mag)).max() <= 0
    assert err.mean() <= 4e-3 * mag.mean()


def test_fused_emulation_with_raised_references_meets_the_fused_bound():
    # scores rising by 16 nats per chunk of 32 keys: every later chunk takes the
    # raise path (recomputed scores, raised reference, rescaled sums), whose extra
    # rescaling must stay within the same bound
    L = np.array([700, 512, 33, 64, 95], np.int32)
    H = 2
    T, d = int(L.sum()), H * 64
    q, k, v = rising_keys(L, H, 16.0, seed=7)
    stats = {}
    got = _rd(_fused_emulation(L, H, q, k, v, 0.125, stats=stats)).astype(np.float64)
    blocks = sum(H * ((n + 31) // 32) * ((n + 31) // 32 - 1) for n in L.tolist())
    assert stats["raises"] == blocks  # every later chunk of every 32-row block
    q32, k32, v32 = (bf16_bits_to_f32(a).reshape(T, d).astype(np.float32) for a in (q, k, v))
    P = oracle.softmax("f32", L, H, oracle.qkt("f32", L, H, 64, q32, d, k32, d, 0.125))
    exact = np.asarray(oracle.attn_v("f32", L, H, 64, P, v32, d), np.float64).reshape(T, d)
    mag = np.asarray(oracle.attn_v("f32", L, H, 64, P, np.abs(v32), d), np.float64).reshape(T, d)
    err = np.abs(got - exact)
    assert (err - (BF16_ATOL + BF16_RTOL * mag)).max() <= 0
    assert err.mean() <= 4e-3 * mag.mean()


def test_fused_rounding_misses_the_elementwise_bound_against_the_rounded_chain():
    # large scores (peaked rows): the chain rounds scores to bf16 before the
    # softmax, the fused kernel keeps them in fp32, so individual outputs move
    # by more than 2e-2 of themselves although both are within rounding of
    # exact attention
    L = np.array([8, 64, 9, 384, 511], np.int32)
    H = 1
    T, d = int(L.sum()), 64
    rng = np.random.default_rng(T + H)
    q, k = (random_storage(rng, (T, d), "bf16", 4.0) for _ in range(2))
    v = random_storage(rng, (T, d), "bf16", 1.0)
    got = _rd(_fused_emulation(L, H, q, k, v, 0.125)).astype(np.float64)
    S = oracle.qkt("bf16", L, H, 64, q, d, k, d, 0.125)
    chain = values(oracle.attn_v("bf16", L, H, 64, oracle.softmax("bf16", L, H, S), v, d), "bf16").reshape(T, d)
    assert (np.abs(got - chain) - (BF16_ATOL + BF16_RTOL * np.abs(chain))).max() > 0


@pytest.mark.parametrize("cid", [3, 5])
def test_emulated_fused_layer_statistics(cid):
    # the GPU layer's arithmetic (fp32 products, bf16 interface tensors, fused
    # attention) emulated on the CPU: the row-scaled bound holds with a margin,
    # each row's mean error stays under ROW_MEAN_TOL, and the element-wise bound
    # fails on a small fraction of elements only -- the levels the GPU tests assert
    wl = make_workload(cid, seed=0, random_ln=True)
    cfg = wl.cfg
    L = wl.lengths
    st = np.concatenate([[0], np.cumsum(L)])
    w = {n: wl.tensors[n] for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    fails = 0
    for b in sorted(set(np.linspace(0, len(L) - 1, 4).round().astype(int).tolist())):
        xs = wl.tensors["x"][st[b]:st[b + 1]]
        ref = oracle.encoder_layer("bf16", L[b:b + 1], xs, w, cfg.d_model, cfg.heads, cfg.d_ff)
        got = _layer_fp32(xs, w, cfg.d_model, cfg.heads, cfg.d_ff, fused=True)
        bits = torch.from_numpy(got).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        stats = bf16_row_stats(bits, ref, cfg.d_model)
        assert stats["row_excess"] < -1e-2 and stats["row_mean"] <= ROW_MEAN_TOL / 2, (b, stats)
        assert stats["elem_pass"] >= ELEM_PASS_MIN, (b, stats)
        fails += stats["elem_pass"] < 1.0
    assert fails > 0  # the element-wise bound does not hold for the fused arithmetic
