"""Pins of the oracle's arithmetic.

The oracle is checked against things other than itself: a brute-force
padded-and-masked dense attention (numpy), library routines (numpy matmul,
torch's CPU LayerNorm / GELU / scaled_dot_product_attention /
TransformerEncoderLayer in float64), hand-worked bf16 rounding cases, and
invariants of the method (rows of P sum to 1, one-token sequences, uniform
lengths reduce to dense batched attention, sequences are independent, and the
layer is equivariant under permutations of the batch).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from workloads import bf16_bits_to_f32, storage_to_f64, to_bf16_bits

F32, BF16 = "f32", "bf16"


def val(a, dtype):
    return storage_to_f64(a, dtype)


def store(x, dtype):
    return np.ascontiguousarray(x, np.float32) if dtype == F32 else to_bf16_bits(x)


def half_ulp(z, dtype):
    """Half the spacing of the storage format at |z| (normal range): a correctly
    rounded result is within this of the exact value."""
    bits = 8 if dtype == BF16 else 24
    e = np.floor(np.log2(np.maximum(np.abs(z), 1e-300)))
    return np.ldexp(1.0, (e - bits).astype(int))


# ----------------------------------------------------------------------------
# bf16 rounding
# ----------------------------------------------------------------------------

def test_bf16_hand_worked_cases():
    cases = {
        1.0: 0x3F80,
        1.0 + 2.0 ** -7: 0x3F81,
        1.0 + 2.0 ** -8: 0x3F80,              # tie -> even (0x3F80)
        1.0 + 3 * 2.0 ** -8: 0x3F82,          # tie -> even (0x3F82)
        1.0 + 2.0 ** -8 + 2.0 ** -30: 0x3F81,  # just above the tie (not a float32 value)
        -2.0: 0xC000,
        2.0 ** -133: 0x0001,                  # smallest subnormal
        2.0 ** -134: 0x0000,                  # half of it: tie -> even (zero)
        3 * 2.0 ** -134: 0x0002,              # 1.5 quanta: tie -> even (2)
        (2 - 2.0 ** -7) * 2.0 ** 127: 0x7F7F,  # largest finite
        (2 - 2.0 ** -8) * 2.0 ** 127: 0x7F80,  # halfway to 2^128: tie -> even -> inf
        math.inf: 0x7F80,
        -math.inf: 0xFF80,
        0.0: 0x0000,
    }
    xs = np.array(list(cases.keys()), np.float64)
    got = oracle.round_bf16(xs)
    assert [hex(v) for v in got.tolist()] == [hex(v) for v in cases.values()]
    assert oracle.round_bf16(np.array([math.nan]))[0] & 0x7FFF > 0x7F80


def test_bf16_matches_torch_on_float32_values():
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-40, 38, 20000),
        # float32 values exactly halfway between two bf16 values
        (bf16_bits_to_f32(rng.integers(0, 0x7F00, 5000).astype(np.uint16)).view(np.uint32) | 0x8000).view(np.float32),
    ]).astype(np.float32)
    ref = to_bf16_bits(x)  # torch's CPU float32 -> bfloat16 (round to nearest even)
    got = oracle.round_bf16(x.astype(np.float64))
    assert (got == ref).all()


def test_bf16_brute_force_on_float64_values():
    # doubles that are not float32 values: pick the nearest of the neighbouring
    # bf16 values by exact comparison, ties to the even bit pattern
    rng = np.random.default_rng(2)
    x = rng.standard_normal(3000) * 10.0 ** rng.integers(-30, 30, 3000)
    got = oracle.round_bf16(x)
    for v, g in zip(x.tolist(), got.tolist()):
        base = int(np.float32(v).view(np.uint32)) >> 16
        cands = [c for c in range(base - 2, base + 3) if 0 <= c < 0x10000]
        vals = [float(bf16_bits_to_f32(np.array([c], np.uint16))[0]) for c in cands]
        dist = [abs(cv - v) for cv in vals]
        best = min(dist)
        winners = [c for c, dd in zip(cands, dist) if dd == best]
        want = winners[0] if len(winners) == 1 else [c for c in winners if c % 2 == 0][0]
        assert g == want, (v, hex(g), hex(want))


# ----------------------------------------------------------------------------
# Token-wise operators
# ----------------------------------------------------------------------------

def _gelu_erf(x):
    return 0.5 * x * (1.0 + np.vectorize(math.erf)(x / math.sqrt(2.0)))


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("act", [oracle.ACT_NONE, oracle.ACT_GELU_ERF, oracle.ACT_GELU_TANH])
@pytest.mark.parametrize("with_bias,with_res", [(True, True), (True, False), (False, True), (False, False)])
def test_linear_matches_numpy(dtype, act, with_bias, with_res):
    rng = np.random.default_rng(3)
    T, K, N = 37, 48, 24  # non-square: a transposed operand cannot line up
    x = store(rng.standard_normal((T, K)), dtype)
    w = store(rng.standard_normal((N, K)) * 0.2, dtype)
    b = store(rng.standard_normal(N), dtype) if with_bias else None
    r = store(rng.standard_normal((T, N)), dtype) if with_res else None
    y = oracle.linear(dtype, x, w, b, r, act)
    z = val(x, dtype) @ val(w, dtype).T
    if with_bias:
        z = z + val(b, dtype)
    if act == oracle.ACT_GELU_ERF:
        z = _gelu_erf(z)
    elif act == oracle.ACT_GELU_TANH:
        z = torch.nn.functional.gelu(torch.from_numpy(z), approximate="tanh").numpy()
    if with_res:
        z = z + val(r, dtype)
    err = np.abs(val(y, dtype) - z)
    assert (err <= half_ulp(z, dtype) * 1.0001 + 1e-12).all()


def test_gelu_identities():
    x = np.linspace(-6, 6, 241)
    xs = store(x.reshape(-1, 1), F32)
    one = store(np.ones((1, 1)), F32)
    g = val(oracle.linear(F32, xs, one, act=oracle.ACT_GELU_ERF), F32)[:, 0]
    gm = val(oracle.linear(F32, store(-x.reshape(-1, 1), F32), one, act=oracle.ACT_GELU_ERF), F32)[:, 0]
    # GELU(x) - GELU(-x) = x, GELU(0) = 0, and GELU(x) -> x for large x
    assert np.allclose(g - gm, x, atol=1e-6)
    assert g[120] == 0.0
    assert abs(g[-1] - 6.0) < 1e-6
    ref = torch.nn.functional.gelu(torch.from_numpy(x)).numpy()
    assert np.allclose(g, ref, rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_layernorm_matches_torch(dtype):
    rng = np.random.default_rng(4)
    T, d = 19, 96
    x = store(rng.standard_normal((T, d)) * 3 + 1, dtype)
    g = store(1 + 0.1 * rng.standard_normal(d), dtype)
    b = store(0.1 * rng.standard_normal(d), dtype)
    y = oracle.layernorm(dtype, x, g, b, 1e-5)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(val(x, dtype)), (d,),
                                         torch.from_numpy(val(g, dtype)), torch.from_numpy(val(b, dtype)),
                                         eps=1e-5).numpy()
    assert (np.abs(val(y, dtype) - ref) <= half_ulp(ref, dtype) * 1.0001 + 1e-9).all()


def test_layernorm_moments():
    rng = np.random.default_rng(5)
    T, d = 11, 512
    x = store(rng.standard_normal((T, d)) * 5 - 2, F32)
    y = val(oracle.layernorm(F32, x, store(np.ones(d), F32), store(np.zeros(d), F32), 1e-5), F32)
    assert np.allclose(y.mean(1), 0, atol=1e-6)
    assert np.allclose(y.var(1), 1, atol=1e-5)


# ----------------------------------------------------------------------------
# Scaled dot-product attention on ragged storage
# ----------------------------------------------------------------------------

def _pack_qkv(rng, L, H, dh, dtype, scale=1.0):
    T = int(np.sum(L))
    return [store(rng.standard_normal((T, H * dh)) * scale, dtype) for _ in range(3)]


def _brute_force_sdpa(L, H, dh, q, k, v, scale):
    """Pad every sequence to max(L), mask padded keys with -inf, run dense
    attention, then keep the real rows.  Returns per-sequence score blocks
    [L, H, L] (the paper's X[b][i][h][j] layout), probabilities likewise, and
    the packed output [T, H*dh]."""
    B, Lm = len(L), int(max(L)) if len(L) else 0
    T = int(np.sum(L))
    Qp = np.zeros((B, Lm, H, dh)); Kp = np.zeros_like(Qp); Vp = np.zeros_like(Qp)
    t = 0
    for b, n in enumerate(L):
        Qp[b, :n] = q[t:t + n].reshape(n, H, dh)
        Kp[b, :n] = k[t:t + n].reshape(n, H, dh)
        Vp[b, :n] = v[t:t + n].reshape(n, H, dh)
        t += n
    S = np.einsum("bihc,bjhc->bhij", Qp, Kp) * scale
    mask = np.arange(Lm)[None, :] < np.asarray(L)[:, None]          # [B, Lm] real keys
    Sm = np.where(mask[:, None, None, :], S, -np.inf)
    P = np.exp(Sm - Sm.max(-1, keepdims=True))
    P = P / P.sum(-1, keepdims=True)
    O = np.einsum("bhij,bjhc->bihc", np.nan_to_num(P), Vp)
    scores, probs, out = [], [], np.zeros((T, H * dh))
    t = 0
    for b, n in enumerate(L):
        scores.append(S[b, :, :n, :n].transpose(1, 0, 2))   # [i, h, j]
        probs.append(P[b, :, :n, :n].transpose(1, 0, 2))
        out[t:t + n] = O[b, :n].reshape(n, H * dh)
        t += n
    return scores, probs, out


def _split(flat, L, H):
    out, o = [], 0
    for n in L:
        n = int(n)
        out.append(flat[o:o + H * n * n].reshape(n, H, n))   # X[b] = [i][h][j]
        o += H * n * n
    return out


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("L,H,dh", [
    ([7, 33, 64, 128], 2, 64),
    ([1, 2, 15, 16, 17], 1, 8),
    ([31, 0, 32, 33, 65], 2, 8),
    ([64], 2, 64),
])
def test_sdpa_matches_brute_force(dtype, L, H, dh):
    rng = np.random.default_rng(sum(L) + H)
    q, k, v = _pack_qkv(rng, L, H, dh, dtype, 0.7)
    scale = 1.0 / math.sqrt(dh)
    S = oracle.qkt(dtype, L, H, dh, q, H * dh, k, H * dh, scale)
    P = oracle.softmax(dtype, L, H, S)
    O = oracle.attn_v(dtype, L, H, dh, P, v, H * dh)
    # each operator against the brute force fed with the oracle's own stored input
    bs, _, _ = _brute_force_sdpa(L, H, dh, val(q, dtype), val(k, dtype), val(v, dtype), scale)
    tol = 2.0 ** -8 if dtype == BF16 else 2.0 ** -23
    for got, ref in zip(_split(val(S, dtype), L, H), bs):
        assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 1e-12)
    Sd = _split(val(S, dtype), L, H)
    for got, s in zip(_split(val(P, dtype), L, H), Sd):
        if s.size == 0:
            continue
        e = np.exp(s - s.max(-1, keepdims=True))
        ref = e / e.sum(-1, keepdims=True)
        assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 1e-12)
    # Attn.V: brute force from the stored P (dense, padded with zero probabilities)
    Pd = _split(val(P, dtype), L, H)
    Vd = val(v, dtype)
    t = 0
    for b, n in enumerate(L):
        if n == 0:
            continue
        ref = np.einsum("ihj,jhc->ihc", Pd[b], Vd[t:t + n].reshape(n, H, dh)).reshape(n, H * dh)
        got = val(O, dtype)[t:t + n]
        scale_ref = np.abs(Pd[b]).sum(-1).max() * (np.abs(Vd).max() if Vd.size else 0)
        assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 4 * tol * 1e-3 * scale_ref + 1e-12)
        t += n


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_softmax_rows_sum_to_one(dtype):
    rng = np.random.default_rng(9)
    L, H = [5, 40, 130], 3
    S = store(rng.standard_normal(oracle.score_elems(L, H)) * 4, dtype)
    P = _split(val(oracle.softmax(dtype, L, H, S), dtype), L, H)
    tol = 1e-2 if dtype == BF16 else 1e-6
    for p in P:
        assert np.all(np.abs(p.sum(-1) - 1) <= tol)
        assert np.all(p >= 0)


def test_single_token_sequences():
    rng = np.random.default_rng(10)
    L, H, dh = [1, 1, 3, 1], 2, 16
    q, k, v = _pack_qkv(rng, L, H, dh, BF16)
    S = oracle.qkt(BF16, L, H, dh, q, H * dh, k, H * dh, 0.25)
    P = oracle.softmax(BF16, L, H, S)
    O = oracle.attn_v(BF16, L, H, dh, P, v, H * dh)
    Pd = _split(val(P, BF16), L, H)
    for b in (0, 1, 3):
        assert (Pd[b] == 1.0).all()
    for t in (0, 1, 5):   # the one-token sequences' rows: O = V exactly
        assert (O[t] == v[t]).all()


def test_uniform_lengths_equal_dense_batched_attention():
    rng = np.random.default_rng(11)
    B, n, H, dh = 3, 24, 4, 16
    L = [n] * B
    q, k, v = _pack_qkv(rng, L, H, dh, F32)
    scale = 1.0 / math.sqrt(dh)
    S = oracle.qkt(F32, L, H, dh, q, H * dh, k, H * dh, scale)
    P = oracle.softmax(F32, L, H, S)
    O = val(oracle.attn_v(F32, L, H, dh, P, v, H * dh), F32)
    to4 = lambda a: torch.from_numpy(val(a, F32).reshape(B, n, H, dh).transpose(0, 2, 1, 3).copy())
    ref = torch.nn.functional.scaled_dot_product_attention(to4(q), to4(k), to4(v), scale=scale)
    ref = ref.numpy().transpose(0, 2, 1, 3).reshape(B * n, H * dh)
    assert np.allclose(O, ref, rtol=1e-5, atol=1e-6)


def test_single_sequence_matches_torch_sdpa():
    rng = np.random.default_rng(12)
    n, H, dh = 77, 2, 64
    q, k, v = _pack_qkv(rng, [n], H, dh, F32, 2.0)
    scale = 1.0 / 8.0
    S = oracle.qkt(F32, [n], H, dh, q, H * dh, k, H * dh, scale)
    O = val(oracle.attn_v(F32, [n], H, dh, oracle.softmax(F32, [n], H, S), v, H * dh), F32)
    to4 = lambda a: torch.from_numpy(val(a, F32).reshape(1, n, H, dh).transpose(0, 2, 1, 3).copy())
    ref = torch.nn.functional.scaled_dot_product_attention(to4(q), to4(k), to4(v), scale=scale)
    assert np.allclose(O, ref.numpy().transpose(0, 2, 1, 3).reshape(n, H * dh), rtol=1e-5, atol=1e-6)


def test_strided_qkv_views():
    # Q, K, V as column blocks of one [T, 3d] buffer (the layer's layout)
    rng = np.random.default_rng(13)
    L, H, dh = [9, 21], 2, 8
    d = H * dh
    T = sum(L)
    qkv = store(rng.standard_normal((T, 3 * d)), BF16)
    q, k, v = (np.ascontiguousarray(qkv[:, i * d:(i + 1) * d]) for i in range(3))
    S1 = oracle.qkt(BF16, L, H, dh, q, d, k, d, 0.3)
    S2 = oracle.qkt(BF16, L, H, dh, qkv, 3 * d, qkv.reshape(-1)[d:], 3 * d, 0.3)
    # passing a buffer starting at column d with stride 3d reads the K block
    assert (S1 == S2).all()


# ----------------------------------------------------------------------------
# The encoder layer
# ----------------------------------------------------------------------------

def _layer_weights(rng, d, dff, dtype):
    sh = {"w_qkv": (3 * d, d), "b_qkv": (3 * d,), "w_o": (d, d), "b_o": (d,),
          "ln1_g": (d,), "ln1_b": (d,), "w_ff1": (dff, d), "b_ff1": (dff,),
          "w_ff2": (d, dff), "b_ff2": (d,), "ln2_g": (d,), "ln2_b": (d,)}
    w = {}
    for name, s in sh.items():
        if name.endswith("_g"):
            w[name] = store(1 + 0.1 * rng.standard_normal(s), dtype)
        elif name.startswith("ln"):
            w[name] = store(0.1 * rng.standard_normal(s), dtype)
        else:
            w[name] = store(rng.standard_normal(s) * (0.1 if name.startswith("w") else 0.05), dtype)
    return w


def _torch_layer(w, d, H, dff):
    layer = torch.nn.TransformerEncoderLayer(d, H, dff, dropout=0.0, activation="gelu",
                                             layer_norm_eps=1e-5, batch_first=True,
                                             norm_first=False).double().eval()
    t = lambda n: torch.from_numpy(val(w[n], F32))
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t("w_qkv"))
        layer.self_attn.in_proj_bias.copy_(t("b_qkv"))
        layer.self_attn.out_proj.weight.copy_(t("w_o"))
        layer.self_attn.out_proj.bias.copy_(t("b_o"))
        layer.linear1.weight.copy_(t("w_ff1")); layer.linear1.bias.copy_(t("b_ff1"))
        layer.linear2.weight.copy_(t("w_ff2")); layer.linear2.bias.copy_(t("b_ff2"))
        layer.norm1.weight.copy_(t("ln1_g")); layer.norm1.bias.copy_(t("ln1_b"))
        layer.norm2.weight.copy_(t("ln2_g")); layer.norm2.bias.copy_(t("ln2_b"))
    return layer


def test_layer_matches_torch_encoder_layer_with_padding_mask():
    rng = np.random.default_rng(14)
    L, H, dh, dff = [5, 17, 1, 12], 4, 8, 64
    d = H * dh
    T = sum(L)
    w = _layer_weights(rng, d, dff, F32)
    x = store(rng.standard_normal((T, d)), F32)
    got = val(oracle.encoder_layer(F32, L, x, w, d, H, dff), F32)
    layer = _torch_layer(w, d, H, dff)
    Lm = max(L)
    xp = torch.zeros(len(L), Lm, d, dtype=torch.float64)
    mask = torch.ones(len(L), Lm, dtype=torch.bool)
    t = 0
    for b, n in enumerate(L):
        xp[b, :n] = torch.from_numpy(val(x, F32)[t:t + n])
        mask[b, :n] = False
        t += n
    with torch.no_grad():
        ref = layer(xp, src_key_padding_mask=mask).numpy()
    t = 0
    for b, n in enumerate(L):
        assert np.allclose(got[t:t + n], ref[b, :n], rtol=1e-4, atol=1e-4)
        t += n


def test_layer_bf16_close_to_fp64_torch():
    rng = np.random.default_rng(15)
    L, H, dh, dff = [23], 2, 16, 64
    d = H * dh
    w = _layer_weights(rng, d, dff, BF16)
    x = store(rng.standard_normal((L[0], d)), BF16)
    got = val(oracle.encoder_layer(BF16, L, x, w, d, H, dff), BF16)
    layer = _torch_layer({k: val(v, BF16).astype(np.float32) for k, v in w.items()}, d, H, dff)
    with torch.no_grad():
        ref = layer(torch.from_numpy(val(x, BF16))[None]).numpy()[0]
    assert np.allclose(got, ref, rtol=3e-2, atol=3e-2)


def test_layer_sequence_independence_and_permutation():
    rng = np.random.default_rng(16)
    L, H, dh, dff = [6, 11, 3], 2, 8, 32
    d = H * dh
    w = _layer_weights(rng, d, dff, BF16)
    x = store(rng.standard_normal((sum(L), d)), BF16)
    out = oracle.encoder_layer(BF16, L, x, w, d, H, dff)
    # change sequence 1's tokens: sequences 0 and 2 are unchanged bit for bit
    x2 = x.copy()
    x2[6:17] = store(rng.standard_normal((11, d)), BF16)
    out2 = oracle.encoder_layer(BF16, L, x2, w, d, H, dff)
    assert (out2[:6] == out[:6]).all() and (out2[17:] == out[17:]).all()
    assert not (out2[6:17] == out[6:17]).all()
    # permute the batch: outputs permute bit for bit
    perm = [2, 0, 1]
    starts = np.concatenate([[0], np.cumsum(L)])
    xp = np.concatenate([x[starts[b]:starts[b + 1]] for b in perm])
    outp = oracle.encoder_layer(BF16, [L[b] for b in perm], xp, w, d, H, dff)
    refp = np.concatenate([out[starts[b]:starts[b + 1]] for b in perm])
    assert (outp == refp).all()
