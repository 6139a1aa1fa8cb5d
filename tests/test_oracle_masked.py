"""Pins of the oracle's masked (causal) attention: position i sees keys j <= i,
the decoder variant of the layer (Section 7.2; Appendix D, masked SDPA).  Checked
against a brute-force dense masked attention, torch's causal SDPA, the prefix
property (row i of a masked sequence is row i of the unmasked attention over its
first i + 1 tokens) and special cases (the first row returns V exactly; entries
above the diagonal are never written)."""
import math

import numpy as np
import pytest
import torch

import oracle
from tests.test_oracle_numerics import BF16, F32, _pack_qkv, _split, val


def _brute_force_causal(L, H, dh, q, k, v, scale):
    """Dense per-sequence attention with an explicit lower-triangular mask (fp64)."""
    out, scores, probs = np.zeros((int(np.sum(L)), H * dh)), [], []
    t = 0
    for n in L:
        n = int(n)
        Q = q[t:t + n].reshape(n, H, dh)
        K = k[t:t + n].reshape(n, H, dh)
        V = v[t:t + n].reshape(n, H, dh)
        S = np.einsum("ihc,jhc->ihj", Q, K) * scale                      # [i, h, j]
        allowed = np.arange(n)[None, :] <= np.arange(n)[:, None]           # [i, j]
        Sm = np.where(allowed[:, None, :], S, -np.inf)
        P = np.exp(Sm - Sm.max(-1, keepdims=True)) if n else Sm
        P = P / P.sum(-1, keepdims=True) if n else P
        out[t:t + n] = np.einsum("ihj,jhc->ihc", P, V).reshape(n, H * dh)
        scores.append((S, allowed))
        probs.append(P)
        t += n
    return scores, probs, out


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("L,H,dh", [([7, 33, 64, 128], 2, 64), ([1, 2, 15, 16, 17], 1, 8), ([31, 0, 32, 65], 2, 8)])
def test_masked_sdpa_matches_brute_force(dtype, L, H, dh):
    rng = np.random.default_rng(sum(L) + 7 * H)
    q, k, v = _pack_qkv(rng, L, H, dh, dtype, 0.7)
    scale = 1.0 / math.sqrt(dh)
    S = oracle.qkt(dtype, L, H, dh, q, H * dh, k, H * dh, scale, causal=True)
    P = oracle.softmax(dtype, L, H, S, causal=True)
    O = oracle.attn_v(dtype, L, H, dh, P, v, H * dh, causal=True)
    bs, bp, _ = _brute_force_causal(L, H, dh, val(q, dtype), val(k, dtype), val(v, dtype), scale)
    tol = 2.0 ** -8 if dtype == BF16 else 2.0 ** -23
    for got, (ref, allowed), p_got in zip(_split(val(S, dtype), L, H), bs, _split(val(P, dtype), L, H)):
        a = np.broadcast_to(allowed[:, None, :], got.shape)
        assert np.all(np.abs(got[a] - ref[a]) <= tol * np.abs(ref[a]) + 1e-12)
        assert np.all(got[~a] == 0) and np.all(p_got[~a] == 0)  # never written
    # softmax from the stored scores, masked entries excluded
    for got, s, (_, allowed) in zip(_split(val(P, dtype), L, H), _split(val(S, dtype), L, H), bs):
        if s.size == 0:
            continue
        sm = np.where(allowed[:, None, :], s, -np.inf)
        e = np.exp(sm - sm.max(-1, keepdims=True))
        ref = e / e.sum(-1, keepdims=True)
        assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 1e-12)
    # Attn.V from the stored probabilities over j <= i
    t = 0
    Vd = val(v, dtype)
    for b, (n, p) in enumerate(zip(L, _split(val(P, dtype), L, H))):
        if n == 0:
            continue
        ref = np.einsum("ihj,jhc->ihc", p, Vd[t:t + n].reshape(n, H, dh)).reshape(n, H * dh)
        got = val(O, dtype)[t:t + n]
        assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 4 * tol * 1e-3 * np.abs(Vd).max() + 1e-12)
        t += n


def test_masked_matches_torch_causal_sdpa():
    rng = np.random.default_rng(21)
    L, H, dh = [40, 1, 77], 2, 64
    q, k, v = _pack_qkv(rng, L, H, dh, F32, 2.0)
    scale = 0.125
    O = val(oracle.attn_v(F32, L, H, dh, oracle.softmax(F32, L, H, oracle.qkt(F32, L, H, dh, q, H * dh, k, H * dh,
                                                                            scale, causal=True), causal=True),
                          v, H * dh, causal=True), F32)
    t = 0
    for n in L:
        to4 = lambda a: torch.from_numpy(val(a, F32)[t:t + n].reshape(1, n, H, dh).transpose(0, 2, 1, 3).astype(np.float64))
        ref = torch.nn.functional.scaled_dot_product_attention(to4(q), to4(k), to4(v), scale=scale, is_causal=True)
        assert np.allclose(O[t:t + n], ref.numpy().transpose(0, 2, 1, 3).reshape(n, H * dh), rtol=1e-5, atol=1e-6)
        t += n


def test_masked_row_is_unmasked_attention_over_the_prefix():
    # row i of a masked sequence = row i of ordinary attention over its first i + 1 tokens
    rng = np.random.default_rng(22)
    n, H, dh = 23, 3, 16
    q, k, v = _pack_qkv(rng, [n], H, dh, F32, 1.5)
    scale = 0.3
    O = oracle.attn_v(F32, [n], H, dh, oracle.softmax(F32, [n], H, oracle.qkt(F32, [n], H, dh, q, H * dh, k, H * dh,
                                                                            scale, causal=True), causal=True),
                      v, H * dh, causal=True)
    for i in (0, 1, 7, n - 1):
        m = i + 1
        Sp = oracle.qkt(F32, [m], H, dh, q[:m], H * dh, k[:m], H * dh, scale)
        Op = oracle.attn_v(F32, [m], H, dh, oracle.softmax(F32, [m], H, Sp), v[:m], H * dh)
        assert np.array_equal(O[i], Op[i])


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_masked_first_row_returns_v(dtype):
    rng = np.random.default_rng(23)
    L, H, dh = [5, 1, 9], 2, 8
    q, k, v = _pack_qkv(rng, L, H, dh, dtype, 3.0)
    P = oracle.softmax(dtype, L, H, oracle.qkt(dtype, L, H, dh, q, H * dh, k, H * dh, 1.0, causal=True), causal=True)
    O = oracle.attn_v(dtype, L, H, dh, P, v, H * dh, causal=True)
    for t in (0, 5, 6):  # position 0 of each sequence sees only itself
        assert np.array_equal(O[t], v[t])


def test_masked_layer_matches_torch_decoder_style_layer():
    # the layer with masked attention against torch's encoder layer with a causal mask, per sequence, fp64
    rng = np.random.default_rng(24)
    L, d, H, dff = [9, 1, 30], 64, 4, 128
    from workloads import BIAS_NAMES, LN_NAMES, WEIGHT_NAMES, layer_param_shapes
    shapes = layer_param_shapes(d, dff)
    w = {nm: (rng.standard_normal(shapes[nm]) * (0.1 if nm in WEIGHT_NAMES else 0.05)).astype(np.float32)
         for nm in WEIGHT_NAMES + BIAS_NAMES}
    w.update({nm: (1.0 + 0.1 * rng.standard_normal(shapes[nm]) if nm.endswith("_g") else
                   0.1 * rng.standard_normal(shapes[nm])).astype(np.float32) for nm in LN_NAMES})
    x = rng.standard_normal((sum(L), d)).astype(np.float32)
    got = oracle.encoder_layer(F32, L, x, w, d, H, dff, causal=True)
    layer = torch.nn.TransformerEncoderLayer(d, H, dff, dropout=0.0, activation="gelu", batch_first=True,
                                             norm_first=False).double().eval()
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(torch.from_numpy(w["w_qkv"]))
        layer.self_attn.in_proj_bias.copy_(torch.from_numpy(w["b_qkv"]))
        layer.self_attn.out_proj.weight.copy_(torch.from_numpy(w["w_o"]))
        layer.self_attn.out_proj.bias.copy_(torch.from_numpy(w["b_o"]))
        layer.linear1.weight.copy_(torch.from_numpy(w["w_ff1"]))
        layer.linear1.bias.copy_(torch.from_numpy(w["b_ff1"]))
        layer.linear2.weight.copy_(torch.from_numpy(w["w_ff2"]))
        layer.linear2.bias.copy_(torch.from_numpy(w["b_ff2"]))
        layer.norm1.weight.copy_(torch.from_numpy(w["ln1_g"]))
        layer.norm1.bias.copy_(torch.from_numpy(w["ln1_b"]))
        layer.norm2.weight.copy_(torch.from_numpy(w["ln2_g"]))
        layer.norm2.bias.copy_(torch.from_numpy(w["ln2_b"]))
        t = 0
        for n in L:
            mask = torch.triu(torch.full((n, n), float("-inf"), dtype=torch.float64), diagonal=1)
            ref = layer(torch.from_numpy(x[t:t + n].astype(np.float64))[None], src_mask=mask)[0].numpy()
            assert np.allclose(got[t:t + n], ref, rtol=1e-4, atol=1e-5), np.abs(got[t:t + n] - ref).max()
            t += n
