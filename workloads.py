"""Seeded synthetic inputs for the ragged encoder-layer workloads.

This module only draws random numbers and packs them into arrays. It holds none
of the method's arithmetic (no offsets, no products, no reductions), so both the
CPU oracle and the GPU path can be fed from it without sharing any code.

The paper's datasets (sequence-length distributions of RACE, SQuAD, MNLI, ...
in Table "Datasets used in our evaluation") are not available here; the five
configurations below are synthetic stand-ins with the same length ranges
(every length <= 512, as in that table) and the layer shapes of the paper's
Transformer-base evaluation (Section 7.2: d=512, 8 heads of 64, FFN 2048) plus a
larger d=1024 / 16-head / FFN-4096 variant.

Draw order per configuration (fixed, so every consumer sees identical values):
lengths -> activations (X, or Q/K/V) -> weights in interface order
(w_qkv, w_o, w_ff1, w_ff2) -> biases (b_qkv, b_o, b_ff1, b_ff2) -> LayerNorm
gamma/beta (ln1_g, ln1_b, ln2_g, ln2_b).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    kind: str            # "sdpa" (ragged QK^T, softmax, Attn.V only) or "layer"
    dtype: str           # F32 or BF16
    batch: int
    heads: int
    head_dim: int
    d_ff: int            # 0 for sdpa-only configs
    lengths: str         # length recipe, see draw_lengths
    input_scale: float = 1.0
    max_len: int = 512

    @property
    def d_model(self) -> int:
        return self.heads * self.head_dim


CONFIGS = {
    1: Config(1, "mha_fp32_b4", "sdpa", F32, 4, 2, 64, 0, "fixed:7,33,64,128", 1.0 / 8.0, 128),
    2: Config(2, "sdpa_bf16_b32_u16_512", "sdpa", BF16, 32, 8, 64, 0, "uniform:16:512", 1.0 / 8.0),
    3: Config(3, "layer_bf16_b32_lognorm60_d512", "layer", BF16, 32, 8, 64, 2048, "lognormal:60:1.0:512"),
    4: Config(4, "layer_bf16_b128_u32_512_d1024", "layer", BF16, 128, 16, 64, 4096, "uniform:32:512"),
    5: Config(5, "layer_bf16_b128_skew_d512", "layer", BF16, 128, 8, 64, 2048, "skew:8:64:384:512:0.1"),
}


def draw_lengths(recipe: str, batch: int, rng: np.random.Generator) -> np.ndarray:
    """Sequence lengths for one batch, as int32.

    fixed:a,b,..          the listed lengths
    uniform:lo:hi         integers uniform in [lo, hi]
    lognormal:med:s:max   round(exp(N(ln med, s))); redrawn until in [1, max]
    skew:a:b:c:e:frac     round(frac*batch) lengths uniform in [c, e], the rest
                          uniform in [a, b], then shuffled
    """
    kind, _, rest = recipe.partition(":")
    if kind == "fixed":
        out = np.array([int(v) for v in rest.split(",")], dtype=np.int32)
        assert out.size == batch
        return out
    if kind == "uniform":
        lo, hi = (int(v) for v in rest.split(":"))
        return rng.integers(lo, hi + 1, size=batch, dtype=np.int64).astype(np.int32)
    if kind == "lognormal":
        med, sigma, mx = rest.split(":")
        mu, sigma, mx = math.log(float(med)), float(sigma), int(mx)
        out = np.empty(batch, dtype=np.int32)
        for b in range(batch):
            while True:
                v = int(np.rint(rng.lognormal(mu, sigma)))
                if 1 <= v <= mx:
                    out[b] = v
                    break
        return out
    if kind == "skew":
        a, b, c, e, frac = rest.split(":")
        n_long = int(round(float(frac) * batch))
        short = rng.integers(int(a), int(b) + 1, size=batch - n_long, dtype=np.int64)
        long_ = rng.integers(int(c), int(e) + 1, size=n_long, dtype=np.int64)
        out = np.concatenate([short, long_]).astype(np.int32)
        rng.shuffle(out)
        return out
    raise ValueError(f"unknown length recipe {recipe!r}")


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round values to bfloat16 (torch's CPU conversion) and return the raw bits as uint16."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def as_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float array to the storage dtype: float32 array, or uint16 bf16 bits."""
    if dtype == F32:
        return np.ascontiguousarray(x, dtype=np.float32)
    return to_bf16_bits(x)


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact value of a stored array as float64."""
    if dtype == F32:
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    return bf16_bits_to_f32(a).astype(np.float64)


@dataclass
class Workload:
    cfg: Config
    lengths: np.ndarray                       # int32 [B]
    tensors: dict = field(default_factory=dict)  # name -> storage array (float32 or uint16 bits)

    @property
    def total_tokens(self) -> int:
        return int(self.lengths.sum())


WEIGHT_NAMES = ("w_qkv", "w_o", "w_ff1", "w_ff2")
BIAS_NAMES = ("b_qkv", "b_o", "b_ff1", "b_ff2")
LN_NAMES = ("ln1_g", "ln1_b", "ln2_g", "ln2_b")


def layer_param_shapes(d: int, d_ff: int) -> dict:
    return {
        "w_qkv": (3 * d, d), "w_o": (d, d), "w_ff1": (d_ff, d), "w_ff2": (d, d_ff),
        "b_qkv": (3 * d,), "b_o": (d,), "b_ff1": (d_ff,), "b_ff2": (d,),
        "ln1_g": (d,), "ln1_b": (d,), "ln2_g": (d,), "ln2_b": (d,),
    }


def make_workload(cid: int, seed: int = 0, lengths: np.ndarray | None = None,
                  random_ln: bool = False, weight_std: float = 0.02,
                  x_scale: float | None = None) -> Workload:
    """Draw one configuration's inputs.

    `lengths` overrides the recipe (same model shape, caller-chosen raggedness).
    `random_ln` draws gamma ~ 1 + N(0, 0.1) and beta ~ N(0, 0.1) instead of 1 / 0.
    `x_scale` overrides the activation scale (e.g. large-magnitude SDPA inputs).
    """
    cfg = CONFIGS[cid]
    rng = np.random.default_rng(seed)
    lens = draw_lengths(cfg.lengths, cfg.batch, rng)
    if lengths is not None:
        lens = np.asarray(lengths, dtype=np.int32)
    T = int(lens.sum())
    d = cfg.d_model
    scale = cfg.input_scale if x_scale is None else x_scale
    wl = Workload(cfg, lens)
    if cfg.kind == "sdpa":
        for name in ("q", "k", "v"):
            wl.tensors[name] = as_storage(rng.standard_normal((T, d)) * scale, cfg.dtype)
        return wl
    wl.tensors["x"] = as_storage(rng.standard_normal((T, d)) * scale, cfg.dtype)
    shapes = layer_param_shapes(d, cfg.d_ff)
    for name in WEIGHT_NAMES + BIAS_NAMES:
        wl.tensors[name] = as_storage(rng.standard_normal(shapes[name]) * weight_std, cfg.dtype)
    for name in LN_NAMES:
        if random_ln:
            base = 1.0 if name.endswith("_g") else 0.0
            v = base + 0.1 * rng.standard_normal(shapes[name])
        else:
            v = np.ones(shapes[name]) if name.endswith("_g") else np.zeros(shapes[name])
        wl.tensors[name] = as_storage(v, cfg.dtype)
    return wl


def random_storage(rng: np.random.Generator, shape, dtype: str, scale: float = 1.0) -> np.ndarray:
    """A standalone seeded N(0, scale^2) tensor in storage form."""
    return as_storage(rng.standard_normal(shape) * scale, dtype)


# ---------------------------------------------------------------------------
# Variable-sized batched GEMM (the paper's matrix-multiplication experiment,
# Section 7.1): every m, n and k drawn uniformly from the multiples of 128 in
# [512, 1408]; operands N(0, 1), packed one problem after another.
# ---------------------------------------------------------------------------
VGEMM_DIM_CHOICES = np.arange(512, 1408 + 1, 128)


def draw_vgemm_dims(batch: int, rng: np.random.Generator) -> np.ndarray:
    """[batch, 3] int32 (m, n, k), each uniform over VGEMM_DIM_CHOICES."""
    return rng.choice(VGEMM_DIM_CHOICES, size=(batch, 3)).astype(np.int32)


def make_vgemm_operands(dims, rng: np.random.Generator, dtype: str, scale: float = 1.0):
    """Packed A (sum m k elements) and B (sum n k elements) storage arrays."""
    d = np.asarray(dims, np.int64).reshape(-1, 3)
    a = random_storage(rng, (int((d[:, 0] * d[:, 2]).sum()),), dtype, scale)
    b = random_storage(rng, (int((d[:, 1] * d[:, 2]).sum()),), dtype, scale)
    return a, b


# ---------------------------------------------------------------------------
# Triangular matrix multiplication (Section 7.1): a square lower-triangular L
# and a dense B, entries N(0, 1); the strict upper triangle of L's storage is
# filled with NaN so that any read of it shows in the result.
# ---------------------------------------------------------------------------
def make_trmm_operands(n: int, m: int, rng: np.random.Generator, dtype: str, nan_upper: bool = True):
    """L [n, n] and B [n, m] storage arrays."""
    lv = rng.standard_normal((n, n))
    if nan_upper:
        lv[np.triu_indices(n, 1)] = np.nan
    return as_storage(lv, dtype), as_storage(rng.standard_normal((n, m)), dtype)
