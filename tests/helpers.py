"""Shared test helpers: host <-> device transfer of storage arrays and the
parity criteria.

Parity criteria (from the required tolerances):
  bf16  element-wise |gpu - oracle| <= 1e-3 + 2e-2 * |oracle| for every single
        operator; for the composed encoder layer the relative term is taken
        against the token row's scale, |gpu - oracle| <= 1e-3 + 2e-2 * max_row |oracle|
        (LayerNorm re-centres each row, so a one-ulp rounding flip upstream
        lands as an absolute error on outputs that happen to be near zero;
        tests/test_tolerance_readings.py shows an independent fp32 pipeline
        doing the same), and each row's mean |gpu - oracle| / max_row |oracle|
        at most ROW_MEAN_TOL
  fp32  per stored row r: max_i |gpu - oracle| <= 1e-5 * max_i |oracle|
        (row-normwise, so entries that cancel to near zero do not dominate)
  integers: exact equality
"""
from __future__ import annotations

import numpy as np
import torch

BF16_ATOL, BF16_RTOL = 1e-3, 2e-2
F32_RTOL = 1e-5


def dev(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Storage array (float32, or uint16 bf16 bits) -> device tensor."""
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(a, np.uint16).view(np.int16)).view(torch.bfloat16)
    return t.to(device)


def host(t: torch.Tensor, dtype: str) -> np.ndarray:
    """Device tensor -> storage array."""
    t = t.detach().cpu().contiguous()
    if dtype == "f32":
        return t.numpy().astype(np.float32)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def values(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(a, np.float32).astype(np.float64)
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_close(got_bits: np.ndarray, ref_bits: np.ndarray):
    """(ok, worst excess over the bf16 tolerance) for bf16 storage arrays."""
    g, o = values(got_bits, "bf16"), values(ref_bits, "bf16")
    if g.shape != o.shape:
        return False, float("inf")
    if g.size == 0:
        return True, 0.0
    excess = np.abs(g - o) - (BF16_ATOL + BF16_RTOL * np.abs(o))
    bad = ~np.isfinite(g)
    worst = float(np.max(excess)) if not bad.any() else float("inf")
    return bool(worst <= 0 and not bad.any()), worst


ROW_MEAN_TOL = 1e-3  # per token row: mean |g - o| / max_row |o|
ELEM_PASS_MIN = 0.98  # composed layer: fraction of elements within the element-wise bound


def bf16_row_stats(got_bits: np.ndarray, ref_bits: np.ndarray, row_len: int) -> dict:
    """Error statistics of a composed-layer output, per token row: the worst
    excess over the row-scaled bound, the worst row mean of |g - o| / max_row |o|,
    the worst excess over the element-wise bound and the fraction of elements
    within it."""
    g = values(got_bits, "bf16").reshape(-1, row_len)
    o = values(ref_bits, "bf16").reshape(-1, row_len)
    if g.size == 0:
        return {"row_excess": 0.0, "row_mean": 0.0, "elem_excess": 0.0, "elem_pass": 1.0, "finite": True}
    finite = bool(np.all(np.isfinite(g)))
    err = np.abs(g - o)
    rowmax = np.maximum(np.abs(o).max(axis=1, keepdims=True), 1e-30)
    elem = err - (BF16_ATOL + BF16_RTOL * np.abs(o))
    return {"row_excess": float((err - (BF16_ATOL + BF16_RTOL * rowmax)).max()),
            "row_mean": float((err / rowmax).mean(axis=1).max()),
            "elem_excess": float(elem.max()), "elem_pass": float((elem <= 0).mean()), "finite": finite}


def bf16_row_close(got_bits: np.ndarray, ref_bits: np.ndarray, row_len: int):
    """(ok, worst excess) for the composed layer: per token row,
    |g - o| <= 1e-3 + 2e-2 * max_row |o| element-wise, and the row's mean
    |g - o| / max_row |o| at most ROW_MEAN_TOL (rounding-level on average)."""
    st = bf16_row_stats(got_bits, ref_bits, row_len)
    if not st["finite"]:
        return False, float("inf")
    return st["row_excess"] <= 0 and st["row_mean"] <= ROW_MEAN_TOL, st["row_excess"]


def rowwise_close(got: np.ndarray, ref: np.ndarray, rtol: float = F32_RTOL, row_len: int | None = None) -> bool:
    """fp32 criterion: rows of `row_len` elements (or the last axis)."""
    g = np.asarray(got, np.float64)
    o = np.asarray(ref, np.float64)
    if g.shape != o.shape or not np.all(np.isfinite(g)):
        return False
    if g.size == 0:
        return True
    if row_len is not None:
        g, o = g.reshape(-1, row_len), o.reshape(-1, row_len)
    elif g.ndim == 1:
        g, o = g[None], o[None]
    err = np.max(np.abs(g - o), axis=-1)
    scale = np.max(np.abs(o), axis=-1)
    return bool(np.all(err <= rtol * scale + 1e-30))


def close(got: np.ndarray, ref: np.ndarray, dtype: str, row_len: int | None = None) -> bool:
    if dtype == "bf16":
        return bf16_close(got, ref)[0]
    return rowwise_close(got, ref, F32_RTOL, row_len)


def score_rows(flat: np.ndarray, lengths, heads) -> list:
    """Split a flat score buffer into per-sequence [L, H, L] blocks."""
    out, o = [], 0
    for n in lengths:
        n = int(n)
        out.append(flat[o:o + heads * n * n].reshape(n, heads, n))
        o += heads * n * n
    return out


def scores_close(got: np.ndarray, ref: np.ndarray, lengths, heads, dtype: str) -> bool:
    """Score / probability buffers: bf16 element-wise; fp32 per score row (L_b entries)."""
    if dtype == "bf16":
        return bf16_close(got, ref)[0]
    for g, o in zip(score_rows(got, lengths, heads), score_rows(ref, lengths, heads)):
        if g.size and not rowwise_close(g.reshape(-1, g.shape[-1]), o.reshape(-1, o.shape[-1])):
            return False
    return True


def canary_buffer(n: int, dtype: str, pad: int = 4096, device="cuda"):
    """A buffer of n elements with `pad` NaN-filled guard elements on each side.
    Returns (whole, view)."""
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    whole = torch.full((n + 2 * pad,), float("nan"), dtype=tdt, device=device)
    return whole, whole[pad:pad + n]


def canary_intact(whole: torch.Tensor, n: int, pad: int = 4096) -> bool:
    w = whole.float().cpu()
    return bool(torch.isnan(w[:pad]).all() and torch.isnan(w[pad + n:]).all())


def rising_keys(lengths, heads: int, step: float, seed: int, scale: float = 0.125):
    """bf16 bits of q, k, v for attention whose scores rise with every chunk of 32
    keys of a sequence: q near a fixed direction, k rows shifted along it so that
    the scaled score of key j is about step * (j // 32) nats plus noise.  Every
    later chunk then holds exponentials far above a running reference set by the
    first chunk (2^23 per 16 nats), so an online softmax must raise its reference
    at every chunk."""
    from workloads import to_bf16_bits

    rng = np.random.default_rng(seed)
    T, d = int(np.sum(lengths)), heads * 64
    q = 1.0 + 0.1 * rng.standard_normal((T, d))
    k = 0.1 * rng.standard_normal((T, d))
    t0 = 0
    for n in np.asarray(lengths, np.int64):
        k[t0:t0 + n] += (np.arange(n) // 32)[:, None] * (step / (scale * 64.0))
        t0 += int(n)
    v = rng.standard_normal((T, d))
    return tuple(to_bf16_bits(a.astype(np.float32)) for a in (q, k, v))
