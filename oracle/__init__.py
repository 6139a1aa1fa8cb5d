"""CPU oracle for the ragged transformer encoder layer (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does: the GPU
path shares no code with it.  The arithmetic lives in ``oracle.c`` (plain C,
double-precision accumulation); this module only marshals numpy arrays.

Every function takes and returns *storage* arrays: float32 for dtype "f32",
uint16 bfloat16 bit patterns for dtype "bf16".
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import NamedTuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F32, BF16 = 0, 1
ACT_NONE, ACT_GELU_ERF, ACT_GELU_TANH = 0, 1, 2
_DT = {"f32": F32, "bf16": BF16, F32: F32, BF16: BF16}


SANITIZE_CC = "/opt/rocm/llvm/bin/clang"  # the compiler of the sanitizer runtime libragged's host code uses


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (strict IEEE: no fast-math,
    no FMA contraction).  `sanitize` builds it with AddressSanitizer and
    UndefinedBehaviorSanitizer instead (clang, whose runtime must then be
    preloaded into the Python process)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cc = [SANITIZE_CC, "-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-g"] if sanitize else ["gcc"]
        subprocess.check_call(cc + ["-O2", "-std=gnu11", "-fPIC", "-shared", "-ffp-contract=off",
                                    "-fno-fast-math", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        l = ctypes.CDLL(_LIB)
        p, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        l.oracle_offsets.restype = ctypes.c_int
        l.oracle_offsets.argtypes = [i32, p, i32, i32, i32, p, p, p, p, p, p, p, i64, p, i64, p]
        l.oracle_qkt.argtypes = [ctypes.c_int, i32, p, i32, i32, p, i64, p, i64, f64, ctypes.c_int, p]
        l.oracle_softmax.argtypes = [ctypes.c_int, i32, p, i32, ctypes.c_int, p, p]
        l.oracle_attn_v.argtypes = [ctypes.c_int, i32, p, i32, i32, ctypes.c_int, p, p, i64, p, i64]
        l.oracle_linear.argtypes = [ctypes.c_int, i64, i32, i32, p, i64, p, p, p, i64, ctypes.c_int, p, i64]
        l.oracle_layernorm.argtypes = [ctypes.c_int, i64, i32, p, i64, p, p, f64, p, i64]
        l.oracle_encoder_layer.restype = ctypes.c_int
        l.oracle_encoder_layer.argtypes = [ctypes.c_int, i32, p, i32, i32, i32, f64, ctypes.c_int, ctypes.c_int, p, p,
                                           p]
        l.oracle_round_bf16.argtypes = [i64, p, p]
        l.oracle_vgemm_offsets.restype = ctypes.c_int
        l.oracle_vgemm_offsets.argtypes = [i32, p, i32, i32, p, p, p, p, p]
        l.oracle_vgemm.argtypes = [ctypes.c_int, i32, p, p, p, p]
        l.oracle_trmm.argtypes = [ctypes.c_int, i32, i32, p, i64, p, i64, p, i64]
        l.oracle_trmm_rows.argtypes = [ctypes.c_int, i32, p, i64, p, i64, p, i32, p, i64]
        _lib = l
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _storage_dtype(dtype):
    return np.float32 if _DT[dtype] == F32 else np.uint16


def _lens(lengths):
    return np.ascontiguousarray(lengths, dtype=np.int32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 bits (round to nearest, ties to even)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_round_bf16(x.size, _ptr(x), _ptr(out))
    return out


class Plan:
    """The prelude's arrays, as computed by the oracle."""

    def __init__(self, tok_off, att_off, order, tok_seq, qkt_item_off, av_item_off,
                 qkt_items, av_items, rc):
        self.tok_off, self.att_off, self.order, self.tok_seq = tok_off, att_off, order, tok_seq
        self.qkt_item_off, self.av_item_off = qkt_item_off, av_item_off
        self.qkt_items, self.av_items, self.rc = qkt_items, av_items, rc


def offsets(lengths, heads: int, tile_m: int = 64, tile_n: int = 64,
            qkt_cap: int | None = None, av_cap: int | None = None) -> Plan:
    L = _lens(lengths)
    B = L.size
    T = int(max(L.sum(), 0))
    if qkt_cap is None:
        qkt_cap = int(sum(heads * (-(-max(int(v), 0) // tile_m)) * (-(-max(int(v), 0) // tile_n)) for v in L))
    if av_cap is None:
        av_cap = int(sum(heads * (-(-max(int(v), 0) // tile_m)) for v in L))
    tok_off = np.zeros(B + 1, np.int64)
    att_off = np.zeros(B + 1, np.int64)
    order = np.zeros(B, np.int32)
    tok_seq = np.zeros(max(T, 1), np.int32)
    qoff = np.zeros(B + 1, np.int64)
    aoff = np.zeros(B + 1, np.int64)
    qitems = np.zeros(max(4 * qkt_cap, 4), np.int32)
    aitems = np.zeros(max(3 * av_cap, 3), np.int32)
    counts = np.zeros(2, np.int64)
    rc = lib().oracle_offsets(B, _ptr(L), heads, tile_m, tile_n, _ptr(tok_off), _ptr(att_off),
                              _ptr(order), _ptr(tok_seq), _ptr(qoff), _ptr(aoff),
                              _ptr(qitems), qkt_cap, _ptr(aitems), av_cap, _ptr(counts))
    nq, na = int(counts[0]), int(counts[1])
    return Plan(tok_off, att_off, order, tok_seq[:T], qoff, aoff,
                qitems[:4 * min(nq, qkt_cap)].reshape(-1, 4), aitems[:3 * min(na, av_cap)].reshape(-1, 3), rc)


def score_elems(lengths, heads: int) -> int:
    L = _lens(lengths).astype(np.int64)
    return int(heads * (L * L).sum())


def qkt(dtype, lengths, heads, head_dim, q, ldq, k, ldk, scale, causal=False):
    """Scores in the X[b][i][h][j] layout; with `causal` only j <= i is written (the rest stays 0)."""
    L = _lens(lengths)
    S = np.zeros(max(score_elems(L, heads), 1), _storage_dtype(dtype))
    lib().oracle_qkt(_DT[dtype], L.size, _ptr(L), heads, head_dim, _ptr(np.ascontiguousarray(q)), ldq,
                     _ptr(np.ascontiguousarray(k)), ldk, float(scale), int(causal), _ptr(S))
    return S[:score_elems(L, heads)]


def softmax(dtype, lengths, heads, S, causal=False):
    """Row softmax; with `causal` row (b, i, h) covers j <= i only (the rest of P stays 0)."""
    L = _lens(lengths)
    S = np.ascontiguousarray(S)
    P = np.zeros(max(S.size, 1), _storage_dtype(dtype))
    lib().oracle_softmax(_DT[dtype], L.size, _ptr(L), heads, int(causal), _ptr(S), _ptr(P))
    return P[:S.size]


def attn_v(dtype, lengths, heads, head_dim, P, v, ldv, ldo=None, causal=False):
    L = _lens(lengths)
    T = int(L.sum())
    ldo = heads * head_dim if ldo is None else ldo
    O = np.zeros(max(T * ldo, 1), _storage_dtype(dtype))
    lib().oracle_attn_v(_DT[dtype], L.size, _ptr(L), heads, head_dim, int(causal), _ptr(np.ascontiguousarray(P)),
                        _ptr(np.ascontiguousarray(v)), ldv, _ptr(O), ldo)
    return O[:T * ldo].reshape(T, ldo)


def linear(dtype, x, w, bias=None, residual=None, act=ACT_NONE):
    """y = act(x w^T + bias) + residual over the rows of x (all arrays in storage form)."""
    x = np.ascontiguousarray(x)
    w = np.ascontiguousarray(w)
    T, K = x.shape
    N = w.shape[0]
    assert w.shape[1] == K
    y = np.zeros((T, N), _storage_dtype(dtype))
    r = None if residual is None else np.ascontiguousarray(residual)
    b = None if bias is None else np.ascontiguousarray(bias)
    lib().oracle_linear(_DT[dtype], T, K, N, _ptr(x), K, _ptr(w), _ptr(b), _ptr(r), N, act, _ptr(y), N)
    return y


def layernorm(dtype, x, gamma, beta, eps=1e-5):
    x = np.ascontiguousarray(x)
    T, d = x.shape
    y = np.zeros((T, d), _storage_dtype(dtype))
    lib().oracle_layernorm(_DT[dtype], T, d, _ptr(x), d, _ptr(np.ascontiguousarray(gamma)),
                           _ptr(np.ascontiguousarray(beta)), float(eps), _ptr(y), d)
    return y


_WNAMES = ("w_qkv", "b_qkv", "w_o", "b_o", "ln1_g", "ln1_b", "w_ff1", "b_ff1", "w_ff2", "b_ff2", "ln2_g", "ln2_b")


def encoder_layer(dtype, lengths, x, weights: dict, d_model, heads, d_ff, eps=1e-5, act=ACT_GELU_ERF, causal=False):
    """One post-LN encoder layer over packed tokens x [T, d_model] (masked attention with `causal`)."""
    L = _lens(lengths)
    T = int(L.sum())
    arrs = [np.ascontiguousarray(weights[n]) for n in _WNAMES]
    wstruct = (ctypes.c_void_p * 12)(*[a.ctypes.data for a in arrs])
    x = np.ascontiguousarray(x)
    out = np.zeros((max(T, 1), d_model), _storage_dtype(dtype))
    rc = lib().oracle_encoder_layer(_DT[dtype], L.size, _ptr(L), d_model, heads, d_ff, float(eps), act, int(causal),
                                    ctypes.cast(wstruct, ctypes.c_void_p), _ptr(x), _ptr(out))
    if rc != 0:
        raise MemoryError("oracle_encoder_layer: allocation failed")
    return out[:T]


VGEMM_TILE_M, VGEMM_TILE_N = 128, 256


class VgemmOffsets(NamedTuple):
    a_off: np.ndarray
    b_off: np.ndarray
    c_off: np.ndarray
    order: np.ndarray
    tile_off: np.ndarray


def vgemm_offsets(dims, tile_m=VGEMM_TILE_M, tile_n=VGEMM_TILE_N) -> VgemmOffsets:
    """Packed-storage offsets, largest-first order and tile prefix of a vgemm batch;
    dims is [B, 3] (m, n, k)."""
    d = np.ascontiguousarray(np.asarray(dims, np.int32).reshape(-1, 3))
    B = d.shape[0]
    a, b, c, t = (np.zeros(B + 1, np.int64) for _ in range(4))
    order = np.zeros(max(B, 1), np.int32)
    rc = lib().oracle_vgemm_offsets(B, _ptr(d), tile_m, tile_n, _ptr(a), _ptr(b), _ptr(c), _ptr(order), _ptr(t))
    if rc != 0:
        raise ValueError("negative vgemm size")
    return VgemmOffsets(a, b, c, order[:B], t)


def vgemm(dtype, dims, a, b):
    """C_b = A_b B_b^T for every problem of the packed batch (storage form in and out)."""
    d = np.ascontiguousarray(np.asarray(dims, np.int32).reshape(-1, 3))
    c_elems = int((d[:, 0].astype(np.int64) * d[:, 1]).sum())
    c = np.zeros(max(c_elems, 1), _storage_dtype(dtype))
    lib().oracle_vgemm(_DT[dtype], d.shape[0], _ptr(d), _ptr(np.ascontiguousarray(a)), _ptr(np.ascontiguousarray(b)),
                       _ptr(c))
    return c[:c_elems]


def trmm(dtype, n: int, m: int, l, b, ldl: int | None = None, ldb: int | None = None):
    """C = tril(L) B for L [n, n] (leading dimension ldl, entries above the
    diagonal ignored) and B [n, m] (ldb); returns C [n, m] in storage form."""
    ldl = n if ldl is None else ldl
    ldb = m if ldb is None else ldb
    l = np.ascontiguousarray(l).reshape(-1)
    b = np.ascontiguousarray(b).reshape(-1)
    if n > 0 and (l.size < (n - 1) * ldl + n or (m > 0 and b.size < (n - 1) * ldb + m)):
        raise ValueError("operand smaller than its declared shape")
    c = np.zeros((n, m), _storage_dtype(dtype))
    lib().oracle_trmm(_DT[dtype], n, m, _ptr(l), ldl, _ptr(b), ldb, _ptr(c), m)
    return c


def trmm_rows(dtype, n: int, m: int, l, b, rows, ldl: int | None = None, ldb: int | None = None):
    """Rows `rows` of tril(L) B (same arguments as trmm); returns [len(rows), m]."""
    ldl = n if ldl is None else ldl
    ldb = m if ldb is None else ldb
    r = np.ascontiguousarray(rows, np.int32)
    if r.size and (r.min() < 0 or r.max() >= n):
        raise ValueError("row out of range")
    l = np.ascontiguousarray(l).reshape(-1)
    b = np.ascontiguousarray(b).reshape(-1)
    c = np.zeros((r.size, m), _storage_dtype(dtype))
    lib().oracle_trmm_rows(_DT[dtype], m, _ptr(l), ldl, _ptr(b), ldb, _ptr(r), r.size, _ptr(c), m)
    return c
