"""Python binding of libragged.so: the ragged (minimally padded) transformer
encoder layer for MI355X (gfx950).

This module only marshals arguments: torch tensors provide device memory and
the current HIP stream; every step of the computation runs in the library's HIP
kernels.  There is no CPU path: importing fails loudly when the library has not
been built (``python paper_2110_10221_amd/_build.py`` or
``__graft_entry__.build()``).

Function names match the C interface in include/ragged.h.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libragged.so")

RAG_OK = 0
RAG_F32, RAG_BF16 = 0, 1
RAG_ACT_NONE, RAG_ACT_GELU_ERF, RAG_ACT_GELU_TANH = 0, 1, 2
RAG_TILE = 64
RAG_HEAD_DIM = 64
RAG_LAYER_UNFUSED_ATTENTION = 1
RAG_LAYER_CAUSAL = 2
RAG_LAYER_BUILD_PLAN = 4
RAG_LAYER_EVENTS = 10
RAG_NOALLOC_SCRATCH_BYTES = 64 << 20
DATA_BITS = {1: "negative length", 2: "length > max_len", 4: "sum of lengths != total_tokens",
             8: "qkt_cap exceeded", 16: "av_cap exceeded", 32: "score buffer too small"}
RAG_VGEMM_TILE_M, RAG_VGEMM_TILE_N = 128, 256
RAG_VGEMM_MAX_BATCH, RAG_VGEMM_MAX_DIM, RAG_VGEMM_MAX_TILES = 4096, 65536, 1 << 30
VGEMM_DATA_BITS = {1: "negative size", 2: "size > RAG_VGEMM_MAX_DIM", 4: "tile_cap exceeded",
                   8: "operand buffer too small", 16: "bf16 needs k % 64 == 0 and n % 8 == 0"}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build the HIP library first "
                      "(python paper_2110_10221_amd/_build.py)")

_lib = ctypes.CDLL(LIB_PATH)

_p, _i32, _i64, _f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float


class RagPlan(ctypes.Structure):
    _fields_ = [("batch", _i32), ("total_tokens", _i32), ("max_len", _i32), ("heads", _i32),
                ("qkt_cap", _i64), ("av_cap", _i64),
                ("lengths", _p), ("tok_off", _p), ("att_off", _p), ("order", _p), ("tok_seq", _p),
                ("qkt_item_off", _p), ("av_item_off", _p), ("qkt_items", _p), ("av_items", _p),
                ("status", _p)]


class RagVgemmPlan(ctypes.Structure):
    _fields_ = [("batch", _i32), ("tile_cap", _i64), ("dims", _p), ("a_off", _p), ("b_off", _p), ("c_off", _p),
                ("order", _p), ("tile_off", _p), ("tile_items", _p), ("status", _p)]


class RagLayerWeights(ctypes.Structure):
    _fields_ = [(n, _p) for n in ("w_qkv", "b_qkv", "w_o", "b_o", "ln1_g", "ln1_b",
                                  "w_ff1", "b_ff1", "w_ff2", "b_ff2", "ln2_g", "ln2_b")]


def _sig(name, args):
    f = getattr(_lib, name)
    f.restype = ctypes.c_int32
    f.argtypes = args
    return f


_lib.ragged_status_string.restype = ctypes.c_char_p
_lib.ragged_status_string.argtypes = [_i32]
_lib.ragged_last_error.restype = ctypes.c_char_p
_lib.ragged_last_error.argtypes = []
_c_plan_capacity = _sig("ragged_plan_capacity", [_i32, _i32, _i32, _i32, ctypes.POINTER(_i64), ctypes.POINTER(_i64)])
_c_offsets = _sig("ragged_offsets", [ctypes.POINTER(RagPlan), _p])
_c_qkt = _sig("ragged_qkt", [ctypes.POINTER(RagPlan), _p, _i32, _p, _i32, _i32, _f32, _p, _i64, _i32, _p])
_c_softmax = _sig("ragged_softmax", [ctypes.POINTER(RagPlan), _p, _p, _i64, _i32, _p])
_c_attn_v = _sig("ragged_attn_v", [ctypes.POINTER(RagPlan), _p, _i64, _p, _i32, _i32, _p, _i32, _i32, _p])
_c_attention = _sig("ragged_attention", [ctypes.POINTER(RagPlan), _p, _i32, _p, _i32, _p, _i32, _i32, _f32, _p,
                                         _i32, _i32, _p])
_c_qkt_causal = _sig("ragged_qkt_causal", list(_c_qkt.argtypes))
_c_softmax_causal = _sig("ragged_softmax_causal", list(_c_softmax.argtypes))
_c_attn_v_causal = _sig("ragged_attn_v_causal", list(_c_attn_v.argtypes))
_c_attention_causal = _sig("ragged_attention_causal", list(_c_attention.argtypes))
_c_linear = _sig("packed_linear", [_p, _i32, _p, _p, _p, _i32, _i32, _p, _i32, _i32, _i32, _i32, _i32, _p])
_c_layernorm = _sig("packed_layernorm", [_p, _i32, _p, _p, _f32, _p, _i32, _i32, _i32, _i32, _p])
_c_vgemm_capacity = _sig("vgemm_plan_capacity", [_i32, _i32, _i32, ctypes.POINTER(_i64)])
_c_vgemm_tile_count = _sig("vgemm_tile_count", [_i32, _p, ctypes.POINTER(_i64)])
_c_vgemm_offsets = _sig("vgemm_offsets", [ctypes.POINTER(RagVgemmPlan), _p])
_c_vgemm = _sig("ragged_vgemm", [ctypes.POINTER(RagVgemmPlan), _p, _i64, _p, _i64, _p, _i64, _i32, _p])
_c_trmm = _sig("ragged_trmm", [_p, _i32, _p, _i32, _p, _i32, _i32, _i32, _i32, _p])
_c_ws = _sig("encoder_layer_workspace", [_i32, _i32, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_size_t)])
_c_layer = _sig("encoder_layer", [ctypes.POINTER(RagPlan), _p, _p, _i32, _i32, _i32, _i32, _f32, _i32, _i32,
                                  ctypes.POINTER(RagLayerWeights), _p, ctypes.c_size_t, _i32, _p, _p])
_c_layer_noalloc = _sig("encoder_layer_noalloc", [ctypes.POINTER(RagPlan), _p, _p, _i32, _i32, _i32, _i32, _f32,
                                                  _i32, _i32, ctypes.POINTER(RagLayerWeights), _i32, _p])


class RaggedError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = _lib.ragged_last_error().decode()
        super().__init__(f"{fn}: {_lib.ragged_status_string(status).decode()}: {msg}")


def _check(fn, status):
    if status != RAG_OK:
        raise RaggedError(fn, status)


def library():
    """The loaded ctypes library (for callers that want the raw C entry points)."""
    return _lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return RAG_BF16
    if t.dtype == torch.float32:
        return RAG_F32
    raise TypeError(f"unsupported tensor dtype {t.dtype} (bfloat16 or float32)")


def _ld(t):
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-D tensor with unit column stride")
    return t.stride(0)


def ragged_plan_capacity(batch, total_tokens, max_len, heads):
    q, a = _i64(), _i64()
    _check("ragged_plan_capacity", _c_plan_capacity(batch, total_tokens, max_len, heads, ctypes.byref(q), ctypes.byref(a)))
    return q.value, a.value


class Plan:
    """Device arrays of one batch's prelude, allocated with torch on `device`.

    `lengths` is an int32 device tensor [B]; `total_tokens` and `max_len` are
    the host-side sizes the caller promises (the device checks them)."""

    def __init__(self, lengths: torch.Tensor, total_tokens: int, max_len: int, heads: int,
                 qkt_cap: int | None = None, av_cap: int | None = None):
        if lengths.dtype != torch.int32 or lengths.dim() != 1:
            raise ValueError("lengths must be a 1-D int32 device tensor")
        if not lengths.is_contiguous():
            raise ValueError("lengths must be contiguous (the kernels read lengths[b] as dense memory)")
        if not lengths.is_cuda:
            raise ValueError("lengths must be a 1-D int32 device tensor")
        dev = lengths.device
        B = lengths.numel()
        cq, ca = ragged_plan_capacity(B, total_tokens, max_len, heads)
        qkt_cap = cq if qkt_cap is None else qkt_cap
        av_cap = ca if av_cap is None else av_cap
        i32 = dict(dtype=torch.int32, device=dev)
        self.lengths = lengths
        self.tok_off = torch.empty(B + 1, **i32)
        self.att_off = torch.empty(B + 1, dtype=torch.int64, device=dev)
        self.order = torch.empty(B, **i32)
        self.tok_seq = torch.empty(max(total_tokens, 1), **i32)
        self.qkt_item_off = torch.empty(B + 1, **i32)
        self.av_item_off = torch.empty(B + 1, **i32)
        self.qkt_items = torch.empty(max(4 * qkt_cap, 4), **i32)
        self.av_items = torch.empty(max(3 * av_cap, 3), **i32)
        self.status = torch.zeros(4, **i32)
        self.batch, self.total_tokens, self.max_len, self.heads = B, total_tokens, max_len, heads
        self.qkt_cap, self.av_cap = qkt_cap, av_cap
        self.c = RagPlan(B, total_tokens, max_len, heads, qkt_cap, av_cap,
                         lengths.data_ptr(), self.tok_off.data_ptr(), self.att_off.data_ptr(),
                         self.order.data_ptr(), self.tok_seq.data_ptr(), self.qkt_item_off.data_ptr(),
                         self.av_item_off.data_ptr(), self.qkt_items.data_ptr(), self.av_items.data_ptr(),
                         self.status.data_ptr())

    def ref(self):
        return ctypes.byref(self.c)

    def data_errors(self):
        """Decode status[0] (synchronises)."""
        f = int(self.status[0].item())
        return [msg for bit, msg in DATA_BITS.items() if f & bit]


def ragged_offsets(plan: Plan, stream=None):
    _check("ragged_offsets", _c_offsets(plan.ref(), _stream(stream)))


def ragged_qkt(plan: Plan, q, k, scores, scale, head_dim=RAG_HEAD_DIM, stream=None):
    _check("ragged_qkt", _c_qkt(plan.ref(), _ptr(q), _ld(q), _ptr(k), _ld(k), head_dim, scale, _ptr(scores),
                                scores.numel(), _dtype_code(q), _stream(stream)))


def ragged_qkt_causal(plan: Plan, q, k, scores, scale, head_dim=RAG_HEAD_DIM, stream=None):
    _check("ragged_qkt_causal", _c_qkt_causal(plan.ref(), _ptr(q), _ld(q), _ptr(k), _ld(k), head_dim, scale,
                                              _ptr(scores), scores.numel(), _dtype_code(q), _stream(stream)))


def ragged_softmax(plan: Plan, scores, probs=None, stream=None):
    probs = scores if probs is None else probs
    _check("ragged_softmax", _c_softmax(plan.ref(), _ptr(scores), _ptr(probs), min(scores.numel(), probs.numel()),
                                        _dtype_code(scores), _stream(stream)))
    return probs


def ragged_softmax_causal(plan: Plan, scores, probs=None, stream=None):
    probs = scores if probs is None else probs
    _check("ragged_softmax_causal", _c_softmax_causal(plan.ref(), _ptr(scores), _ptr(probs),
                                                      min(scores.numel(), probs.numel()), _dtype_code(scores),
                                                      _stream(stream)))
    return probs


def ragged_attn_v(plan: Plan, probs, v, out, head_dim=RAG_HEAD_DIM, stream=None):
    _check("ragged_attn_v", _c_attn_v(plan.ref(), _ptr(probs), probs.numel(), _ptr(v), _ld(v), head_dim, _ptr(out),
                                      _ld(out), _dtype_code(v), _stream(stream)))


def ragged_attn_v_causal(plan: Plan, probs, v, out, head_dim=RAG_HEAD_DIM, stream=None):
    _check("ragged_attn_v_causal", _c_attn_v_causal(plan.ref(), _ptr(probs), probs.numel(), _ptr(v), _ld(v),
                                                    head_dim, _ptr(out), _ld(out), _dtype_code(v), _stream(stream)))


def ragged_attention(plan: Plan, q, k, v, out, scale, head_dim=RAG_HEAD_DIM, stream=None):
    _check("ragged_attention", _c_attention(plan.ref(), _ptr(q), _ld(q), _ptr(k), _ld(k), _ptr(v), _ld(v), head_dim,
                                            scale, _ptr(out), _ld(out), _dtype_code(q), _stream(stream)))


def ragged_attention_causal(plan: Plan, q, k, v, out, scale, head_dim=RAG_HEAD_DIM, stream=None):
    _check("ragged_attention_causal", _c_attention_causal(plan.ref(), _ptr(q), _ld(q), _ptr(k), _ld(k), _ptr(v),
                                                          _ld(v), head_dim, scale, _ptr(out), _ld(out),
                                                          _dtype_code(q), _stream(stream)))


def packed_linear(x, w, y, bias=None, residual=None, act=RAG_ACT_NONE, stream=None):
    T, K = x.shape
    N = w.shape[0]
    ldr = _ld(residual) if residual is not None else 0
    _check("packed_linear", _c_linear(_ptr(x), _ld(x), _ptr(w), _ptr(bias), _ptr(residual), ldr, act, _ptr(y), _ld(y),
                                      T, K, N, _dtype_code(x), _stream(stream)))


def packed_layernorm(x, gamma, beta, y, eps=1e-5, stream=None):
    T, d = x.shape
    _check("packed_layernorm", _c_layernorm(_ptr(x), _ld(x), _ptr(gamma), _ptr(beta), eps, _ptr(y), _ld(y), T, d,
                                            _dtype_code(x), _stream(stream)))


def encoder_layer_workspace(total_tokens, max_len, d_model, heads, d_ff, dtype=RAG_BF16, flags=0):
    n = ctypes.c_size_t()
    _check("encoder_layer_workspace", _c_ws(total_tokens, max_len, d_model, heads, d_ff, dtype, flags,
                                            ctypes.byref(n)))
    return n.value


WEIGHT_ORDER = ("w_qkv", "b_qkv", "w_o", "b_o", "ln1_g", "ln1_b", "w_ff1", "b_ff1", "w_ff2", "b_ff2", "ln2_g", "ln2_b")


def layer_weights(weights: dict) -> RagLayerWeights:
    return RagLayerWeights(*[weights[n].data_ptr() for n in WEIGHT_ORDER])


def encoder_layer(plan: Plan, x, y, weights, d_ff, workspace, heads=None, head_dim=RAG_HEAD_DIM, ln_eps=1e-5,
                  act=RAG_ACT_GELU_ERF, flags=0, stream=None, events=None):
    """`weights`: dict of device tensors (WEIGHT_ORDER names) or a RagLayerWeights;
    `events`: optional ctypes array of RAG_LAYER_EVENTS hipEvent_t handles."""
    T, d = x.shape
    heads = plan.heads if heads is None else heads
    w = weights if isinstance(weights, RagLayerWeights) else layer_weights(weights)
    _check("encoder_layer", _c_layer(plan.ref(), _ptr(x), _ptr(y), d, heads, head_dim, d_ff, ln_eps, act, flags,
                                     ctypes.byref(w), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _dtype_code(x), _stream(stream),
                                     None if events is None else ctypes.cast(events, ctypes.c_void_p)))


def encoder_layer_noalloc(plan: Plan, x, y, weights, d_ff, heads=None, head_dim=RAG_HEAD_DIM, ln_eps=1e-5,
                          act=RAG_ACT_GELU_ERF, flags=0, stream=None):
    """encoder_layer with the library's fixed device scratch array as its workspace
    (RAG_NOALLOC_SCRATCH_BYTES): no workspace argument, nothing allocated."""
    T, d = x.shape
    heads = plan.heads if heads is None else heads
    w = weights if isinstance(weights, RagLayerWeights) else layer_weights(weights)
    _check("encoder_layer_noalloc", _c_layer_noalloc(plan.ref(), _ptr(x), _ptr(y), d, heads, head_dim, d_ff, ln_eps,
                                                     act, flags, ctypes.byref(w), _dtype_code(x), _stream(stream)))


def vgemm_plan_capacity(batch, max_m, max_n):
    n = _i64()
    _check("vgemm_plan_capacity", _c_vgemm_capacity(batch, max_m, max_n, ctypes.byref(n)))
    return n.value


def vgemm_tile_count(host_dims):
    """Exact tile count of a batch from its (m, n, k) sizes held on the host."""
    import numpy as np

    d = np.ascontiguousarray(np.asarray(host_dims, dtype=np.int32).reshape(-1, 3))
    n = _i64()
    _check("vgemm_tile_count", _c_vgemm_tile_count(d.shape[0], d.ctypes.data_as(ctypes.c_void_p), ctypes.byref(n)))
    return n.value


class VgemmPlan:
    """Device arrays of a vgemm batch's prelude, allocated with torch.

    `dims` is an int32 device tensor [B, 3] of (m, n, k).  `tile_cap` defaults to
    the exact tile count when `host_dims` (the same sizes on the host) is given,
    else to the bound from `max_m` / `max_n`."""

    def __init__(self, dims: torch.Tensor, tile_cap: int | None = None, host_dims=None, max_m=None, max_n=None):
        if dims.dtype != torch.int32 or not dims.is_cuda or dims.dim() != 2 or dims.shape[1] != 3:
            raise ValueError("dims must be a [B, 3] int32 device tensor")
        if not dims.is_contiguous():
            raise ValueError("dims must be contiguous")
        dev = dims.device
        B = dims.shape[0]
        if tile_cap is None:
            if host_dims is not None:
                tile_cap = vgemm_tile_count(host_dims)
            elif max_m is not None and max_n is not None:
                tile_cap = vgemm_plan_capacity(B, max_m, max_n)
            else:
                raise ValueError("give tile_cap, host_dims or max_m and max_n")
        i64 = dict(dtype=torch.int64, device=dev)
        self.dims = dims
        self.a_off, self.b_off, self.c_off = (torch.empty(B + 1, **i64) for _ in range(3))
        self.order = torch.empty(B, dtype=torch.int32, device=dev)
        self.tile_off = torch.empty(B + 1, **i64)
        self.tile_items = torch.empty(max(4 * tile_cap, 4), dtype=torch.int32, device=dev)
        self.status = torch.zeros(3, dtype=torch.int32, device=dev)
        self.batch, self.tile_cap = B, tile_cap
        self.c = RagVgemmPlan(B, tile_cap, dims.data_ptr(), self.a_off.data_ptr(), self.b_off.data_ptr(),
                              self.c_off.data_ptr(), self.order.data_ptr(), self.tile_off.data_ptr(),
                              self.tile_items.data_ptr(), self.status.data_ptr())

    def ref(self):
        return ctypes.byref(self.c)

    def data_errors(self):
        """Decode status[0] (synchronises)."""
        f = int(self.status[0].item())
        return [msg for bit, msg in VGEMM_DATA_BITS.items() if f & bit]

    def n_tiles(self):
        return int(self.status[1].item())


def vgemm_offsets(plan: VgemmPlan, stream=None):
    _check("vgemm_offsets", _c_vgemm_offsets(plan.ref(), _stream(stream)))


def ragged_vgemm(plan: VgemmPlan, a, b, c, stream=None):
    """C_b = A_b B_b^T for every problem of the packed batch: a, b, c are 1-D
    tensors of one dtype holding the packed operands."""
    if not (a.dtype == b.dtype == c.dtype):
        raise TypeError("a, b and c must share one dtype")
    for t in (a, b, c):
        if not t.is_contiguous():
            raise ValueError("a, b and c must be contiguous")
    _check("ragged_vgemm", _c_vgemm(plan.ref(), _ptr(a), a.numel(), _ptr(b), b.numel(), _ptr(c), c.numel(),
                                    _dtype_code(a), _stream(stream)))


def ragged_trmm(l, b, c, stream=None):
    """C = tril(L) B: l [n, n], b and c [n, m], 2-D tensors of one dtype with unit
    column stride (entries of l above the diagonal are ignored)."""
    n, m = b.shape
    if l.shape[0] != n or l.shape[1] < n or c.shape != b.shape:
        raise ValueError("expected l [n, n], b [n, m] and c [n, m]")
    if not (l.dtype == b.dtype == c.dtype):
        raise TypeError("l, b and c must share one dtype")
    _check("ragged_trmm", _c_trmm(_ptr(l), _ld(l), _ptr(b), _ld(b), _ptr(c), _ld(c), n, m, _dtype_code(b),
                                  _stream(stream)))
