"""Benchmark of the ragged encoder layer on one MI355X.

One step = one pass of the whole hot path over one synthetic batch: the
prelude (the plan ragged_offsets builds; here the layer builds it, its
workgroups carried by the QKV projection's launch) and one encoder layer (QKV
projection, fused ragged attention, output projection + residual, LayerNorm,
FF1 + GELU, FF2 + residual, LayerNorm).  The workload is the batch-128 layer: lengths
uniform in [32, 512], d_model 1024, 16 heads of 64, FFN 4096, bf16, seeded
synthetic data and random-initialised weights (std 0.02).

Prints ONE JSON line (rank 0, N = 1).  Per-kernel times come from HIP events
recorded by the library on the stream the kernels run on; the CPU baseline
times the oracle on a bounded sample of the same batch.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import math
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PEAK_F32_TFLOPS = 157.3     # MI355X dense fp32 MFMA
METRIC = "ms/encoder layer + useful (unpadded) TFLOP/s, fraction of bf16 MFMA peak"

# stage index (events[k] .. events[k+1]) -> kernel symbol
STAGES = ["qkv_proj", "qkt", "softmax", "attention", "out_proj", "layernorm1", "ff1", "ff2", "layernorm2"]


def stage_kernels(T, d, dff):
    """Kernel symbol of each timed stage of the bf16 layer with fused attention, following the
    library's launch rules: one GEMM kernel per epilogue (128-token tiles, a sparse last
    round as 64-token halves); LayerNorm instantiated for the power of two >= d / 512
    16-byte chunks per lane."""
    chunks = -(-d // 8 // 64)  # 16-byte chunks per lane, rounded up to a power of two
    ln = f"k_layernorm<true, {1 << max(0, (chunks - 1).bit_length())}>"
    return {
        "qkv_proj": "k_gemm_bf16<0, true, false>",
        "attention": "k_attention_bf16<false>",
        "out_proj": "k_gemm_bf16<0, true, true>",
        "ff2": "k_gemm_bf16<0, true, true>",
        "ff1": "k_gemm_bf16<1, true, false>",
        "layernorm1": ln,
        "layernorm2": ln,
    }
KERNEL_SOURCES = {
    "k_gemm_bf16": "paper_2110_10221_amd/csrc/gemm.hip",
    "k_attention_bf16": "paper_2110_10221_amd/csrc/attention.hip",
    "k_layernorm": "paper_2110_10221_amd/csrc/layernorm.hip",
    "k_vgemm_bf16": "paper_2110_10221_amd/csrc/gemm.hip",
    "k_trmm_bf16": "paper_2110_10221_amd/csrc/gemm.hip",
    "k_qkt_bf16": "paper_2110_10221_amd/csrc/attention.hip",
    "k_softmax": "paper_2110_10221_amd/csrc/attention.hip",
    "k_attn_v_bf16": "paper_2110_10221_amd/csrc/attention.hip",
    "k_plan_fused": "paper_2110_10221_amd/csrc/offsets.hip",
    "k_plan_small": "paper_2110_10221_amd/csrc/offsets.hip",
    "k_plan_fill": "paper_2110_10221_amd/csrc/offsets.hip",
}
# unfused operator measurements: kernels of each operator, and the tag under which
# their counters are stored per workload (the same symbols run at both shapes)
SDPA_TAGS = {2: "sdpa_b32", 4: "layer_b128"}
SDPA_KERNELS = {"offsets": ["k_plan_fused"], "qkt": ["k_qkt_bf16"], "softmax": ["k_softmax<true>"],
                "attn_v": ["k_attn_v_bf16"]}


def stage_work(T, d, H, dff, s2):
    """Algorithmic FLOPs and HBM bytes (bf16) of each stage: every operand read
    once, every result written once."""
    e = 2
    return {
        "qkv_proj": (2.0 * T * d * 3 * d, e * (T * d + 3 * d * d + 3 * d + T * 3 * d)),
        "attention": (4.0 * d * s2, e * (3 * T * d + T * d)),
        "out_proj": (2.0 * T * d * d, e * (T * d + d * d + d + 2 * T * d)),
        "layernorm1": (8.0 * T * d, e * (2 * T * d + 2 * d)),
        "ff1": (2.0 * T * d * dff, e * (T * d + dff * d + dff + T * dff)),
        "ff2": (2.0 * T * dff * d, e * (T * dff + d * dff + d + 2 * T * d)),
        "layernorm2": (8.0 * T * d, e * (2 * T * d + 2 * d)),
    }


def useful_flops(L, d, dff):
    L = np.asarray(L, np.float64)
    T, s2 = L.sum(), (L * L).sum()
    return 2 * T * d * (3 * d + d + 2 * dff) + 4 * d * s2


def padded_fraction(L, d, dff):
    Lp = np.full(len(L), float(np.max(L)))
    return 1.0 - useful_flops(L, d, dff) / useful_flops(Lp, d, dff)


CSRC = "paper_2110_10221_amd/csrc"


def source_hash(path):
    """Hash of a kernel's source together with every local header of the
    library's source folder (any of them may be included by it)."""
    h = hashlib.sha256()
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, CSRC)) if f.endswith(".h"))
    for p in [path] + [f"{CSRC}/{f}" for f in headers]:
        h.update(p.encode())
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


def length_text(recipe):
    """Human-readable length distribution of a workload recipe (workloads.draw_lengths)."""
    kind, _, rest = recipe.partition(":")
    v = rest.split(":")
    if kind == "fixed":
        return f"lengths {{{rest.replace(',', ', ')}}}"
    if kind == "uniform":
        return f"lengths uniform [{v[0]}, {v[1]}]"
    if kind == "lognormal":
        return f"lengths lognormal (median {v[0]}, sigma {v[1]}, max {v[2]})"
    if kind == "skew":
        return (f"lengths skewed ({round(100 * float(v[4]))}% uniform [{v[2]}, {v[3]}], "
                f"the rest uniform [{v[0]}, {v[1]}])")
    return f"lengths {recipe}"


def load_traffic(kernel):
    """HBM bytes per launch measured with rocprofv3 counters (profiles/traffic.json),
    only while the kernel's source is unchanged since the measurement.  `kernel` may
    carry a workload tag ("k_softmax<true>@layer_b128")."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec:
        return None
    src = KERNEL_SOURCES.get(kernel.split("@")[0].split("<")[0])
    if src is None or rec.get("source_sha") != source_hash(src):
        return None
    return rec.get("bytes_per_launch")


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch already loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]

    def create(self, n):
        arr = (ctypes.c_void_p * n)()
        for i in range(n):
            ev = ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(ev)) == 0
            arr[i] = ev.value
        return arr

    def record(self, ev, stream):
        assert self.hip.hipEventRecord(ctypes.c_void_p(ev), ctypes.c_void_p(stream)) == 0

    def elapsed(self, a, b):
        ms = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) == 0
        return ms.value

    def destroy(self, arr):
        for ev in arr:
            self.hip.hipEventDestroy(ctypes.c_void_p(ev))


def cpu_baseline(wl, target_flops):
    """Time the oracle's encoder layer on the first sequences of the batch whose
    useful FLOPs reach `target_flops` (single thread)."""
    import oracle
    from workloads import BIAS_NAMES, LN_NAMES, WEIGHT_NAMES

    cfg = wl.cfg
    L = wl.lengths
    n, acc = 0, 0.0
    while n < len(L) and acc < target_flops:
        acc += useful_flops(L[n:n + 1], cfg.d_model, cfg.d_ff)
        n += 1
    Ls = L[:n]
    x = wl.tensors["x"][:int(Ls.sum())]
    w = {k: wl.tensors[k] for k in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    t0 = time.perf_counter()
    oracle.encoder_layer("bf16", Ls, x, w, cfg.d_model, cfg.heads, cfg.d_ff)
    dt = time.perf_counter() - t0
    fl = useful_flops(Ls, cfg.d_model, cfg.d_ff)
    return {"value": round(fl / dt / 1e12, 6), "unit": "TFLOP/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of {len(L)} sequences ({int(Ls.sum())} tokens), full layer, same weights; "
                      f"{dt:.1f} s for {fl:.3g} useful FLOP; host has {os.cpu_count()} logical CPUs, oracle is single-threaded",
            "ms_per_layer_extrapolated": round(useful_flops(L, cfg.d_model, cfg.d_ff) / (fl / dt) * 1e3, 1)}


def _counter_per_dispatch(path, counter):
    """kernel name -> mean counter value per dispatch (KiB for FETCH_SIZE / WRITE_SIZE)."""
    import csv
    import collections

    tot, cnt = collections.defaultdict(float), collections.defaultdict(int)
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            tot[r["Kernel_Name"]] += float(r["Counter_Value"])
            cnt[r["Kernel_Name"]] += 1
    return {k: tot[k] / cnt[k] for k in tot}


def _short(name):
    """Demangled kernel name -> 'k_name<args>' as returned by stage_kernels()."""
    base = name.replace("rag::(anonymous namespace)::", "").replace("void ", "", 1)
    return base.split("(")[0].strip()


def derive_traffic(fetch_csv, write_csv, cal_fetch_csv, cal_write_csv, copy_mib, kernels=None, tag=None):
    """HBM bytes per launch of every library kernel: FETCH_SIZE + WRITE_SIZE (KiB per
    dispatch), each scaled by copy_bytes / counter for a plain copy of known size.
    With `kernels` (base names, no template arguments), only those entries are replaced in the existing
    file, so each kernel's figure can come from a run in which all its dispatches
    have the shape the bench line reports.  With `tag`, entries are stored as
    "name@tag" (one workload's dispatches of a symbol that runs at several shapes)."""
    fetch, write = _counter_per_dispatch(fetch_csv, "FETCH_SIZE"), _counter_per_dispatch(write_csv, "WRITE_SIZE")
    cf, cw = _counter_per_dispatch(cal_fetch_csv, "FETCH_SIZE"), _counter_per_dispatch(cal_write_csv, "WRITE_SIZE")
    big = lambda d: max(d.values())  # the copy kernel is the dispatch with the largest counts
    copy_kib = copy_mib * 1024.0
    sf, sw = copy_kib / big(cf), copy_kib / big(cw)
    out = {"_calibration": {"copy_mib": copy_mib, "fetch_scale": sf, "write_scale": sw,
                            "copy_fetch_kib": big(cf), "copy_write_kib": big(cw)}}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if (kernels is not None or tag) and os.path.exists(path):
        out = {**json.load(open(path)), **out}
    for k in fetch:
        short = _short(k)
        src = KERNEL_SOURCES.get(short.split("<")[0])
        if src is None or (kernels is not None and short.split("<")[0] not in kernels):
            continue
        out[short + (f"@{tag}" if tag else "")] = {"bytes_per_launch": round((fetch[k] * sf + write.get(k, 0.0) * sw) * 1024.0),
                      "fetch_kib_raw": fetch[k], "write_kib_raw": write.get(k), "source_sha": source_hash(src)}
    with open(path, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    print(json.dumps(out, indent=1, sort_keys=True))


def _timed(fn, iters=20, warm_ms=150.0):
    """Mean ms per call of fn on the current stream: fn runs untimed until the GPU has
    been busy for warm_ms (its clock ramps up over the first tens of ms of load),
    then `iters` calls are timed with events."""
    import torch

    t0 = time.perf_counter()
    n = 0
    while n < 5 or (time.perf_counter() - t0) * 1e3 < warm_ms:
        fn()
        n += 1
        if n % 5 == 0:
            torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters


def masked_measurement(rag, plan, wl, x, wstruct, ws, y, flags, iters=20):
    """Masked (causal) attention on the same batch: the fused kernel with and without the
    mask on packed Q, K, V of the layer's shape, and the masked layer.  Useful FLOPs of
    masked attention count the lower triangles only: 2 * d * sum L (L + 1)."""
    import torch

    cfg = wl.cfg
    L = wl.lengths.astype(np.float64)
    T, d, dff = wl.total_tokens, cfg.d_model, cfg.d_ff
    g = torch.Generator(device="cuda").manual_seed(1)
    q, k, v = (torch.randn(T, d, device="cuda", generator=g).bfloat16() for _ in range(3))
    o = torch.empty(T, d, device="cuda", dtype=torch.bfloat16)
    scale = 1.0 / math.sqrt(64)

    timed = lambda fn: _timed(fn, iters)

    rag.ragged_offsets(plan)
    ms_full = timed(lambda: rag.ragged_attention(plan, q, k, v, o, scale))
    ms_mask = timed(lambda: rag.ragged_attention_causal(plan, q, k, v, o, scale))
    ms_layer = timed(lambda: rag.encoder_layer(plan, x, y, wstruct, dff, ws, flags=flags | rag.RAG_LAYER_CAUSAL))
    assert not plan.data_errors(), plan.data_errors()
    fl_mask = 2.0 * d * float((L * (L + 1)).sum())
    fl_layer = 2.0 * T * d * (4 * d + 2 * dff) + fl_mask
    return {"attention_ms": round(ms_mask, 4), "attention_unmasked_ms": round(ms_full, 4),
            "speedup_vs_unmasked": round(ms_full / ms_mask, 3),
            "attention_useful_tflops": round(fl_mask / (ms_mask * 1e-3) / 1e12, 1),
            "layer_ms": round(ms_layer, 4), "layer_useful_tflops": round(fl_layer / (ms_layer * 1e-3) / 1e12, 1),
            "note": "fused causal attention and the masked layer (plan included once, not per call)"}


def sdpa_measurement(rag, cid, seed=0, iters=30):
    """The unfused ragged attention operators one by one (ragged_offsets,
    ragged_qkt, ragged_softmax, ragged_attn_v; bf16, scale 1/8) on configuration
    `cid`'s lengths and shape, each against its own roofline: the prelude and the
    softmax as algorithmic bytes / time against HBM, QK^T and Attn.V as useful
    FLOPs / time against bf16 MFMA peak (their bytes are reported too: the score
    buffer makes them HBM-heavy)."""
    import torch

    from tests.helpers import dev
    from workloads import CONFIGS, make_workload

    cfg = CONFIGS[cid]
    wl = make_workload(cid, seed=seed)
    L = wl.lengths.astype(np.int64)
    T, d, H = wl.total_tokens, cfg.d_model, cfg.heads
    s2 = float((L * L).sum())
    plan = rag.Plan(torch.from_numpy(wl.lengths).cuda(), T, cfg.max_len, H)
    if cfg.kind == "sdpa":
        q, k, v = (dev(wl.tensors[n], "bf16").view(T, d) for n in ("q", "k", "v"))
    else:
        g = torch.Generator(device="cuda").manual_seed(1)
        q, k, v = (torch.randn(T, d, device="cuda", generator=g).bfloat16() for _ in range(3))
    n_s = int(H * s2)
    S = torch.empty(n_s, dtype=torch.bfloat16, device="cuda")
    P = torch.empty_like(S)
    O = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    rag.ragged_offsets(plan)
    torch.cuda.synchronize()
    n_qkt, n_av = int(plan.status[1].item()), int(plan.status[2].item())
    ms_off = _timed(lambda: rag.ragged_offsets(plan), iters)
    ms_qkt = _timed(lambda: rag.ragged_qkt(plan, q, k, S, 0.125), iters)
    ms_sm = _timed(lambda: rag.ragged_softmax(plan, S, P), iters)
    ms_av = _timed(lambda: rag.ragged_attn_v(plan, P, v, O), iters)
    assert not plan.data_errors(), plan.data_errors()
    e = 2.0
    B = len(L)  # lengths in; tok_off, att_off, order, two item prefixes, tok_seq, items, status out
    by = {"offsets": 4.0 * B + 4.0 * (B + 1) + 8.0 * (B + 1) + 4.0 * B + 8.0 * (B + 1) + 4.0 * T + 16.0 * n_qkt
                     + 12.0 * n_av + 16.0,
          "qkt": e * (2 * T * d + H * s2), "softmax": e * 2 * H * s2, "attn_v": e * (H * s2 + 2 * T * d)}
    fl = {"qkt": 2.0 * d * s2, "attn_v": 2.0 * d * s2}
    ms = {"offsets": ms_off, "qkt": ms_qkt, "softmax": ms_sm, "attn_v": ms_av}
    ops = {}
    for n, t in ms.items():
        o = {"ms": round(t, 5), "algorithmic_bytes": by[n], "GB_per_s": round(by[n] / (t * 1e-3) / 1e9, 1),
             "frac_of_hbm_peak": round(by[n] / (t * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
        if n in fl:
            o["useful_tflops"] = round(fl[n] / (t * 1e-3) / 1e12, 1)
            o["frac_of_bf16_peak"] = round(fl[n] / (t * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
        hbm = [load_traffic(f"{k}@{SDPA_TAGS[cid]}") for k in SDPA_KERNELS[n]] if cid in SDPA_TAGS else [None]
        if None not in hbm:  # counter-measured HBM bytes of the operator's kernels (one call)
            o["hbm_bytes_per_call"] = sum(hbm)
            o["hbm_GB_per_s"] = round(sum(hbm) / (t * 1e-3) / 1e9, 1)
            o["hbm_frac_of_peak"] = round(sum(hbm) / (t * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
        ops[n] = o
    return {"workload": f"config {cid}: batch {cfg.batch}, lengths {cfg.lengths.replace(':', ' ')}, {H} heads x 64, bf16, "
                        f"T = {T}, {n_s} scores", "ops": ops,
            "kernels": {"offsets": "k_plan_fused" if len(L) <= 256 else
                        "k_plan_small + k_plan_fill" if len(L) <= 1024 else "k_plan_scan/rank/items/fill",
                        "qkt": "k_qkt_bf16", "softmax": "k_softmax<true>", "attn_v": "k_attn_v_bf16"}}


def uniform_control_measurement(rag, iters=30):
    """A control for the cost of raggedness (the overhead study of Section 7.4 and
    Appendix D runs a batch of 64 sequences all of length 512): the batch-128 layer
    shape (d_model 1024, 16 heads x 64, FFN 4096, bf16) on 64 sequences of exactly
    512 tokens, so nothing is padded and every tile is full.  The layer runs with
    its plan built inside the QKV projection's launch (as the bench line does) and
    with the plan built once and reused; their difference is what the ragged
    machinery costs per layer, and the useful rate beside the ragged batch-128 one
    shows what the lengths' spread costs the kernels."""
    import torch

    from tests.helpers import dev
    from workloads import BIAS_NAMES, CONFIGS, LN_NAMES, WEIGHT_NAMES, make_workload

    wl = make_workload(4, seed=0)  # its weights; x is its first 32768 token rows
    cfg = wl.cfg
    d, H, dff = cfg.d_model, cfg.heads, cfg.d_ff
    L = np.full(64, 512, dtype=np.int32)
    T = int(L.sum())
    plan = rag.Plan(torch.from_numpy(L).cuda(), T, 512, H)
    x = dev(wl.tensors["x"], "bf16")[:T].contiguous()
    wd = {n: dev(wl.tensors[n], "bf16") for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    wstruct = rag.layer_weights(wd)
    ws = torch.empty(rag.encoder_layer_workspace(T, 512, d, H, dff, rag.RAG_BF16, 0), dtype=torch.uint8,
                     device="cuda")
    y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    ms = _timed(lambda: rag.encoder_layer(plan, x, y, wstruct, dff, ws, flags=rag.RAG_LAYER_BUILD_PLAN), iters)
    ms_reused = _timed(lambda: rag.encoder_layer(plan, x, y, wstruct, dff, ws), iters)
    assert not plan.data_errors(), plan.data_errors()
    uf = useful_flops(L, d, dff)
    return {"workload": f"batch 64, lengths fixed 512, {H} heads x 64, FFN {dff}, bf16, T = {T}",
            "ms_per_layer": round(ms, 4), "ms_per_layer_plan_reused": round(ms_reused, 4),
            "plan_share": round((ms - ms_reused) / ms, 4),
            "useful_tflops": round(uf / (ms * 1e-3) / 1e12, 1),
            "frac_of_bf16_peak": round(uf / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}


def other_configs_measurement(rag, iters=30):
    """The other four configurations of the workload table, each on its own path:
    1 (fp32, operator-level SDPA: prelude + ragged_qkt + ragged_softmax +
    ragged_attn_v), 2 (bf16 SDPA: the fused kernel, and the operator chain), 3 and 5
    (bf16 encoder layers, prelude included per layer).  Useful FLOPs count real
    tokens only; the padded fraction compares them with every sequence padded to
    the batch's longest."""
    import torch

    from tests.helpers import dev
    from workloads import BIAS_NAMES, CONFIGS, LN_NAMES, WEIGHT_NAMES, make_workload

    out = {}
    for cid in (1, 2, 3, 5):
        cfg = CONFIGS[cid]
        wl = make_workload(cid, seed=0)
        L = wl.lengths.astype(np.float64)
        T, d, H, dff = wl.total_tokens, cfg.d_model, cfg.heads, cfg.d_ff
        s2 = float((L * L).sum())
        plan = rag.Plan(torch.from_numpy(wl.lengths).cuda(), T, cfg.max_len, H)
        rec = {"workload": f"config {cid}: batch {cfg.batch}, lengths {cfg.lengths}, {H} heads x 64"
                           + (f", FFN {dff}" if dff else "") + f", {cfg.dtype}, T = {T}"}
        if cfg.kind == "sdpa":
            q, k, v = (dev(wl.tensors[n], cfg.dtype).view(T, d) for n in ("q", "k", "v"))
            tdt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
            S = torch.empty(int(H * s2), dtype=tdt, device="cuda")
            O = torch.empty(T, d, dtype=tdt, device="cuda")

            def chain():
                rag.ragged_offsets(plan)
                rag.ragged_qkt(plan, q, k, S, 0.125)
                rag.ragged_softmax(plan, S)
                rag.ragged_attn_v(plan, S, v, O)

            fl = 4.0 * d * s2
            ms = _timed(chain, iters)
            rec.update({"operator_chain_ms": round(ms, 4),
                        "operator_chain_useful_tflops": round(fl / (ms * 1e-3) / 1e12, 2)})
            if cfg.dtype == "bf16":
                rag.ragged_offsets(plan)
                ms_f = _timed(lambda: rag.ragged_attention(plan, q, k, v, O, 0.125), iters)
                rec.update({"fused_attention_ms": round(ms_f, 4),
                            "fused_attention_useful_tflops": round(fl / (ms_f * 1e-3) / 1e12, 2)})
            rec["padded_fraction"] = round(1.0 - s2 / (len(L) * float(L.max()) ** 2), 4)
        else:
            x = dev(wl.tensors["x"], "bf16")
            wd = {n: dev(wl.tensors[n], "bf16") for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
            wstruct = rag.layer_weights(wd)
            ws = torch.empty(rag.encoder_layer_workspace(T, cfg.max_len, d, H, dff, rag.RAG_BF16, 0),
                             dtype=torch.uint8, device="cuda")
            y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")

            # the layer builds its plan (the prelude rides in the QKV projection's launch)
            ms = _timed(lambda: rag.encoder_layer(plan, x, y, wstruct, dff, ws, flags=rag.RAG_LAYER_BUILD_PLAN), iters)
            ms_reused = _timed(lambda: rag.encoder_layer(plan, x, y, wstruct, dff, ws), iters)
            uf = useful_flops(L, d, dff)
            rec.update({"ms_per_layer": round(ms, 4),
                        "ms_per_layer_prelude_amortised_6_layers": round((ms + 5 * ms_reused) / 6, 4),
                        "useful_tflops": round(uf / (ms * 1e-3) / 1e12, 1),
                        "frac_of_bf16_peak": round(uf / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                        "padded_fraction": round(padded_fraction(L, d, dff), 4)})
            if cid == 3:
                # the same layer in fp32 (fp32 storage, products and accumulation; the
                # operator attention chain), against the fp32 matrix peak
                from workloads import bf16_bits_to_f32
                xf = dev(bf16_bits_to_f32(wl.tensors["x"]), "f32")
                wdf = {n: dev(bf16_bits_to_f32(wl.tensors[n]), "f32") for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
                wf = rag.layer_weights(wdf)  # wdf keeps the tensors alive
                wsf = torch.empty(rag.encoder_layer_workspace(T, cfg.max_len, d, H, dff, rag.RAG_F32, 0),
                                  dtype=torch.uint8, device="cuda")
                yf = torch.empty(T, d, dtype=torch.float32, device="cuda")
                msf = _timed(lambda: rag.encoder_layer(plan, xf, yf, wf, dff, wsf, flags=rag.RAG_LAYER_BUILD_PLAN),
                             iters)
                rec["fp32_layer"] = {"ms_per_layer": round(msf, 4),
                                     "useful_tflops": round(uf / (msf * 1e-3) / 1e12, 2),
                                     "frac_of_f32_peak": round(uf / (msf * 1e-3) / 1e12 / PEAK_F32_TFLOPS, 4)}
        assert not plan.data_errors(), plan.data_errors()
        out[f"config{cid}"] = rec
    return out


def measured_peaks(rag, iters=20):
    """What this GPU sustains next to its published peaks: HBM as torch's 1 GiB
    device-to-device copy (bytes read + written per second; a lower bound on the
    sustainable rate, the LayerNorm kernel reaches 6.5 TB/s), and bf16 matrix
    throughput of hipBLASLt (through torch.mm) and of this library's packed_linear
    on an 8192^3 product."""
    import torch

    n = (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ms_copy = _timed(lambda: dst.copy_(src), iters)
    gbs = 2.0 * n * 4 / (ms_copy * 1e-3) / 1e9
    del src, dst
    m = 8192
    g = torch.Generator(device="cuda").manual_seed(3)
    a = torch.randn(m, m, device="cuda", generator=g).bfloat16()
    b = torch.randn(m, m, device="cuda", generator=g).bfloat16()
    c = torch.empty(m, m, device="cuda", dtype=torch.bfloat16)
    fl = 2.0 * m ** 3
    # y = a b^T, the layout of a linear layer (a 2-D product: hipBLASLt's fastest form
    # here, ~1.65 PFLOP/s, against ~1.25 with a contiguous [K, N] operand)
    ms_blas = _timed(lambda: torch.mm(a, b.t(), out=c), iters)
    ms_ours = _timed(lambda: rag.packed_linear(a, b, c), iters)
    return {"hbm_torch_copy_GB_per_s": round(gbs, 1), "hbm_torch_copy_frac_of_peak": round(gbs / PEAK_HBM_GBS, 4),
            "bf16_gemm_8192_hipblaslt_tflops": round(fl / (ms_blas * 1e-3) / 1e12, 1),
            "bf16_gemm_8192_packed_linear_tflops": round(fl / (ms_ours * 1e-3) / 1e12, 1),
            "note": "the roofline fractions in this line are against the published peaks "
                    f"({PEAK_HBM_GBS:.0f} GB/s, {PEAK_BF16_TFLOPS:.0f} TFLOP/s bf16)"}


def vgemm_measurement(rag, batch=128, iters=20):
    """Variable-sized batched GEMM (the paper's matrix-multiplication experiment):
    `batch` problems with m, n, k uniform over the multiples of 128 in [512, 1408],
    packed operands, against two library stand-ins on the same sizes: a fully
    padded batched GEMM (every problem padded to the largest m, n, k; torch.bmm)
    and one library GEMM per problem (torch.matmul in a loop).  Useful FLOPs are
    2 * sum m n k for all three."""
    import torch

    from workloads import draw_vgemm_dims

    dims = draw_vgemm_dims(batch, np.random.default_rng(batch))
    d64 = dims.astype(np.int64)
    a_n, b_n, c_n = (int(v) for v in ((d64[:, 0] * d64[:, 2]).sum(), (d64[:, 1] * d64[:, 2]).sum(),
                                       (d64[:, 0] * d64[:, 1]).sum()))
    g = torch.Generator(device="cuda").manual_seed(2)
    a = torch.randn(a_n, device="cuda", generator=g).bfloat16()
    b = torch.randn(b_n, device="cuda", generator=g).bfloat16()
    c = torch.empty(c_n, device="cuda", dtype=torch.bfloat16)
    plan = rag.VgemmPlan(torch.from_numpy(dims).cuda(), host_dims=dims)
    rag.vgemm_offsets(plan)

    timed = lambda fn: _timed(fn, iters)

    ms = timed(lambda: rag.ragged_vgemm(plan, a, b, c))
    assert not plan.data_errors(), plan.data_errors()
    ms_plan = timed(lambda: rag.vgemm_offsets(plan))
    useful = 2.0 * float((d64[:, 0] * d64[:, 1] * d64[:, 2]).sum())
    M, N, K = (int(v) for v in dims.max(axis=0))
    ap = torch.randn(batch, M, K, device="cuda", generator=g).bfloat16()
    bp = torch.randn(batch, K, N, device="cuda", generator=g).bfloat16()   # contiguous [K, N] right operands
    cp = torch.empty(batch, M, N, device="cuda", dtype=torch.bfloat16)
    ms_pad = timed(lambda: torch.bmm(ap, bp, out=cp))
    del ap, bp, cp
    offs = np.concatenate([[0], np.cumsum(d64[:, 0] * d64[:, 2])]), np.concatenate([[0], np.cumsum(d64[:, 1] * d64[:, 2])])
    coff = np.concatenate([[0], np.cumsum(d64[:, 0] * d64[:, 1])])
    views = [(a[offs[0][p]:offs[0][p + 1]].view(m, k), b[offs[1][p]:offs[1][p + 1]].view(n, k).t(),
              c[coff[p]:coff[p + 1]].view(m, n)) for p, (m, n, k) in enumerate(d64.tolist())]

    def per_problem():
        for x, wt, y in views:
            torch.matmul(x, wt, out=y)

    ms_loop = timed(per_problem)
    tf = useful / (ms * 1e-3) / 1e12
    alg_bytes = 2.0 * (a_n + b_n + c_n)
    return {"workload": f"vgemm, batch {batch}, m n k uniform over multiples of 128 in [512, 1408] (seed {batch})",
            "ms": round(ms, 4), "useful_tflops": round(tf, 1), "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "kernel": "k_vgemm_bf16", "tiles": plan.n_tiles(), "plan_ms": round(ms_plan, 4),
            "algorithmic_bytes": alg_bytes, "hbm_bytes_per_launch": load_traffic("k_vgemm_bf16"),
            "padded_bmm_ms": round(ms_pad, 4), "speedup_vs_padded_bmm": round(ms_pad / ms, 3),
            "per_problem_matmul_ms": round(ms_loop, 4), "speedup_vs_per_problem_matmul": round(ms_loop / ms, 3),
            "useful_fraction_of_padded": round(useful / (2.0 * batch * M * N * K), 4),
            "note": "library stand-ins run hipBLASLt through torch on the same sizes (padded: every problem "
                    "at the batch's largest m, n, k)"}


def trmm_measurement(rag, n=8192, m=8192, iters=20):
    """Triangular matrix multiplication (the paper's trmm experiment): C = tril(L) B
    with L n x n and B n x m in bf16, against the dense product of the same
    (zero-filled) triangle with torch.matmul, the fully padded GEMM the paper
    compares with.  Useful FLOPs: m n (n + 1) (the k <= i multiply-adds)."""
    import torch

    g = torch.Generator(device="cuda").manual_seed(3)
    L = torch.randn(n, n, device="cuda", generator=g).bfloat16().tril_()
    B = torch.randn(n, m, device="cuda", generator=g).bfloat16()
    C = torch.empty(n, m, device="cuda", dtype=torch.bfloat16)

    timed = lambda fn: _timed(fn, iters)

    ms = timed(lambda: rag.ragged_trmm(L, B, C))
    ms_dense = timed(lambda: torch.matmul(L, B, out=C))
    useful = float(m) * n * (n + 1)
    tf = useful / (ms * 1e-3) / 1e12
    return {"workload": f"trmm, lower-triangular {n} x {n} times dense {n} x {m}, bf16",
            "ms": round(ms, 4), "useful_tflops": round(tf, 1), "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "kernel": "k_trmm_bf16", "dense_matmul_ms": round(ms_dense, 4),
            "algorithmic_bytes": 2.0 * (n * (n + 1) / 2 + 2.0 * n * m), "hbm_bytes_per_launch": load_traffic("k_trmm_bf16"),
            "speedup_vs_dense_matmul": round(ms_dense / ms, 3),
            "note": "dense stand-in: torch.matmul (hipBLASLt) of the zero-filled triangle, 2 n^2 m FLOPs"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps first (the GPU clock needs tens of ms of load to settle)")
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--flags", type=int, default=0, help="encoder_layer flags (1 = unfused attention)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-masked", action="store_true", help="skip the masked (causal) attention measurement")
    ap.add_argument("--no-vgemm", action="store_true", help="skip the variable-sized batched GEMM measurement")
    ap.add_argument("--no-trmm", action="store_true", help="skip the triangular matrix multiplication measurement")
    ap.add_argument("--no-sdpa", action="store_true", help="skip the unfused attention operator measurements")
    ap.add_argument("--no-configs", action="store_true", help="skip configurations 1, 2, 3 and 5")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured HBM copy and 8192^3 GEMM rates")
    ap.add_argument("--layer-only", action="store_true",
                    help="time the layer steps only (no auxiliary measurements, no CPU baseline), so that a "
                         "profile of the run sees every dispatch of the layer's kernels at the layer's shape")
    ap.add_argument("--ops-only", type=int, default=0, choices=(0, 2, 4), metavar="CONFIG",
                    help="only time the unfused attention operators on configuration 2 or 4 and print their entry "
                         "(the run a profile of those kernels uses)")
    ap.add_argument("--cpu-target-flops", type=float, default=2.0e10)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (counter calibration) and exit")
    ap.add_argument("--derive-traffic", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "CAL_FETCH_CSV", "CAL_WRITE_CSV"),
                    help="turn rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE counter files of a bench run and of a "
                         "copy-calibration run into profiles/traffic.json, then exit")
    ap.add_argument("--copy-mib", type=int, default=512, help="size of the calibration copy (for --derive-traffic)")
    ap.add_argument("--traffic-tag", default=None, help="store --derive-traffic entries as name@TAG")
    ap.add_argument("--traffic-kernels", default=None,
                    help="comma-separated kernel base names (e.g. k_vgemm_bf16): --derive-traffic replaces only their entries")
    args = ap.parse_args()
    if args.layer_only:
        args.no_masked = args.no_sdpa = args.no_vgemm = args.no_trmm = True
        args.no_configs = args.no_peaks = args.no_cpu_baseline = True
    if args.derive_traffic:
        kernels = set(args.traffic_kernels.split(",")) if args.traffic_kernels else None
        derive_traffic(*args.derive_traffic, copy_mib=args.copy_mib, kernels=kernels, tag=args.traffic_tag)
        return
    if args.copy_calibration:
        import torch

        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_mib": args.copy_calibration, "repeats": 5}))
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the build targets a single MI355X; sharding is a design note only)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2110_10221_amd as rag
    from tests.helpers import dev
    from workloads import BIAS_NAMES, LN_NAMES, WEIGHT_NAMES, make_workload

    torch.cuda.set_device(0)
    if args.ops_only:
        print(json.dumps({SDPA_TAGS[args.ops_only]: sdpa_measurement(rag, args.ops_only)}))
        return
    wl = make_workload(args.config, seed=args.seed)
    cfg = wl.cfg
    L = wl.lengths
    T, d, H, dff = wl.total_tokens, cfg.d_model, cfg.heads, cfg.d_ff
    s2 = float((L.astype(np.float64) ** 2).sum())
    max_len = cfg.max_len
    lens = torch.from_numpy(L).cuda()
    plan = rag.Plan(lens, T, max_len, H)
    x = dev(wl.tensors["x"], "bf16")
    wd = {n: dev(wl.tensors[n], "bf16") for n in WEIGHT_NAMES + BIAS_NAMES + LN_NAMES}
    wstruct = rag.layer_weights(wd)
    ws = torch.empty(rag.encoder_layer_workspace(T, max_len, d, H, dff, rag.RAG_BF16, args.flags),
                     dtype=torch.uint8, device="cuda")
    y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    hip = HipEvents()
    n_ev = rag.RAG_LAYER_EVENTS

    # one step = the prelude and the layer: encoder_layer builds the batch's plan
    # itself (RAG_LAYER_BUILD_PLAN: the prelude's workgroups ride in the QKV
    # projection's launch, behind its tiles)
    def step(ev=None, pre=None, flags=args.flags | rag.RAG_LAYER_BUILD_PLAN):
        if pre is not None:
            hip.record(pre, sh)
        rag.encoder_layer(plan, x, y, wstruct, dff, ws, flags=flags, events=ev)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    assert not plan.data_errors(), plan.data_errors()

    # the timed steps run bare: an event recorded between two stages costs a few
    # microseconds of its own, so the per-stage breakdown comes from a second,
    # untimed run of the same steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = elapsed * 1e3 / args.steps

    n_bd = min(args.steps, 20)
    events = [hip.create(n_ev) for _ in range(n_bd)]
    for k in range(n_bd):
        step(events[k])
    torch.cuda.synchronize()
    stage_ms = {s: 0.0 for s in STAGES}
    for k in range(n_bd):
        for i, s in enumerate(STAGES):
            stage_ms[s] += hip.elapsed(events[k][i], events[k][i + 1])
    stage_ms = {s: v / n_bd for s, v in stage_ms.items()}
    for arr in events:
        hip.destroy(arr)

    # the same layer with its plan built once and reused (the paper shares the
    # prelude's arrays across a model's layers): the amortised figure below
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(flags=args.flags)
    torch.cuda.synchronize()
    ms_reused = (time.perf_counter() - t0) * 1e3 / args.steps

    uf = useful_flops(L, d, dff)
    work = stage_work(T, d, H, dff, s2)
    # group stages by kernel symbol; the dominant kernel has the largest total time
    per_kernel = {}
    for s, kname in stage_kernels(T, d, dff).items():
        fl, by = work[s]
        pk = per_kernel.setdefault(kname, {"ms": 0.0, "flops": 0.0, "bytes": 0.0, "launches": 0})
        pk["ms"] += stage_ms[s]
        pk["flops"] += fl
        pk["bytes"] += by
        pk["launches"] += 1
    dom = max(per_kernel, key=lambda k: per_kernel[k]["ms"])
    pk = per_kernel[dom]
    avg_ms = pk["ms"] / pk["launches"]
    if dom.startswith("k_gemm") or dom.startswith("k_attention"):
        achieved = pk["flops"] / pk["launches"] / (avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    else:
        achieved = pk["bytes"] / pk["launches"] / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["traffic"] = load_traffic(dom)
    roof["kernel"] = dom
    roof["avg_launch_ms"] = round(avg_ms, 5)
    roof["launches_per_step"] = pk["launches"]

    gemm_ms = sum(stage_ms[s] for s in ("qkv_proj", "out_proj", "ff1", "ff2"))
    gemm_fl = sum(work[s][0] for s in ("qkv_proj", "out_proj", "ff1", "ff2"))
    attn_ms = sum(stage_ms[s] for s in ("qkt", "softmax", "attention"))
    out = {
        "metric": METRIC,
        "value": round(uf / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"ragged encoder layer, batch {cfg.batch}, {length_text(cfg.lengths)} (seed {args.seed}), "
                               f"d_model {d}, {H} heads x 64, FFN {dff}, GELU, post-LN",
                   "global_batch": cfg.batch, "total_tokens": T, "max_len": int(L.max()),
                   "parallelism": "single GPU", "attention": "unfused" if args.flags & 1 else "fused"},
        "ms_per_layer": round(ms_step, 4),
        "ms_per_layer_prelude_amortised_6_layers": round((ms_step + 5 * ms_reused) / 6, 4),
        "ms_per_layer_plan_reused": round(ms_reused, 4),
        "useful_tflop_per_layer": round(uf / 1e12, 4),
        "frac_of_bf16_peak": round(uf / (ms_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "padded_fraction": round(padded_fraction(L, d, dff), 4),
        "gemm_tflops": round(gemm_fl / (gemm_ms * 1e-3) / 1e12, 1),
        "gemm_frac_of_peak": round(gemm_fl / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "attention_tflops": round(work["attention"][0] / (attn_ms * 1e-3) / 1e12, 1) if attn_ms > 0 else None,
        "prelude": "built by the layer, its workgroups in the QKV projection's launch (qkv_proj stage)",
        "stage_ms": {s: round(v, 4) for s, v in stage_ms.items()},
        "ms_per_step_with_stage_events": round(sum(stage_ms.values()), 4),
        "roofline": roof,
    }
    if not args.no_masked:
        out["masked"] = masked_measurement(rag, plan, wl, x, wstruct, ws, y, args.flags)
    if not args.no_sdpa:
        out["sdpa_unfused"] = {"sdpa_b32": sdpa_measurement(rag, 2), "layer_b128": sdpa_measurement(rag, 4)}
    if not args.no_vgemm:
        out["vgemm"] = vgemm_measurement(rag)
    if not args.no_trmm:
        out["trmm"] = trmm_measurement(rag)
    if not args.no_configs:
        out["other_configs"] = other_configs_measurement(rag)
        out["uniform_control"] = uniform_control_measurement(rag)
    if not args.no_peaks:
        out["measured_peaks"] = measured_peaks(rag)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_target_flops)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out))


if __name__ == "__main__":
    main()
