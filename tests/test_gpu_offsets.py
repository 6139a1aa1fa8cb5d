"""GPU parity of the prelude (ragged_offsets): bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from workloads import CONFIGS, make_workload

pytestmark = pytest.mark.gpu


def _gpu_plan(L, H, max_len=None, total=None, **caps):
    import paper_2110_10221_amd as rag

    L = np.asarray(L, np.int32)
    T = int(L.sum()) if total is None else total
    mx = int(max(L.max(), 0)) if max_len is None else max_len
    plan = rag.Plan(torch.from_numpy(L).cuda(), T, mx, H, **caps)
    rag.ragged_offsets(plan)
    torch.cuda.synchronize()
    return plan


def _check_equal(plan, L, H):
    ref = oracle.offsets(L, H)
    assert ref.rc == 0
    B, T = len(L), int(np.sum(L))
    st = plan.status.cpu().numpy()
    assert st[0] == 0, plan.data_errors()
    assert st[1] == len(ref.qkt_items) and st[2] == len(ref.av_items)
    assert st[3] == int(np.max(L))
    assert (plan.tok_off.cpu().numpy() == ref.tok_off).all()
    assert (plan.att_off.cpu().numpy() == ref.att_off).all()
    assert (plan.order.cpu().numpy() == ref.order).all()
    assert (plan.tok_seq.cpu().numpy()[:T] == ref.tok_seq).all()
    assert (plan.qkt_item_off.cpu().numpy() == ref.qkt_item_off).all()
    assert (plan.av_item_off.cpu().numpy() == ref.av_item_off).all()
    nq, na = len(ref.qkt_items), len(ref.av_items)
    assert (plan.qkt_items.cpu().numpy()[:4 * nq].reshape(-1, 4) == ref.qkt_items).all()
    assert (plan.av_items.cpu().numpy()[:3 * na].reshape(-1, 3) == ref.av_items).all()


@pytest.mark.parametrize("cid", sorted(CONFIGS))
def test_offsets_configs(cid):
    wl = make_workload(cid, seed=0)
    print(f"offsets config {cid}: B={len(wl.lengths)} T={wl.total_tokens}", flush=True)
    plan = _gpu_plan(wl.lengths, wl.cfg.heads)
    _check_equal(plan, wl.lengths, wl.cfg.heads)


@pytest.mark.parametrize("L,H", [
    ([0, 5, 0, 0, 70, 0], 2),          # zero-length sequences
    ([1], 1),                          # one token
    ([64, 64, 64, 64], 3),             # ties, exact tiles
    ([63, 65, 127, 128, 129], 16),     # tile boundaries
    ([0, 0, 0], 4),                    # no tokens at all
    ([3000, 1, 2048], 2),              # long sequences
])
def test_offsets_edge_cases(L, H):
    plan = _gpu_plan(L, H, max_len=max(max(L), 1))
    _check_equal(plan, np.asarray(L, np.int32), H)


@pytest.mark.parametrize("B", [129, 255, 256, 257, 1023, 1024, 1025, 5000, 65536])
def test_offsets_large_batches(B):
    rng = np.random.default_rng(B)
    L = rng.integers(0, 40, size=B).astype(np.int32)  # many ties
    plan = _gpu_plan(L, 2)
    _check_equal(plan, L, 2)


def test_plan_rebuild_for_new_lengths():
    import paper_2110_10221_amd as rag

    L1 = np.array([10, 200, 3], np.int32)
    L2 = np.array([150, 12, 51], np.int32)  # same total (213), new raggedness
    lens = torch.from_numpy(L1).cuda()
    plan = rag.Plan(lens, 213, 256, 4)
    rag.ragged_offsets(plan)
    lens.copy_(torch.from_numpy(L2))
    rag.ragged_offsets(plan)
    torch.cuda.synchronize()
    _check_equal(plan, L2, 4)


@pytest.mark.parametrize("L,total,max_len,caps,bit", [
    ([5, -1, 7], 11, 8, {}, 1),                       # negative length
    ([5, 9, 7], 21, 8, {}, 2),                        # length above max_len
    ([5, 6, 7], 19, 8, {}, 4),                        # wrong token total
    ([100, 100], 200, 100, {"qkt_cap": 3}, 8),        # qkt list overflow
    ([100, 100], 200, 100, {"av_cap": 1}, 16),        # av list overflow
])
def test_offsets_data_errors(L, total, max_len, caps, bit):
    plan = _gpu_plan(L, 2, max_len=max_len, total=total, **caps)
    st = plan.status.cpu().numpy()
    assert st[0] & bit
    assert st[1] == 0 and st[2] == 0


def test_sync_check_reports_data_errors():
    # RAG_SYNC_CHECK=1 (read once per process, so a child process of its own):
    # a call whose plan reports data errors returns RAG_ERR_DATA, a valid one RAG_OK
    import os
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = r"""
import sys
sys.path.insert(0, sys.argv[1])
import numpy as np, torch
import paper_2110_10221_amd as rag
plan = rag.Plan(torch.tensor([5, -3, 7], dtype=torch.int32, device="cuda"), 9, 7, 2)
try:
    rag.ragged_offsets(plan)
    raise SystemExit("negative length not reported")
except rag.RaggedError as e:
    assert e.status == -7 and "negative length" in plan.data_errors(), (str(e), plan.data_errors())
L = np.array([5, 70, 33], np.int32)
T, H, d, dff = int(L.sum()), 2, 128, 256
w = {n: torch.zeros(s, dtype=torch.bfloat16, device="cuda") for n, s in (
    ("w_qkv", (3 * d, d)), ("b_qkv", (3 * d,)), ("w_o", (d, d)), ("b_o", (d,)), ("ln1_g", (d,)), ("ln1_b", (d,)),
    ("w_ff1", (dff, d)), ("b_ff1", (dff,)), ("w_ff2", (d, dff)), ("b_ff2", (d,)), ("ln2_g", (d,)), ("ln2_b", (d,)))}
flags = rag.RAG_LAYER_BUILD_PLAN
bad = rag.Plan(torch.from_numpy(L).cuda(), T + 1, 70, H)   # token count disagrees with the lengths
ws = torch.empty(rag.encoder_layer_workspace(T + 1, 70, d, H, dff, rag.RAG_BF16, flags), dtype=torch.uint8, device="cuda")
x = torch.zeros(T + 1, d, dtype=torch.bfloat16, device="cuda")
y = torch.empty_like(x)
try:
    rag.encoder_layer(bad, x, y, w, dff, ws, flags=flags)
    raise SystemExit("token count not reported")
except rag.RaggedError as e:
    assert e.status == -7 and "sum of lengths != total_tokens" in bad.data_errors(), (str(e), bad.data_errors())
good = rag.Plan(torch.from_numpy(L).cuda(), T, 70, H)
rag.encoder_layer(good, x[:T], y[:T], w, dff, ws, flags=flags)
print("sync check ok")
"""
    env = dict(os.environ, RAG_SYNC_CHECK="1")
    r = subprocess.run([sys.executable, "-c", code, root], env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "sync check ok" in r.stdout, r.stdout + r.stderr
