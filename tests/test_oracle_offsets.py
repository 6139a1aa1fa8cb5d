"""Pins of the oracle's prelude arrays (offsets, order, token map, work lists).

Each check compares the oracle with something other than itself: hand-worked
values, closed forms evaluated by numpy, a brute-force tile enumeration, or a
library sort.
"""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "offsets_lengths_7_33_64_128_h2.txt")


def _read_golden(path):
    out = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = [int(v) for v in vals]
    return out


def test_golden_worked_example():
    g = _read_golden(GOLDEN)
    p = oracle.offsets(g["lengths"], g["heads"][0])
    assert p.rc == 0
    assert p.tok_off.tolist() == g["tok_off"]
    assert p.att_off.tolist() == g["att_off"]
    assert p.order.tolist() == g["order"]
    assert len(p.qkt_items) == g["n_qkt"][0]
    assert len(p.av_items) == g["n_av"][0]


def _random_lengths(rng, B, lo=0, hi=300):
    return rng.integers(lo, hi + 1, size=B).astype(np.int32)


@pytest.mark.parametrize("seed", range(6))
def test_prefix_sums_closed_form(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40))
    H = int(rng.integers(1, 17))
    L = _random_lengths(rng, B)
    p = oracle.offsets(L, H)
    Li = L.astype(np.int64)
    assert p.tok_off.tolist() == [0] + np.cumsum(Li).tolist()
    assert p.att_off.tolist() == [0] + np.cumsum(H * Li * Li).tolist()
    assert p.tok_off[-1] == Li.sum() and p.att_off[-1] == H * (Li * Li).sum()


@pytest.mark.parametrize("seed", range(6))
def test_order_is_stable_descending_sort(seed):
    rng = np.random.default_rng(100 + seed)
    B = int(rng.integers(1, 60))
    L = rng.integers(0, 8, size=B).astype(np.int32)  # many ties
    p = oracle.offsets(L, 2)
    assert p.order.tolist() == np.argsort(-L.astype(np.int64), kind="stable").tolist()


def test_token_map():
    rng = np.random.default_rng(7)
    L = _random_lengths(rng, 17, 0, 50)
    p = oracle.offsets(L, 3)
    assert p.tok_seq.tolist() == np.repeat(np.arange(L.size), L).tolist()


@pytest.mark.parametrize("tiles", [(64, 64), (32, 64), (16, 16), (64, 32)])
@pytest.mark.parametrize("seed", range(3))
def test_work_lists_cover_every_score_once(tiles, seed):
    tm, tn = tiles
    rng = np.random.default_rng(200 + seed)
    B = int(rng.integers(1, 9))
    H = int(rng.integers(1, 4))
    L = _random_lengths(rng, B, 0, 140)
    p = oracle.offsets(L, H, tm, tn)
    # brute force: paint every (b, h, i, j) covered by a qkt tile
    cover = [np.zeros((H, int(n), int(n)), np.int32) for n in L]
    for b, h, ti, tj in p.qkt_items:
        n = L[b]
        assert 0 <= ti * tm < n and 0 <= tj * tn < n
        cover[b][h, ti * tm:min(n, ti * tm + tm), tj * tn:min(n, tj * tn + tn)] += 1
    for c in cover:
        assert (c == 1).all()
    rows = [np.zeros((H, int(n)), np.int32) for n in L]
    for b, h, ti in p.av_items:
        rows[b][h, ti * tm:min(L[b], ti * tm + tm)] += 1
    for r in rows:
        assert (r == 1).all()
    # counts: closed form
    ceil = lambda a, b: -(-a // b)
    assert len(p.qkt_items) == sum(H * ceil(int(n), tm) * ceil(int(n), tn) for n in L)
    assert len(p.av_items) == sum(H * ceil(int(n), tm) for n in L)


def test_work_list_order_longest_first():
    rng = np.random.default_rng(5)
    L = _random_lengths(rng, 20, 0, 200)
    H = 3
    p = oracle.offsets(L, H)
    seqs = p.qkt_items[:, 0]
    # sequences appear in one contiguous run each, in the sorted order
    runs = [s for k, s in enumerate(seqs) if k == 0 or seqs[k - 1] != s]
    assert runs == [b for b in p.order.tolist() if L[b] > 0]
    # within a sequence: lexicographic (head, ti, tj)
    for b in set(seqs.tolist()):
        sub = p.qkt_items[seqs == b][:, 1:]
        keys = [tuple(r) for r in sub.tolist()]
        assert keys == sorted(keys)
    # per-sequence item prefix offsets agree with the lists
    for k, b in enumerate(p.order):
        q0, q1 = p.qkt_item_off[k], p.qkt_item_off[k + 1]
        assert (p.qkt_items[q0:q1, 0] == b).all()
        a0, a1 = p.av_item_off[k], p.av_item_off[k + 1]
        assert (p.av_items[a0:a1, 0] == b).all()


def test_zero_lengths_emit_nothing():
    L = np.array([0, 5, 0, 0, 70, 0], np.int32)
    p = oracle.offsets(L, 2)
    assert set(p.qkt_items[:, 0].tolist()) == {1, 4}
    assert p.tok_off.tolist() == [0, 0, 5, 5, 5, 75, 75]
    assert p.order.tolist() == [4, 1, 0, 2, 3, 5]


def test_error_codes():
    assert oracle.offsets(np.array([3, -1, 4], np.int32), 2).rc == 1
    p = oracle.offsets(np.array([100, 100], np.int32), 2, qkt_cap=3, av_cap=100)
    assert p.rc == 2
    assert len(p.qkt_items) == 3
