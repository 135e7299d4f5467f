"""Pins for the oracle's Binary Sparse Block layout and work list (CPU only).

Section 3.1 defines the layout (16-row windows, all-zero columns removed, the
compacted window cut into blocks, one bitmap per block; Table 3 gives its
size); Section 3.2 defines the reordering (windows by decreasing block
count).  The pins: a hand-derived fixture, brute force with Python sets on
random small patterns, an exact decode back to the pattern at workload scale,
and Table 3's footprint formula.
"""
import json
import os

import numpy as np
import pytest

from paper_2505_08098_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _bit(r, c):
    return 4 * (r + 16 * (c // 4)) + (c % 4)


def _decode(b, N):
    """Edge set encoded by a BSB layout (inverse of the construction)."""
    edges = set()
    T = len(b["blk_off"]) - 1
    for w in range(T):
        for blk in range(b["blk_off"][w], b["blk_off"][w + 1]):
            for r in range(16):
                for c in range(16):
                    k = _bit(r, c)
                    if (int(b["mask"][8 * blk + k // 32]) >> (k % 32)) & 1:
                        col = int(b["cols"][16 * blk + c])
                        assert col >= 0, "bit set on a padding column"
                        edges.add((16 * w + r, col))
    return edges


def _edges(rp, ci):
    return set((i, int(c)) for i in range(len(rp) - 1) for c in ci[rp[i]:rp[i + 1]])


def test_hand_derived_fixture(oracle):
    g = json.load(open(os.path.join(GOLD, "bsb_small.json")))
    N = g["N"]
    rows = [g["rows"].get(str(i), []) for i in range(N)]
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.array([c for r in rows for c in r], dtype=np.int32)
    b = oracle.bsb(rp, ci, N)
    assert b["u"].tolist() == g["u"]
    assert b["nb"].tolist() == g["nb"]
    assert b["blk_off"].tolist() == g["blk_off"]
    assert b["cols"].tolist() == g["cols"]
    assert b["mask"].tolist() == g["mask"]
    wl = g["worklist_case"]
    items, merges = oracle.worklist(np.array(wl["nb"]), np.array(wl["blk_off"]),
                                    wl["piece"])
    assert items.tolist() == wl["items"]
    assert merges.tolist() == wl["merges"]


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_random_patterns(oracle, seed):
    rng = np.random.default_rng(100 + seed)
    N = int(rng.integers(1, 70))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 40), empty_frac=0.2, dup_frac=0.3)
    b = oracle.bsb(rp, ci, N)
    T = (N + 15) // 16
    assert len(b["blk_off"]) == T + 1
    for w in range(T):
        r0, r1 = 16 * w, min(16 * w + 16, N)
        distinct = sorted(set(ci[rp[r0]:rp[r1]].tolist()))
        assert b["u"][w] == len(distinct)
        assert b["nb"][w] == -(-len(distinct) // 16)
        lo, hi = b["blk_off"][w], b["blk_off"][w + 1]
        assert hi - lo == b["nb"][w]
        slots = b["cols"][16 * lo:16 * hi].tolist()
        assert slots == distinct + [-1] * (16 * (hi - lo) - len(distinct))
    assert _decode(b, N) == _edges(rp, ci)


@pytest.mark.parametrize("k", [1, 4])
def test_decode_recovers_workload_pattern(oracle, k):
    c = W.make_config(k, with_features=False)
    b = oracle.bsb(c["row_ptr"], c["col_idx"], c["N"])
    assert _decode(b, c["N"]) == _edges(c["row_ptr"], c["col_idx"])


def test_table3_footprint(oracle):
    """Table 3: BSB needs 32(N/r + b c) + b r c bits (32-bit offsets and
    column ids, one r x c bitmap per block).  With r = c = 16 the arrays the
    oracle returns must have exactly those sizes (the offset array carries
    one extra closing entry)."""
    c = W.make_config(1, with_features=False)
    N = c["N"]
    b = oracle.bsb(c["row_ptr"], c["col_idx"], N)
    B = int(b["blk_off"][-1])
    bits = 32 * (len(b["blk_off"]) - 1) + 32 * len(b["cols"]) + 32 * len(b["mask"])
    assert bits == 32 * (N // 16 + B * 16) + B * 16 * 16


@pytest.mark.parametrize("piece", [2, 4, 8, 32])
def test_worklist_properties(oracle, piece):
    rng = np.random.default_rng(piece)
    nb = rng.integers(0, 40, size=300)
    nb[::37] = 0
    nb[5] = 333
    blk_off = np.concatenate([[0], np.cumsum(nb)]).astype(np.int64)
    items, merges = oracle.worklist(nb, blk_off, piece)
    # every window's blocks covered exactly once, in pieces of <= piece
    cover = {w: [] for w in range(len(nb))}
    for w, b0, b1, slot in items.tolist():
        assert b1 >= b0
        cover[w].append((b0, b1, slot))
        if slot >= 0:
            assert b1 - b0 <= piece and b0 % 2 == blk_off[w] % 2
    for w, segs in cover.items():
        segs.sort()
        assert segs[0][0] == blk_off[w] and segs[-1][1] == blk_off[w + 1]
        for (a0, a1, _), (c0, _, _) in zip(segs, segs[1:]):
            assert a1 == c0
        assert (len(segs) > 1) == (nb[w] > piece)
    # slots are 0..n-1, the merge records point at them
    slots = sorted(s for *_, s in items.tolist() if s >= 0)
    assert slots == list(range(len(slots)))
    for w, first, npieces in merges.tolist():
        assert nb[w] > piece and npieces == -(-nb[w] // piece)
        assert sorted(s for ww, *_, s in items.tolist() if ww == w) == \
            list(range(first, first + npieces))
    # heavy first: keys never increase along the list
    keys = [piece if s >= 0 else b1 - b0 for _, b0, b1, s in items.tolist()]
    assert all(a >= b for a, b in zip(keys, keys[1:]))


def test_worklist_without_reordering_keeps_window_order(oracle):
    nb = np.array([3, 0, 40, 7, 2])
    blk_off = np.concatenate([[0], np.cumsum(nb)])
    items, merges = oracle.worklist(nb, blk_off, 16, reorder=False)
    assert items[:, 0].tolist() == [0, 1, 2, 2, 2, 3, 4]
    assert merges.tolist() == [[2, 0, 3]]
    sorted_items, _ = oracle.worklist(nb, blk_off, 16)
    assert sorted_items[:, 0].tolist() == [2, 2, 2, 3, 0, 4, 1]
