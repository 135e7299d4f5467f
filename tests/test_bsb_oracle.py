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
    r0s = b.get("win_row", [16 * w for w in range(T)])
    for w in range(T):
        for blk in range(b["blk_off"][w], b["blk_off"][w + 1]):
            for r in range(16):
                for c in range(16):
                    k = _bit(r, c)
                    if (int(b["mask"][8 * blk + k // 32]) >> (k % 32)) & 1:
                        col = int(b["cols"][16 * blk + c])
                        assert col >= 0, "bit set on a padding column"
                        edges.add((int(r0s[w]) + r, col))
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


# ---- windows aligned to the graphs of a batch (Section 4.2's future work) ----

def test_segment_windows_hand_example(oracle):
    """Graphs of 15, 45, 3, 5, 20, 0 and 32 rows (N = 120), windows by hand:
    [0,15) the first graph (the 45-row graph does not fit beside it);
    [15,31) [31,47) 16-row steps of the 45-row graph, whose last 13 rows
    [47,60) take the 3-row graph too (16 rows) but not the 5-row one;
    [60,63) is packed: [63,68) the 5-row graph alone (the 20-row one does
    not fit); [68,84) a 16-row step of the 20-row graph, [84,88) its last
    4 rows with the empty graph; [88,104) [104,120) the 32-row graph."""
    got = oracle.segment_windows([0, 15, 60, 63, 68, 88, 88, 120]).tolist()
    assert got == [0, 15, 31, 47, 63, 68, 84, 88, 104, 120]


def _check_segment_windows(seg, wr):
    """The rule of segment_windows, restated as properties of the result."""
    seg = [int(x) for x in seg]
    N = seg[-1]
    wr = [int(x) for x in wr]
    assert wr[0] == 0 and wr[-1] == N
    for a, b in zip(wr, wr[1:]):
        assert 1 <= b - a <= 16
        g = max(k for k in range(len(seg) - 1) if seg[k] <= a < seg[k + 1])
        assert (a - seg[g]) % 16 == 0          # starts at a 16-row step
        rest = seg[g + 1] - a
        if rest > 16:
            assert b == a + 16                 # a step inside a long graph
        else:
            assert b in seg                    # ends at a graph boundary ...
            later = [s for s in seg if s > b]
            if later:
                assert min(later) - a > 16     # ... and the next graph did not fit


@pytest.mark.parametrize("seed", range(8))
def test_segment_windows_properties(oracle, seed):
    rng = np.random.default_rng(300 + seed)
    sizes = rng.integers(0, 50, size=int(rng.integers(1, 40)))
    sizes[rng.random(sizes.size) < 0.2] = 0
    sizes[rng.random(sizes.size) < 0.3] //= 8
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    if seg[-1] == 0:
        assert oracle.segment_windows(seg).tolist() == [0]
        return
    _check_segment_windows(seg, oracle.segment_windows(seg))


def test_segment_windows_molecule_batch(oracle):
    c = W.make_config(4, with_features=False)
    wr = oracle.segment_windows(c["seg_ptr"])
    _check_segment_windows(c["seg_ptr"], wr)
    # the batch is block-diagonal: a window's columns lie inside the graphs
    # its rows belong to
    seg = c["seg_ptr"]
    b = oracle.bsb(c["row_ptr"], c["col_idx"], c["N"], win_row=wr)
    g0 = np.searchsorted(seg, wr[:-1], side="right") - 1
    g1 = np.searchsorted(seg, wr[1:] - 1, side="right") - 1
    for w in range(len(wr) - 1):
        lo, hi = b["blk_off"][w], b["blk_off"][w + 1]
        cl = b["cols"][16 * lo:16 * hi]
        cl = cl[cl >= 0]
        assert cl.min() >= seg[g0[w]] and cl.max() < seg[g1[w] + 1]
    assert _decode(b, c["N"]) == _edges(c["row_ptr"], c["col_idx"])


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_segment_windows(oracle, seed):
    """Layout over windows of 1..16 rows against Python sets, and its decode."""
    rng = np.random.default_rng(400 + seed)
    N = int(rng.integers(1, 90))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 40), empty_frac=0.2, dup_frac=0.3)
    cuts = np.sort(rng.choice(np.arange(1, N), size=min(N - 1, int(rng.integers(0, 8))),
                              replace=False)) if N > 1 else np.array([], dtype=int)
    seg = np.concatenate([[0], cuts, [N]]).astype(np.int32)
    wr = oracle.segment_windows(seg)
    b = oracle.bsb(rp, ci, N, win_row=wr)
    T = len(wr) - 1
    assert len(b["blk_off"]) == T + 1
    for w in range(T):
        r0, r1 = int(wr[w]), int(wr[w + 1])
        distinct = sorted(set(ci[rp[r0]:rp[r1]].tolist()))
        assert b["u"][w] == len(distinct)
        assert b["nb"][w] == -(-len(distinct) // 16)
        lo, hi = b["blk_off"][w], b["blk_off"][w + 1]
        slots = b["cols"][16 * lo:16 * hi].tolist()
        assert slots == distinct + [-1] * (16 * (hi - lo) - len(distinct))
        for blk in range(lo, hi):                # no bit beyond the window's rows
            for r in range(r1 - r0, 16):
                for c in range(16):
                    k = _bit(r, c)
                    assert not (int(b["mask"][8 * blk + k // 32]) >> (k % 32)) & 1
    assert _decode(b, N) == _edges(rp, ci)


def test_window_rows_reject_bad_windows(oracle):
    rp = np.array([0, 1, 2], dtype=np.int32)
    ci = np.array([0, 1], dtype=np.int32)
    for wr in ([0, 0, 2], [0, 2, 1], [1, 2]):
        with pytest.raises(ValueError):
            oracle.bsb(rp, ci, 2, win_row=np.array(wr + ([2] if wr[-1] != 2 else []),
                                                   dtype=np.int32))
    with pytest.raises(ValueError):
        oracle.segment_windows([0, 5, 3])
