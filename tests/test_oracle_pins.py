"""Pins for the oracle's 3S operator (CPU only).

Each test checks the oracle against something other than itself: a library
routine (torch's CPU attention, scipy's softmax, numpy's binary16 decoding), a
closed form, a hand-worked fixture, or an invariant of the definition
(Section 2.1 Eq. 1 with the masked reading, Section 3.5 Eq. 7).
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from paper_2505_08098_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _qkv(rng, N, d, scale=1.0):
    return tuple((scale * rng.standard_normal((N, d))).astype(np.float16)
                 for _ in range(3))


def _dense_mask(row_ptr, col_idx, N):
    m = np.zeros((N, N), dtype=bool)
    for i in range(N):
        m[i, col_idx[row_ptr[i]:row_ptr[i + 1]]] = True
    return m


def test_half_decoder_matches_numpy_on_every_bit_pattern(oracle):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_worked_example_golden(oracle):
    g = json.load(open(os.path.join(GOLD, "worked_3s.json")))
    Q = np.array(g["Q"], dtype=np.float16)
    K = np.array(g["K"], dtype=np.float16)
    V = np.array(g["V"], dtype=np.float16)
    O, P = oracle.attention_f64(g["row_ptr"], g["col_idx"], Q, K, V, g["scale"],
                                want_p=True)
    np.testing.assert_allclose(O, np.array(g["O"]), rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(P, np.array(g["P_per_entry"]), rtol=1e-14)


@pytest.mark.parametrize("N,d,seed", [(1, 8, 0), (15, 16, 1), (16, 32, 2),
                                      (17, 8, 3), (33, 24, 4), (64, 64, 5)])
def test_matches_torch_masked_attention(oracle, N, d, seed):
    """Library pin: torch's scaled_dot_product_attention (fp64, CPU) with a
    boolean mask is the masked softmax attention by definition."""
    rng = np.random.default_rng(seed)
    rp, ci = W.random_csr(rng, N, max_deg=N, dup_frac=0.3)
    # one full row to cover the dense case
    Q, K, V = _qkv(rng, N, d)
    scale = 0.37
    O = oracle.attention_f64(rp, ci, Q, K, V, scale)
    mask = _dense_mask(rp, ci, N)
    t = lambda a: torch.from_numpy(a.astype(np.float64))[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(
        t(Q), t(K), t(V), attn_mask=torch.from_numpy(mask)[None, None],
        scale=scale)[0, 0].numpy()
    rows = mask.any(axis=1)
    np.testing.assert_allclose(O[rows], ref[rows], rtol=1e-12, atol=1e-12)
    assert np.all(O[~rows] == 0)


def test_full_pattern_is_dense_softmax_attention(oracle):
    """Every row attends to every column: scipy softmax over QK^T rows."""
    rng = np.random.default_rng(11)
    N, d = 40, 16
    rp = np.arange(0, N * N + 1, N, dtype=np.int32)
    ci = np.tile(np.arange(N, dtype=np.int32), N)
    Q, K, V = _qkv(rng, N, d)
    scale = 1 / math.sqrt(d)
    S = scale * (Q.astype(np.float64) @ K.astype(np.float64).T)
    ref = scipy.special.softmax(S, axis=1) @ V.astype(np.float64)
    O = oracle.attention_f64(rp, ci, Q, K, V, scale)
    np.testing.assert_allclose(O, ref, rtol=1e-12, atol=1e-12)


def test_transposed_scores_would_fail(oracle):
    """Q K^T is not K Q^T: a non-symmetric case distinguishes them."""
    rng = np.random.default_rng(12)
    N, d = 6, 4
    rp = np.arange(0, N * N + 1, N, dtype=np.int32)
    ci = np.tile(np.arange(N, dtype=np.int32), N)
    Q, K, V = _qkv(rng, N, d)
    O = oracle.attention_f64(rp, ci, Q, K, V, 1.0)
    S_wrong = K.astype(np.float64) @ Q.astype(np.float64).T
    wrong = scipy.special.softmax(S_wrong, axis=1) @ V.astype(np.float64)
    assert np.abs(O - wrong).max() > 1e-3


def test_single_neighbour_row_is_exactly_v(oracle):
    rng = np.random.default_rng(2)
    N, d = 50, 32
    j = rng.integers(0, N, size=N)
    rp = np.arange(N + 1, dtype=np.int32)
    Q, K, V = _qkv(rng, N, d, scale=10.0)
    O = oracle.attention_f64(rp, j.astype(np.int32), Q, K, V, 3.0)
    assert np.array_equal(O, V[j].astype(np.float64))


def test_zero_queries_give_neighbour_mean(oracle):
    rng = np.random.default_rng(3)
    N, d = 64, 16
    rp, ci = W.random_csr(rng, N, max_deg=20)
    _, K, V = _qkv(rng, N, d)
    Q = np.zeros((N, d), dtype=np.float16)
    O = oracle.attention_f64(rp, ci, Q, K, V, 0.125)
    for i in range(N):
        nb = np.unique(ci[rp[i]:rp[i + 1]])
        np.testing.assert_allclose(O[i], V[nb].astype(np.float64).mean(axis=0),
                                   rtol=1e-14, atol=1e-14)


def test_probability_rows_sum_to_one(oracle):
    rng = np.random.default_rng(4)
    N, d = 200, 32
    rp, ci = W.random_csr(rng, N, max_deg=40, empty_frac=0.1, dup_frac=0.2)
    Q, K, V = _qkv(rng, N, d, scale=2.0)
    _, P = oracle.attention_f64(rp, ci, Q, K, V, 0.5, want_p=True)
    sums = np.add.reduceat(P, rp[:-1]) if len(P) else np.zeros(N)
    for i in range(N):
        if rp[i + 1] > rp[i]:
            assert abs(sums[i] - 1.0) < 1e-14
            assert np.all(P[rp[i]:rp[i + 1]] >= 0)


def test_neighbour_order_does_not_matter(oracle):
    rng = np.random.default_rng(5)
    N, d = 100, 16
    rp, ci = W.random_csr(rng, N, max_deg=30, shuffle=False)
    Q, K, V = _qkv(rng, N, d)
    O1 = oracle.attention_f64(rp, ci, Q, K, V, 0.3)
    ci2 = ci.copy()
    for i in range(N):
        seg = ci2[rp[i]:rp[i + 1]]
        rng.shuffle(seg)
    O2 = oracle.attention_f64(rp, ci2, Q, K, V, 0.3)
    np.testing.assert_allclose(O1, O2, rtol=0, atol=1e-12)


def test_node_relabelling_permutes_rows(oracle):
    rng = np.random.default_rng(6)
    N, d = 90, 8
    rp, ci = W.random_csr(rng, N, max_deg=25)
    Q, K, V = _qkv(rng, N, d)
    O = oracle.attention_f64(rp, ci, Q, K, V, 0.4)
    pi = rng.permutation(N)              # old id -> new id
    inv = np.argsort(pi)                 # new id -> old id
    rows, cols = [], []
    for new in range(N):
        old = inv[new]
        cols.append(pi[ci[rp[old]:rp[old + 1]]])
    rp2 = np.zeros(N + 1, dtype=np.int32)
    rp2[1:] = np.cumsum([c.size for c in cols])
    ci2 = np.concatenate(cols).astype(np.int32)
    O2 = oracle.attention_f64(rp2, ci2, Q[inv], K[inv], V[inv], 0.4)
    np.testing.assert_allclose(O2, O[inv], rtol=0, atol=1e-12)


def test_constant_values_are_reproduced(oracle):
    rng = np.random.default_rng(7)
    N, d = 80, 16
    rp, ci = W.random_csr(rng, N, max_deg=30, empty_frac=0.1)
    Q, K, _ = _qkv(rng, N, d, scale=3.0)
    V = np.full((N, d), 2.5, dtype=np.float16)
    O = oracle.attention_f64(rp, ci, Q, K, V, 1.0)
    nonempty = np.diff(rp) > 0
    np.testing.assert_allclose(O[nonempty], 2.5, rtol=1e-14)
    assert np.all(O[~nonempty] == 0)


@pytest.mark.parametrize("gap", [40.0, 1000.0])
def test_dominant_score_selects_one_row(oracle, gap):
    """One neighbour's score exceeds every other by ``gap``: P -> one-hot.
    gap = 1000 also exceeds the e^89 fp32 overflow point of a naive softmax."""
    N, d = 8, 4
    rp = np.array([0, N] + [N] * (N - 1), dtype=np.int32)
    ci = np.arange(N, dtype=np.int32)
    Q = np.zeros((N, d), dtype=np.float16)
    Q[0, 0] = 1.0
    K = np.zeros((N, d), dtype=np.float16)
    K[5, 0] = 1.0
    rng = np.random.default_rng(8)
    V = rng.standard_normal((N, d)).astype(np.float16)
    O = oracle.attention_f64(rp, ci, Q, K, V, gap)
    assert np.all(np.isfinite(O))
    tail = (N - 1) * math.exp(-gap) * np.abs(V.astype(np.float64)).max()
    np.testing.assert_allclose(O[0], V[5].astype(np.float64), rtol=0,
                               atol=tail + 1e-15)


def test_repeated_entries_count_once(oracle):
    rng = np.random.default_rng(9)
    N, d = 60, 16
    rp, ci = W.random_csr(rng, N, max_deg=15)
    Q, K, V = _qkv(rng, N, d)
    O1 = oracle.attention_f64(rp, ci, Q, K, V, 0.5)
    rows = []
    for i in range(N):
        seg = ci[rp[i]:rp[i + 1]]
        rows.append(np.concatenate([seg, seg[: (len(seg) + 1) // 2]]))
    rp2 = np.zeros(N + 1, dtype=np.int32)
    rp2[1:] = np.cumsum([r.size for r in rows])
    O2 = oracle.attention_f64(rp2, np.concatenate(rows).astype(np.int32), Q, K, V, 0.5)
    np.testing.assert_allclose(O1, O2, rtol=0, atol=1e-13)


def test_empty_rows_are_zero(oracle):
    rng = np.random.default_rng(10)
    N, d = 37, 8
    rp, ci = W.random_csr(rng, N, max_deg=9, empty_frac=0.5)
    Q, K, V = _qkv(rng, N, d)
    O, lse = oracle.attention_f64(rp, ci, Q, K, V, 1.0, want_lse=True)
    empty = np.diff(rp) == 0
    assert empty.any()
    assert np.all(O[empty] == 0)
    assert np.all(np.isneginf(lse[empty]))
    assert np.all(np.isfinite(lse[~empty]))


def test_malformed_csr_is_rejected(oracle):
    assert oracle.check_csr([1, 1], [0], 1) != 0          # row_ptr[0] != 0
    assert oracle.check_csr([0, 2, 1], [0, 1], 2) != 0    # decreasing
    assert oracle.check_csr([0, 1], [1], 1) != 0          # column out of range
    assert oracle.check_csr([0, 1], [-1], 1) != 0
    assert oracle.check_csr([0, 1, 1], [1], 2) == 0


def _segment_softmax_reference(rp, ci, Q, K, V, scale, chunk=65536):
    """Independent vectorised reference: per-edge scores, numpy reduceat for
    the row max and the row sum, gathered V rows (Eq. 1, Eq. 7)."""
    N, d = Q.shape
    O = np.zeros((N, d))
    rows = np.repeat(np.arange(N), np.diff(rp))
    starts = 0
    while starts < N:
        stop = min(N, starts + chunk)
        e0, e1 = rp[starts], rp[stop]
        r = rows[e0:e1]
        c = ci[e0:e1]
        s = scale * np.einsum("ij,ij->i", Q[r].astype(np.float64),
                              K[c].astype(np.float64))
        seg = rp[starts:stop] - e0
        nonempty = np.diff(rp[starts:stop + 1]) > 0
        seg_ne = seg[nonempty]
        m = np.maximum.reduceat(s, seg_ne)
        rid = r - starts
        mrow = np.zeros(stop - starts)
        mrow[nonempty] = m
        e = np.exp(s - mrow[rid])
        l = np.zeros(stop - starts)
        l[nonempty] = np.add.reduceat(e, seg_ne)
        p = e / l[rid]
        acc = np.zeros((stop - starts, d))
        np.add.at(acc, rid, p[:, None] * V[c].astype(np.float64))
        O[starts:stop] = acc
        starts = stop
    return O


@pytest.mark.parametrize("k", [1, 4, 2])
def test_matches_segment_softmax_on_workloads(oracle, k):
    c = W.make_config(k)
    O = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                             c["scale"])
    ref = _segment_softmax_reference(c["row_ptr"], c["col_idx"], c["Q"], c["K"],
                                     c["V"], c["scale"])
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-10)


def test_row_sample_matches_full_operator(oracle):
    c = W.make_config(1)
    full = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"],
                                c["V"], c["scale"])
    part = oracle.attention_rows_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"],
                                     c["V"], c["scale"], 100, 357)
    assert np.array_equal(part, full[100:357])
