"""Seeded input generators: determinism and the structure each workload
promises (CPU only)."""
import hashlib

import numpy as np
import pytest

from paper_2505_08098_amd import workloads as W


def _digest(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def _check_csr(rp, ci, N):
    assert rp.dtype == np.int32 and ci.dtype == np.int32
    assert rp[0] == 0 and len(rp) == N + 1 and rp[-1] == len(ci)
    assert np.all(np.diff(rp) >= 0)
    assert ci.min() >= 0 and ci.max() < N


@pytest.mark.parametrize("k", [1, 4])
def test_deterministic(k):
    a = W.make_config(k, seed=0)
    b = W.make_config(k, seed=0)
    c = W.make_config(k, seed=1)
    da = _digest(a["row_ptr"], a["col_idx"], a["Q"], a["K"], a["V"])
    assert da == _digest(b["row_ptr"], b["col_idx"], b["Q"], b["K"], b["V"])
    assert da != _digest(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"])


def _has_self_loops(rp, ci):
    rows = np.repeat(np.arange(len(rp) - 1), np.diff(rp))
    return np.all(np.bincount(rows[rows == ci], minlength=len(rp) - 1) == 1)


def _symmetric(rp, ci):
    N = len(rp) - 1
    rows = np.repeat(np.arange(N, dtype=np.int64), np.diff(rp))
    a = np.sort(rows * N + ci)
    b = np.sort(ci.astype(np.int64) * N + rows)
    return np.array_equal(a, b)


def test_er_structure():
    c = W.make_config(1)
    rp, ci = c["row_ptr"], c["col_idx"]
    _check_csr(rp, ci, 1024)
    assert _has_self_loops(rp, ci) and _symmetric(rp, ci)
    assert 15.0 < np.diff(rp).mean() < 17.0
    assert c["Q"].dtype == np.float16 and c["Q"].shape == (1024, 64)
    assert abs(float(c["Q"].astype(np.float64).std()) - 1.0) < 0.02


def test_chung_lu_21_structure():
    c = W.make_config(2, with_features=False)
    rp, ci = c["row_ptr"], c["col_idx"]
    _check_csr(rp, ci, 65536)
    assert _has_self_loops(rp, ci) and _symmetric(rp, ci)
    deg = np.diff(rp)
    assert 18.0 < deg.mean() < 21.5
    assert deg.max() <= 4097 and deg.max() > 1000      # heavy hub, capped
    assert deg[-16:].mean() > 20 * deg.mean()          # hubs in the last ids


def test_chung_lu_weights_hit_the_mean():
    w = W.chung_lu_weights(65536, 2.1, 20.0, 4096.0)
    assert abs(w.mean() - 20.0) < 1e-6 and w.max() <= 4096.0


def test_molecules_structure():
    c = W.make_config(4, with_features=False)
    rp, ci = c["row_ptr"], c["col_idx"]
    N = c["N"]
    _check_csr(rp, ci, N)
    assert _has_self_loops(rp, ci) and _symmetric(rp, ci)
    assert 4096 * 15 <= N <= 4096 * 45 and N % 16 != 0
    # block diagonal: every edge stays inside its component (union-find free
    # check: components are contiguous id ranges, so the sorted row's columns
    # never jump over an id that has no path back)
    rows = np.repeat(np.arange(N), np.diff(rp))
    assert np.abs(rows - ci).max() < 45


def test_sequence_window_structure():
    c = W.make_config(5, with_features=False)
    rp, ci = c["row_ptr"], c["col_idx"]
    L = c["N"]
    _check_csr(rp, ci, L)
    deg = np.diff(rp)
    assert np.all(deg[128:L - 127] == 320)
    i = 5000
    row = ci[rp[i]:rp[i + 1]]
    win = (row >= i - 128) & (row <= i + 127)
    assert win.sum() == 256 and (~win).sum() == 64


def test_random_csr_options():
    rng = np.random.default_rng(0)
    rp, ci = W.random_csr(rng, 50, 10, empty_frac=0.3, dup_frac=0.5)
    _check_csr(rp, ci, 50)
    assert (np.diff(rp) == 0).any()
