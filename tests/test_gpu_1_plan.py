"""GPU plan (CSR -> BSB layout + work list) against the oracle, bit for bit.

Section 3.1 (layout) and Section 3.2 (reordered work list) define integer
results; the plan built by the HIP kernels must equal the oracle's exactly.
"""
import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu


def _plan(f3s, rp, ci, N):
    dev = torch.device("cuda:0")
    return f3s.Plan(torch.from_numpy(np.ascontiguousarray(rp)).to(dev),
                    torch.from_numpy(np.ascontiguousarray(ci)).to(dev), N)


def _check_plan_against_oracle(f3s, oracle, rp, ci, N):
    print(f"plan check N={N} nnz={int(rp[-1])}", flush=True)
    plan = _plan(f3s, rp, ci, N)
    got = plan.export()
    ref = oracle.bsb(rp, ci, N)
    info = plan.info
    assert info["n_windows"] == (N + 15) // 16
    assert np.array_equal(got["blk_off"], ref["blk_off"])
    assert np.array_equal(got["cols"], ref["cols"])
    assert np.array_equal(got["mask"], ref["mask"])
    assert info["n_blocks"] == int(ref["blk_off"][-1])
    assert info["n_unique"] == int(ref["u"].sum())
    assert info["max_blocks"] == (int(ref["nb"].max()) if len(ref["nb"]) else 0)
    # distinct (row, col) pairs = set bits of all bitmaps
    assert info["nnz"] == int(np.unpackbits(ref["mask"].view(np.uint8)).sum())
    items, merges = oracle.worklist(ref["nb"], ref["blk_off"], info["piece_blocks"],
                                    reorder=not (info["flags"] & 1))
    assert np.array_equal(got["items"], items)
    assert np.array_equal(got["merges"], merges)
    assert info["n_items"] == len(items) and info["n_split"] == len(merges)
    assert info["n_pieces"] == int((items[:, 3] >= 0).sum())
    assert info["bsb_bytes"] == 4 * (info["n_windows"] + 1) + 64 * info["n_blocks"] \
        + 32 * info["n_blocks"]
    plan.close()
    return info


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_plan_matches_oracle_on_workloads(gpu, oracle, k):
    c = W.make_config(k, with_features=False)
    info = _check_plan_against_oracle(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"])
    print(k, info, flush=True)


@pytest.mark.parametrize("seed", range(8))
def test_plan_matches_oracle_on_random_patterns(gpu, oracle, seed):
    rng = np.random.default_rng(1000 + seed)
    N = int(rng.integers(1, 300))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 60), empty_frac=0.2, dup_frac=0.3)
    _check_plan_against_oracle(gpu, oracle, rp, ci, N)


@pytest.mark.parametrize("N,per_row,min_blocks", [(40000, 600, 256), (200000, 2000, 1408)])
def test_plan_heavy_window_above_lds_capacity(gpu, oracle, N, per_row, min_blocks):
    """A window with more entries than the LDS sort holds takes the column-
    bitmap path; its block bitmaps are built in LDS up to the workgroup's
    budget (1408 blocks with two column chunks at N = 200,000) and with
    atomics on the staging area beyond it."""
    rng = np.random.default_rng(7)
    rows = [rng.choice(N, size=per_row, replace=True) if i < 16 else
            rng.choice(N, size=3, replace=False) for i in range(N)]
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32)
    info = _check_plan_against_oracle(gpu, oracle, rp, ci, N)
    assert info["max_blocks"] > min_blocks


def test_plan_more_windows_than_one_scan_tile(gpu, oracle):
    """81,250 windows, more than one scan workgroup covers (65,536), so the
    scans over windows take the tiled path (tiles, their totals, the add)."""
    rng = np.random.default_rng(5)
    N = 1_300_000
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum(rng.integers(0, 4, size=N))
    ci = rng.integers(0, N, size=int(rp[-1])).astype(np.int32)
    info = _check_plan_against_oracle(gpu, oracle, rp, ci, N)
    assert info["n_windows"] > 65536


def test_plan_more_windows_than_two_scan_passes(gpu, oracle):
    """4.2 M windows, more than a two-pass scan covers (1024 tiles of 4096
    elements = 4,194,304), so the scans over windows scan their tile totals
    separately (three launches)."""
    rng = np.random.default_rng(6)
    N = 67_200_000
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum(rng.integers(0, 2, size=N, dtype=np.int32))
    ci = rng.integers(0, N, size=int(rp[-1]), dtype=np.int32)
    info = _check_plan_against_oracle(gpu, oracle, rp, ci, N)
    assert info["n_windows"] > 4_194_304


def _windows_of_sizes(rng, sizes, N, dup_frac=0.3):
    """CSR whose window w holds sizes[w] entries spread over its 16 rows, with
    duplicates and unsorted columns; the remaining rows are empty."""
    rows = [[] for _ in range(N)]
    for w, n in enumerate(sizes):
        pool = rng.choice(N, size=max(1, int(n * (1 - dup_frac))), replace=False)
        cols = rng.choice(pool, size=n, replace=True)
        which = rng.integers(0, 16, size=n)
        for r in range(16):
            rows[16 * w + r] = cols[which == r].tolist()
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.array([c for r in rows for c in r], dtype=np.int32)
    return rp, ci


@pytest.mark.parametrize("N", [9000, 140000])
def test_plan_window_size_classes(gpu, oracle, N):
    """Every sorting path of the plan: one wavefront with 1, 2, 4, 8 or 16 keys
    per lane (up to 64, 128, 256, 512, 1024 entries), the workgroup LDS sort
    (up to 4096) and the column-bitmap path above it (one chunk of 2^17
    columns, or several), each at its edges."""
    rng = np.random.default_rng(11)
    sizes = [0, 1, 17, 64, 65, 100, 128, 129, 256, 257, 400, 512, 513, 1000,
             1024, 1025, 4096, 4097, 6000, 3, 0, 64, 9000]
    rp, ci = _windows_of_sizes(rng, sizes, N)
    _check_plan_against_oracle(gpu, oracle, rp, ci, N)


@pytest.mark.parametrize("size,N", [(100, 9000), (600, 9000), (2000, 9000), (5000, 9000),
                                    (5000, 140000)])
def test_plan_rejects_bad_column_in_each_path(gpu, size, N):
    """An out-of-range column is reported whichever path sorts its window."""
    rng = np.random.default_rng(size)
    rp, ci = _windows_of_sizes(rng, [50, size, 20], N)
    lo, hi = int(rp[16]), int(rp[32])
    for bad in (N, -1):
        c2 = ci.copy()
        c2[(lo + hi) // 2] = bad
        with pytest.raises(gpu.F3SError) as e:
            _plan(gpu, rp, c2, N)
        assert e.value.code == 2  # F3S_ERR_INVALID_CSR


def test_plan_split_windows(gpu, oracle, monkeypatch):
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")
    c = W.make_config(2, with_features=False)
    info = _check_plan_against_oracle(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"])
    assert info["piece_blocks"] == 4 and info["n_split"] > 100


def test_plan_forced_piece_above_the_estimate(gpu, oracle, monkeypatch):
    """A forced piece size larger than any window: capped at the largest
    window (nothing split), the work list is the stable sort by block count."""
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "100000")
    c = W.make_config(2, with_features=False)
    info = _check_plan_against_oracle(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"])
    assert info["n_split"] == 0
    assert info["piece_blocks"] >= info["max_blocks"]


def test_plan_empty_and_degenerate(gpu, oracle):
    # N = 0
    plan = _plan(gpu, np.zeros(1, dtype=np.int32), np.zeros(0, dtype=np.int32), 0)
    assert plan.info["n_windows"] == 0 and plan.info["n_items"] == 0
    plan.close()
    # all rows empty
    _check_plan_against_oracle(gpu, oracle, np.zeros(50, dtype=np.int32),
                               np.zeros(0, dtype=np.int32), 49)
    # single node with a self loop
    _check_plan_against_oracle(gpu, oracle, np.array([0, 1], dtype=np.int32),
                               np.array([0], dtype=np.int32), 1)


@pytest.mark.parametrize("rp,ci,N", [
    ([1, 1], [0], 1),                 # row_ptr[0] != 0
    ([0, 2, 1], [0, 1], 2),           # decreasing row_ptr
    ([0, 1, 2], [0, 2], 2),           # column == N
    ([0, 1, 2], [0, -1], 2),          # negative column
])
def test_plan_rejects_malformed_csr(gpu, rp, ci, N):
    with pytest.raises(gpu.F3SError) as e:
        _plan(gpu, np.array(rp, dtype=np.int32), np.array(ci, dtype=np.int32), N)
    assert e.value.code == 2  # F3S_ERR_INVALID_CSR


def test_plan_with_and_without_workspace(gpu):
    """f3s_plan (library-allocated scratch) and f3s_plan_ws (lent scratch, what
    Plan uses) build the same plan; a short or misaligned workspace is
    rejected."""
    import ctypes
    L = gpu.load_library()
    c = W.make_config(2, with_features=False)
    dev = torch.device("cuda:0")
    rp = torch.from_numpy(c["row_ptr"]).to(dev)
    ci = torch.from_numpy(c["col_idx"]).to(dev)
    N = c["N"]
    a = gpu.Plan(rp, ci, N).export()
    h = L.f3s_plan(rp.data_ptr(), ci.data_ptr(), N)
    assert h
    b = gpu.Plan._from_handle(h, dev, N).export()
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    need = L.f3s_plan_workspace_bytes(N, ci.numel())
    assert need > 4 * ci.numel()
    ws = torch.empty(need + 512, dtype=torch.uint8, device=dev)
    for ptr, size in ((ws.data_ptr(), need - 256), (ws.data_ptr() + 4, need),
                      (None, need)):
        assert not L.f3s_plan_ws(rp.data_ptr(), ci.data_ptr(), N, ptr, size)
        assert L.f3s_last_error() == 1  # F3S_ERR_INVALID_VALUE
    h = L.f3s_plan_ws(rp.data_ptr(), ci.data_ptr(), N, ws.data_ptr(), need)
    assert h
    b = gpu.Plan._from_handle(h, dev, N).export()
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_plan_is_deterministic(gpu):
    c = W.make_config(2, with_features=False)
    a = _plan(gpu, c["row_ptr"], c["col_idx"], c["N"]).export()
    b = _plan(gpu, c["row_ptr"], c["col_idx"], c["N"]).export()
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_work_list_order_rule(gpu, oracle, k, monkeypatch):
    """Unforced, the work list keeps window order exactly when the windows
    are nearly uniform: at least 2048 of them, the largest holding at most
    twice the mean block count (configs 4 and 5); F3S_NO_REORDER=0 sorts
    every plan.  Both lists equal the oracle's for that order."""
    c = W.make_config(k, with_features=False)
    nb = oracle.bsb(c["row_ptr"], c["col_idx"], c["N"])["nb"].astype(np.int64)
    uniform = nb.size >= 2048 and int(nb.max()) * nb.size <= 2 * int(nb.sum())
    assert uniform == (k in (4, 5))
    monkeypatch.delenv("F3S_NO_REORDER", raising=False)
    info = _check_plan_against_oracle(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"])
    assert bool(info["flags"] & 1) == uniform
    monkeypatch.setenv("F3S_NO_REORDER", "0")
    info = _check_plan_against_oracle(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"])
    assert not info["flags"] & 1


def test_plan_without_reordering(gpu, oracle, monkeypatch):
    """Ablation switch: the work list keeps window order (Section 3.2 off)."""
    monkeypatch.setenv("F3S_NO_REORDER", "1")
    c = W.make_config(2, with_features=False)
    info = _check_plan_against_oracle(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"])
    assert info["flags"] & 1
