"""Fused 3S on the GPU against the fp64 oracle, element by element.

Tolerance (fixed by the operator's precision scheme, Table 5: fp16 inputs,
fp32 scores and softmax, probabilities rounded to fp16 before the value
product, fp32 output): max-abs error <= 5e-3 and relative Frobenius error
<= 1e-3, no non-finite outputs.  The dominant error is the fp16 rounding of
the probabilities (unit roundoff 2^-11), which gives a relative Frobenius
error near 3e-4 on N(0,1) inputs.
"""
import math

import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W
from _subproblem import rows_subproblem

pytestmark = pytest.mark.gpu

MAX_ABS = 5e-3
REL_FRO = 1e-3
DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    diff = got - ref
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(diff)) / nref if nref > 0 else float(np.linalg.norm(diff))
    return max_abs, rel


def _assert_parity(got, ref, max_abs=MAX_ABS, rel_fro=REL_FRO):
    assert np.all(np.isfinite(got)), "non-finite output"
    ma, rf = _errors(got, ref)
    print(f"  max_abs={ma:.3e} rel_fro={rf:.3e}", flush=True)
    assert ma <= max_abs and rf <= rel_fro, (ma, rf)
    return ma, rf


def _run(f3s, rp, ci, N, Q, K, V, scale, plan=None, out=None, stream=None):
    if plan is None:
        plan = f3s.Plan(_dev(rp), _dev(ci), N)
    O = f3s.run(plan, _dev(Q), _dev(K), _dev(V), scale=scale, out=out, stream=stream)
    torch.cuda.synchronize()
    return O.cpu().numpy(), plan


def _qkv(rng, N, d, scale=1.0):
    return tuple((scale * rng.standard_normal((N, d))).astype(np.float16) for _ in range(3))


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_workload_parity(gpu, oracle, k):
    c = W.make_config(k)
    print(f"workload {k} ({c['name']}) N={c['N']} nnz={int(c['row_ptr'][-1])} d={c['d']}",
          flush=True)
    O, plan = _run(gpu, c["row_ptr"], c["col_idx"], c["N"], c["Q"], c["K"], c["V"],
                   c["scale"])
    ref = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                               c["scale"])
    print(f"  plan {plan.info}", flush=True)
    _assert_parity(O, ref)


@pytest.mark.parametrize("waves", ["1", "2", "4"])
@pytest.mark.parametrize("d", [32, 64, 96, 128, 160, 192, 224, 256])
@pytest.mark.parametrize("N", [1, 17, 200])
def test_feature_sizes_and_ragged_windows(gpu, oracle, d, N, waves, monkeypatch):
    """Every feature size, ragged last windows, with one, two or four waves per work item
    sharing it (their partials combined in LDS)."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    rng = np.random.default_rng(d * 1000 + N)
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 70), empty_frac=0.1, dup_frac=0.2)
    Q, K, V = _qkv(rng, N, d)
    scale = 1 / math.sqrt(d)
    O, _ = _run(gpu, rp, ci, N, Q, K, V, scale)
    _assert_parity(O, oracle.attention_f64(rp, ci, Q, K, V, scale))


@pytest.mark.parametrize("d", [64, 128, 256])
def test_four_waves_per_item_with_split_windows(gpu, oracle, d, monkeypatch):
    """Four waves sharing each work item, on pieces of split windows too (a
    piece's combined partial goes to the merge launch)."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", "4")
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "6")
    rng = np.random.default_rng(d + 7)
    N = 700
    rows = [rng.choice(N, size=400, replace=False) if i < 20 else
            rng.choice(N, size=int(rng.integers(0, 40)), replace=False) for i in range(N)]
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32)
    Q, K, V = _qkv(rng, N, d)
    scale = 1 / math.sqrt(d)
    O, plan = _run(gpu, rp, ci, N, Q, K, V, scale)
    assert plan.info["n_split"] > 0
    _assert_parity(O, oracle.attention_f64(rp, ci, Q, K, V, scale))


def test_single_neighbour_rows_are_exact(gpu):
    rng = np.random.default_rng(1)
    N, d = 333, 64
    j = rng.integers(0, N, size=N).astype(np.int32)
    rp = np.arange(N + 1, dtype=np.int32)
    Q, K, V = _qkv(rng, N, d, scale=4.0)
    O, _ = _run(gpu, rp, j, N, Q, K, V, 0.3)
    assert np.array_equal(O, V[j].astype(np.float32))


def test_zero_queries_average_neighbours(gpu, oracle):
    rng = np.random.default_rng(2)
    N, d = 500, 128
    rp, ci = W.random_csr(rng, N, max_deg=90)
    _, K, V = _qkv(rng, N, d)
    Q = np.zeros((N, d), dtype=np.float16)
    O, _ = _run(gpu, rp, ci, N, Q, K, V, 0.1)
    _assert_parity(O, oracle.attention_f64(rp, ci, Q, K, V, 0.1), max_abs=1e-5, rel_fro=1e-6)


def test_constant_values_are_reproduced(gpu):
    rng = np.random.default_rng(3)
    N, d = 400, 64
    rp, ci = W.random_csr(rng, N, max_deg=50, empty_frac=0.1)
    Q, K, _ = _qkv(rng, N, d, scale=2.0)
    V = np.full((N, d), -1.75, dtype=np.float16)
    O, _ = _run(gpu, rp, ci, N, Q, K, V, 0.25)
    nonempty = np.diff(rp) > 0
    # the fp16 probabilities are summed into the normaliser, so they sum to 1
    # up to fp32 rounding
    np.testing.assert_allclose(O[nonempty], -1.75, rtol=1e-5)
    assert np.all(O[~nonempty] == 0)


@pytest.mark.parametrize("gap", [30.0, 1000.0])
def test_dominant_score_and_overflow_safety(gpu, oracle, gap):
    """One neighbour scores `gap` above the rest; gap = 1000 would overflow a
    naive softmax (e^89 is the fp32 limit)."""
    rng = np.random.default_rng(4)
    N, d = 64, 32
    rp = np.arange(0, N * N + 1, N, dtype=np.int32)   # dense rows
    ci = np.tile(np.arange(N, dtype=np.int32), N)
    Q = np.zeros((N, d), dtype=np.float16)
    K = np.zeros((N, d), dtype=np.float16)
    Q[:, 0] = 1.0
    K[np.arange(N) % 7 == 3, 0] = 1.0   # several equal winners per row
    V = rng.standard_normal((N, d)).astype(np.float16)
    O, _ = _run(gpu, rp, ci, N, Q, K, V, gap)
    _assert_parity(O, oracle.attention_f64(rp, ci, Q, K, V, gap))


def test_repeated_and_unsorted_entries(gpu, oracle):
    rng = np.random.default_rng(5)
    N, d = 300, 64
    rp, ci = W.random_csr(rng, N, max_deg=40, dup_frac=1.0, shuffle=True)
    Q, K, V = _qkv(rng, N, d)
    O, _ = _run(gpu, rp, ci, N, Q, K, V, 0.125)
    _assert_parity(O, oracle.attention_f64(rp, ci, Q, K, V, 0.125))
    # the deduplicated, sorted pattern gives the bit-identical result
    rows = [np.unique(ci[rp[i]:rp[i + 1]]) for i in range(N)]
    rp2 = np.zeros(N + 1, dtype=np.int32)
    rp2[1:] = np.cumsum([r.size for r in rows])
    O2, _ = _run(gpu, rp2, np.concatenate(rows).astype(np.int32), N, Q, K, V, 0.125)
    assert np.array_equal(O, O2)


def test_empty_rows_and_all_empty(gpu):
    rng = np.random.default_rng(6)
    N, d = 77, 64
    rp, ci = W.random_csr(rng, N, max_deg=10, empty_frac=0.6)
    Q, K, V = _qkv(rng, N, d)
    O, _ = _run(gpu, rp, ci, N, Q, K, V, 0.5)
    assert np.all(O[np.diff(rp) == 0] == 0)
    rp0 = np.zeros(N + 1, dtype=np.int32)
    O0, _ = _run(gpu, rp0, np.zeros(0, dtype=np.int32), N, Q, K, V, 0.5)
    assert np.all(O0 == 0)


def test_hub_window_above_lds_capacity(gpu, oracle):
    rng = np.random.default_rng(8)
    N, d = 30000, 64
    rows = [rng.choice(N, size=2000, replace=False) if i < 5 else
            rng.choice(N, size=4, replace=False) for i in range(N)]
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32)
    Q, K, V = _qkv(rng, N, d)
    O, plan = _run(gpu, rp, ci, N, Q, K, V, 0.125)
    assert plan.info["max_blocks"] > 256
    _assert_parity(O, oracle.attention_f64(rp, ci, Q, K, V, 0.125))


@pytest.mark.parametrize("piece", [2, 4, 16])
def test_split_windows_merge(gpu, oracle, monkeypatch, piece):
    monkeypatch.setenv("F3S_PIECE_BLOCKS", str(piece))
    c = W.make_config(2)
    O, plan = _run(gpu, c["row_ptr"], c["col_idx"], c["N"], c["Q"], c["K"], c["V"],
                   c["scale"])
    assert plan.info["n_split"] > 0
    ref = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                               c["scale"])
    _assert_parity(O, ref)


def test_relabelling_equivariance(gpu, oracle):
    c = W.make_config(4)
    N = c["N"]
    rng = np.random.default_rng(9)
    pi = rng.permutation(N)
    inv = np.argsort(pi)
    rp, ci = c["row_ptr"], c["col_idx"]
    cols = [pi[ci[rp[o]:rp[o + 1]]] for o in inv]
    rp2 = np.zeros(N + 1, dtype=np.int32)
    rp2[1:] = np.cumsum([x.size for x in cols])
    ci2 = np.concatenate(cols).astype(np.int32)
    O1, _ = _run(gpu, rp, ci, N, c["Q"], c["K"], c["V"], c["scale"])
    O2, _ = _run(gpu, rp2, ci2, N, c["Q"][inv], c["K"][inv], c["V"][inv], c["scale"])
    _assert_parity(O2, O1[inv].astype(np.float64))


def test_deterministic_and_every_row_written(gpu):
    c = W.make_config(2)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    Q, K, V = _dev(c["Q"]), _dev(c["K"]), _dev(c["V"])
    out = torch.full((c["N"], c["d"]), float("nan"), device=DEV)
    a = gpu.run(plan, Q, K, V, scale=c["scale"], out=out).clone()
    b = gpu.run(plan, Q, K, V, scale=c["scale"])
    torch.cuda.synchronize()
    assert torch.isfinite(a).all()
    assert torch.equal(a, b)


def test_non_default_stream(gpu, oracle):
    c = W.make_config(1)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    Q, K, V = _dev(c["Q"]), _dev(c["K"]), _dev(c["V"])
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        O = gpu.run(plan, Q, K, V, scale=c["scale"], stream=s)
    s.synchronize()
    ref = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                               c["scale"])
    _assert_parity(O.cpu().numpy(), ref)


def test_aliased_q_k_v(gpu, oracle):
    """AGNN form (Section 2.1): Q = K = V = H in one buffer."""
    rng = np.random.default_rng(10)
    N, d = 1000, 64
    rp, ci = W.random_csr(rng, N, max_deg=30)
    H = rng.standard_normal((N, d)).astype(np.float16)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    Hd = _dev(H)
    O = gpu.run(plan, Hd, Hd, Hd, scale=0.2)
    torch.cuda.synchronize()
    _assert_parity(O.cpu().numpy(), oracle.attention_f64(rp, ci, H, H, H, 0.2))


def test_run_argument_errors(gpu):
    c = W.make_config(1)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    Q = _dev(c["Q"])
    O = torch.empty((c["N"], c["d"]), dtype=torch.float32, device=DEV)
    s = torch.cuda.current_stream().cuda_stream
    base = Q.data_ptr()
    assert gpu.run_raw(plan, base, base, base, O.data_ptr(), 48, 0.1, s) == 3  # d
    assert gpu.run_raw(plan, base, base, base, O.data_ptr(), 288, 0.1, s) == 3
    assert gpu.run_raw(plan, base + 2, base, base, O.data_ptr(), 64, 0.1, s) == 1
    assert gpu.run_raw(plan, 0, base, base, O.data_ptr(), 64, 0.1, s) == 1
    assert gpu.run_raw(plan, base, base, base, O.data_ptr(), 64, float("inf"), s) == 1
    # O overlapping an input
    assert gpu.run_raw(plan, base, base, base, base, 64, 0.1, s) == 1
    assert gpu.load_library().f3s_last_error() == 1
    assert gpu.status_string(2) == "F3S_ERR_INVALID_CSR"


def test_binding_rejects_wrong_out_and_lse_before_launch(gpu):
    """A caller-supplied out or lse of the wrong shape, or an operand on
    another device than the plan, is refused by the binding before any
    launch (the library writes N * H * d values through the pointer)."""
    c = W.make_config(1)
    N, d = c["N"], c["d"]
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), N)
    Q = _dev(c["Q"])
    sentinel = -7.0
    for shape in ((N - 1, d), (N, d // 2), (N, 2, d)):
        out = torch.full(shape, sentinel, dtype=torch.float32, device=DEV)
        with pytest.raises(ValueError):
            gpu.forward(plan, Q, Q, Q, out=out)
        with pytest.raises(ValueError):
            gpu.run(plan, Q, Q, Q, out=out)
        with pytest.raises(ValueError):
            gpu.forward_typed(plan, Q, Q, Q, out=out)
        torch.cuda.synchronize()
        assert bool((out == sentinel).all())
    with pytest.raises(ValueError):
        gpu.forward(plan, Q, Q, Q, lse=torch.empty(N - 1, device=DEV))
    with pytest.raises(TypeError):     # a host tensor
        gpu.forward(plan, Q, Q, Q, out=torch.empty((N, d)))
    with pytest.raises(TypeError):
        gpu.forward(plan, Q, Q, Q, lse=torch.empty(N))


def _head_order(monkeypatch, order):
    """Workgroup order of several heads, forced either way: item-major (a
    K/V size threshold no input reaches) or head-major (a threshold of 0)."""
    if order == "head":
        monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", "0")
    else:
        monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", str(1 << 40))


@pytest.mark.parametrize("order", ["item", "head"])
@pytest.mark.parametrize("H,d", [(2, 64), (4, 32), (8, 64), (3, 128)])
def test_multi_head_matches_oracle_per_head(gpu, oracle, H, d, order, monkeypatch):
    """f3s_run_mh: H heads sharing one plan (Section 2.1, Eq. 4 per head)."""
    _head_order(monkeypatch, order)
    rng = np.random.default_rng(100 + H * d)
    N = 700
    rp, ci = W.random_csr(rng, N, max_deg=60, empty_frac=0.05, dup_frac=0.1)
    Q, K, V = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(3))
    scale = 1 / math.sqrt(d)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    O = gpu.run(plan, _dev(Q), _dev(K), _dev(V), scale=scale)
    torch.cuda.synchronize()
    O = O.cpu().numpy()
    for h in range(H):
        ref = oracle.attention_f64(rp, ci, Q[:, h], K[:, h], V[:, h], scale)
        _assert_parity(O[:, h], ref)


@pytest.mark.parametrize("k,H", [(2, 4), (5, 4), (3, 2), (4, 2), (4, 4), (5, 8)])
def test_multi_head_workloads(gpu, oracle, k, H):
    """Several heads over a workload graph (fresh seeded N(0,1) features of
    shape [N, H, d]); each head against the oracle, on every row for the
    smaller graphs and, for the million-node graph, on the sub-problem of
    20,000 random rows and the 8 longest rows with their full neighbour
    lists (the rows' outputs are exact there)."""
    c = W.make_config(k, with_features=False)
    rp, ci, N, d = c["row_ptr"], c["col_idx"], c["N"], c["d"]
    rng = np.random.default_rng(40 + k)
    X = [rng.standard_normal((N, H, d), dtype=np.float32).astype(np.float16)
         for _ in range(3)]
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    O = gpu.run(plan, *(_dev(x) for x in X), scale=c["scale"])
    torch.cuda.synchronize()
    print(f"workload {k}, {H} heads, N={N} d={d}", flush=True)
    if k == 3:
        rows = np.unique(np.concatenate([rng.integers(0, N, size=20000),
                                         np.argsort(np.diff(rp), kind="stable")[-8:]]))
        mrp, mci, U = rows_subproblem(rp, ci, rows)
        sel = torch.from_numpy(rows).to(DEV)
        got = O.index_select(0, sel).cpu().numpy()
        for h in range(H):
            ref = oracle.attention_f64(mrp, mci, *(np.ascontiguousarray(x[U, h]) for x in X),
                                       c["scale"])
            _assert_parity(got[:, h], ref[np.searchsorted(U, rows)])
    else:
        O = O.cpu().numpy()
        for h in range(H):
            ref = oracle.attention_f64(rp, ci, *(np.ascontiguousarray(x[:, h]) for x in X),
                                       c["scale"])
            _assert_parity(O[:, h], ref)


@pytest.mark.parametrize("k,d", [(3, 64), (3, 256), (2, 128), (2, 256), (4, 128), (4, 256),
                                 (5, 128), (5, 256)])
def test_workloads_at_other_feature_sizes(gpu, oracle, k, d):
    """The feature-size sweep of the measurements (the paper varies d over
    64, 128 and 256): each workload graph at the other sizes, every row, or
    for the million-node graph the sub-problem of 20,000 random rows and the
    8 longest rows."""
    c = W.make_config(k, d=d)
    rp, ci, N = c["row_ptr"], c["col_idx"], c["N"]
    print(f"workload {k} N={N} d={d}", flush=True)
    O, _ = _run(gpu, rp, ci, N, c["Q"], c["K"], c["V"], c["scale"])
    if k == 3:
        rng = np.random.default_rng(70 + d)
        rows = np.unique(np.concatenate([rng.integers(0, N, size=20000),
                                         np.argsort(np.diff(rp), kind="stable")[-8:]]))
        mrp, mci, U = rows_subproblem(rp, ci, rows)
        ref = oracle.attention_f64(mrp, mci, c["Q"][U], c["K"][U], c["V"][U], c["scale"])
        _assert_parity(O[rows], ref[np.searchsorted(U, rows)])
    else:
        _assert_parity(O, oracle.attention_f64(rp, ci, c["Q"], c["K"], c["V"], c["scale"]))


@pytest.mark.parametrize("k,H", [(5, 1), (2, 3), (4, 1), (4, 2), (2, 4), (5, 8), (4, 3),
                                 (5, 6), (1, 16)])
def test_xcd_ranges_order_gives_identical_results(gpu, k, H, monkeypatch):
    """Each XCD taking a consecutive range of the work list (with 2, 4 or 8
    heads, of one head's list) only reorders independent work items: O and
    lse are bit-identical to the round-robin order, with split windows (a
    merge launch follows) and several heads in both head orders (window-major
    with 3 heads keeps round-robin order; head by head takes ranges of each
    head's list with any head count)."""
    c = W.make_config(k, with_features=False)
    N, d = c["N"], W.WORKLOADS[k]["d"]
    rng = np.random.default_rng(60 + k)
    shape = (N, H, d) if H > 1 else (N, d)
    q, kk, v = (_dev(rng.standard_normal(shape).astype(np.float16)) for _ in range(3))
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), N)
    for head_major in ("0", "1000000000000"):
        monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", head_major)
        outs = []
        for chunks in ("0", "1"):
            monkeypatch.setenv("F3S_XCD_CHUNKS", chunks)
            outs.append(gpu.forward(plan, q, kk, v, scale=0.125))
        torch.cuda.synchronize()
        assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_dram_scale_graph_sampled(gpu, oracle):
    """The graph bench.py runs to measure the bandwidth the kernel sustains
    from DRAM (8,388,608 nodes, self + 16 uniform random neighbours, d = 128,
    N(0,1) fp16 features drawn on the device): the whole call on the GPU,
    4,000 random rows and the last window against the oracle on their
    sub-problem."""
    rp, ci = W.uniform_random_graph(0)
    N, d = len(rp) - 1, 128
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(0)
    Q, K, V = (torch.randn((N, d), generator=gen, device=DEV).half() for _ in range(3))
    O = gpu.run(plan, Q, K, V, scale=1 / math.sqrt(d))
    torch.cuda.synchronize()
    rng = np.random.default_rng(8)
    rows = np.unique(np.concatenate([rng.integers(0, N, size=4000),
                                     np.arange(N - 16, N)]))
    mrp, mci, U = rows_subproblem(rp, ci, rows)
    idx = torch.from_numpy(U).to(DEV)
    q, k, v = (x.index_select(0, idx).cpu().numpy() for x in (Q, K, V))
    ref = oracle.attention_f64(mrp, mci, q, k, v, 1 / math.sqrt(d))
    got = O.index_select(0, torch.from_numpy(rows).to(DEV)).cpu().numpy()
    print(f"  {rows.size} rows, sub-problem of {U.size} nodes", flush=True)
    _assert_parity(got, ref[np.searchsorted(U, rows)])
    plan.close()
    del Q, K, V, O
    torch.cuda.empty_cache()


@pytest.mark.parametrize("waves", ["1", "2", "4"])
@pytest.mark.parametrize("order", ["item", "head"])
@pytest.mark.parametrize("piece", [4, 1000000])
def test_multi_head_equals_single_head_runs(gpu, monkeypatch, piece, order, waves):
    """Head h of the multi-head call is bit-identical to a single-head call on
    the head's slice, with and without split windows (H * d > 256 also
    exercises the head groups that bound the partial-result scratch), in
    either workgroup order, with one, two or four waves per work item (fixed for
    both calls: the combination of the waves' partials rounds differently)."""
    _head_order(monkeypatch, order)
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    monkeypatch.setenv("F3S_PIECE_BLOCKS", str(piece))
    c = W.make_config(2, with_features=False)
    N, H, d = c["N"], 6, 64
    rng = np.random.default_rng(5)
    Q, K, V = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(3))
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), N)
    if piece == 4:
        assert plan.info["n_split"] > 0
    O = gpu.run(plan, _dev(Q), _dev(K), _dev(V), scale=0.125)
    for h in (0, 3, 5):
        Oh = gpu.run(plan, _dev(np.ascontiguousarray(Q[:, h])), _dev(np.ascontiguousarray(K[:, h])),
                     _dev(np.ascontiguousarray(V[:, h])), scale=0.125)
        torch.cuda.synchronize()
        assert torch.equal(O[:, h], Oh)


def test_multi_head_argument_errors(gpu):
    c = W.make_config(1)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    Q = torch.zeros((c["N"], 2, 64), dtype=torch.float16, device=DEV)
    O = torch.empty((c["N"], 2, 64), dtype=torch.float32, device=DEV)
    L = gpu.load_library()
    s = ctypes_stream()
    assert L.f3s_run_mh(plan.handle, Q.data_ptr(), Q.data_ptr(), Q.data_ptr(), O.data_ptr(),
                        0, 64, 0.1, s) == 1
    assert L.f3s_run_mh(plan.handle, Q.data_ptr(), Q.data_ptr(), Q.data_ptr(), O.data_ptr(),
                        2, 40, 0.1, s) == 3
    assert L.f3s_run_mh(plan.handle, Q.data_ptr(), Q.data_ptr(), Q.data_ptr(), O.data_ptr(),
                        2, 64, 0.1, s) == 0
    torch.cuda.synchronize()


def ctypes_stream():
    import ctypes
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("d", [32, 64, 96, 128, 160, 192, 224, 256])
@pytest.mark.parametrize("many", [False, True])
def test_split_windows_merge_all_feature_sizes(gpu, oracle, monkeypatch, d, many):
    """Pieces of 2 blocks: every window above 2 blocks is split and merged
    (the merge kernel's column coverage differs for d = 32, 96, 160, 224);
    two heads share each launch where 2 * d <= 256.  `many`: windows of up to
    ~60 blocks, so some have more than 16 pieces (several rounds of the merge's
    loads)."""
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "2")
    rng = np.random.default_rng(500 + d + (7 if many else 0))
    N, H = (1003, 2) if many else (300, 2)
    rp, ci = W.random_csr(rng, N, max_deg=300 if many else 80, empty_frac=0.05,
                          dup_frac=0.1)
    Q, K, V = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(3))
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    assert plan.info["n_split"] > 0
    max_pieces = -(-plan.info["max_blocks"] // plan.info["piece_blocks"])
    assert (max_pieces > 16) == many
    O, lse = gpu.forward(plan, _dev(Q), _dev(K), _dev(V), scale=1 / math.sqrt(d))
    torch.cuda.synchronize()
    O, lse = O.cpu().numpy(), lse.cpu().numpy()
    for h in range(H):
        ref, reflse = oracle.attention_f64(rp, ci, np.ascontiguousarray(Q[:, h]),
                                           np.ascontiguousarray(K[:, h]),
                                           np.ascontiguousarray(V[:, h]), 1 / math.sqrt(d),
                                           want_lse=True)
        _assert_parity(O[:, h], ref)
        fin = np.isfinite(reflse)
        assert np.array_equal(np.isfinite(lse[:, h]), fin)
        assert np.abs(lse[fin, h] - reflse[fin]).max() < 2e-3


@pytest.mark.parametrize("k", [1, 2, 4, 5, 3])
def test_narrow_gather_ablation_is_bit_identical(gpu, oracle, monkeypatch, k):
    """F3S_NARROW_GATHER=1 only changes how K and V rows reach LDS (4-byte
    words instead of 16-byte chunks): same tiles, same arithmetic, so the
    output is bit-identical (the ablation runs one wave per work item, so the
    reference does too), and it meets the oracle on every row; other type
    pairs are refused."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", "1")
    c = W.make_config(k)
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    ref, ref_lse = gpu.forward(plan, q, kk, v, scale=c["scale"])
    monkeypatch.setenv("F3S_NARROW_GATHER", "1")
    narrow = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    assert narrow.info["flags"] & 2
    got, got_lse = gpu.forward(narrow, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    assert torch.equal(got, ref) and torch.equal(got_lse, ref_lse)
    _assert_parity(got.cpu().numpy(), oracle.attention_f64(
        c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"], c["scale"]))
    with pytest.raises(gpu.F3SError) as e:
        gpu.forward_typed(narrow, q, kk, v, out_dtype=torch.float16)
    assert e.value.code == 3


@pytest.mark.parametrize("k", [1, 2, 4, 5, 3])
def test_split_row_ablation_matches_oracle(gpu, oracle, monkeypatch, k):
    """F3S_SPLIT_ROW=1 (the paper's split-row partition): the waves of a work
    item split the feature dimension -- partial scores summed through LDS
    once per block pair, each wave's own output columns -- instead of the
    block pairs.  Same plan arrays; only the order of the score's partial
    sums differs from the default kernel, so it meets the oracle on every
    row; other type pairs are refused."""
    c = W.make_config(k)
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    ref_gpu, _ = gpu.forward(plan, q, kk, v, scale=c["scale"])
    monkeypatch.setenv("F3S_SPLIT_ROW", "1")
    sr = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    assert sr.info["flags"] & 8
    for key in ("n_blocks", "n_items", "n_split"):
        assert sr.info[key] == plan.info[key]
    got, got_lse = gpu.forward(sr, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    ref, ref_lse = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                        c["scale"], want_lse=True)
    _assert_parity(got.cpu().numpy(), ref)
    got_lse = got_lse.cpu().numpy()
    fin = np.isfinite(ref_lse)
    assert np.array_equal(np.isfinite(got_lse), fin)
    assert np.abs(got_lse[fin] - ref_lse[fin]).max() < 2e-3
    # a different rounding of a score can move a probability's fp16 rounding
    # by one unit, so the two kernels agree to the parity bound, not bit for bit
    assert float((got - ref_gpu).abs().max()) <= MAX_ABS
    with pytest.raises(gpu.F3SError) as e:
        gpu.forward_typed(sr, q, kk, v, out_dtype=torch.float16)
    assert e.value.code == 3


@pytest.mark.parametrize("d,H", [(64, 3), (128, 2), (192, 1), (256, 1)])
def test_split_row_ablation_heads_split_windows_ragged(gpu, oracle, monkeypatch, d, H):
    """The split-row instance at every feature size it takes (2 waves at
    d = 64 and 192, 4 at 128 and 256), with several heads, split windows
    (merge launch) and a ragged last window, against the oracle per head."""
    rng = np.random.default_rng(300 + d + H)
    N = 1003
    rp, ci = W.random_csr(rng, N, max_deg=300, empty_frac=0.05, dup_frac=0.1)
    Q, K, V = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(3))
    monkeypatch.setenv("F3S_SPLIT_ROW", "1")
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    assert plan.info["flags"] & 8 and plan.info["n_split"] > 0
    O, lse = gpu.forward(plan, _dev(Q), _dev(K), _dev(V), scale=1 / math.sqrt(d))
    torch.cuda.synchronize()
    O, lse = O.cpu().numpy(), lse.cpu().numpy()
    for h in range(H):
        ref, reflse = oracle.attention_f64(rp, ci, np.ascontiguousarray(Q[:, h]),
                                           np.ascontiguousarray(K[:, h]),
                                           np.ascontiguousarray(V[:, h]), 1 / math.sqrt(d),
                                           want_lse=True)
        _assert_parity(O[:, h], ref)
        fin = np.isfinite(reflse)
        assert np.array_equal(np.isfinite(lse[:, h]), fin)
        assert np.abs(lse[fin, h] - reflse[fin]).max() < 2e-3


def test_split_row_ablation_refuses_other_shapes(gpu, monkeypatch):
    """d not a multiple of 64, or the narrow-gather ablation as well: refused
    before any launch (F3S_ERR_UNSUPPORTED)."""
    rng = np.random.default_rng(5)
    N = 64
    rp, ci = W.random_csr(rng, N, max_deg=8)
    monkeypatch.setenv("F3S_SPLIT_ROW", "1")
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    for d in (32, 96, 160, 224):
        q = _dev(rng.standard_normal((N, d)).astype(np.float16))
        with pytest.raises(gpu.F3SError) as e:
            gpu.forward(plan, q, q, q)
        assert e.value.code == 3
    monkeypatch.setenv("F3S_NARROW_GATHER", "1")
    both = gpu.Plan(_dev(rp), _dev(ci), N)
    assert both.info["flags"] & 10 == 10
    q = _dev(rng.standard_normal((N, 64)).astype(np.float16))
    with pytest.raises(gpu.F3SError) as e:
        gpu.forward(both, q, q, q)
    assert e.value.code == 3


def _sample_rows_reference(oracle, rp, ci, S, Q, K, V, scale):
    """Oracle rows S of a large problem: the rows S and their neighbours are
    copied into a small problem (neighbour-only rows empty) and the oracle
    runs on that; rows of S come back in order."""
    rp = rp.cpu().numpy().astype(np.int64)
    nb = {int(i): ci[int(rp[i]):int(rp[i + 1])].cpu().numpy() for i in S}
    U = sorted(set(int(i) for i in S) | set(int(j) for a in nb.values() for j in a))
    loc = {u: k for k, u in enumerate(U)}
    rows = [[loc[int(j)] for j in nb[u]] if u in nb else [] for u in U]
    mrp = np.zeros(len(U) + 1, dtype=np.int32)
    mrp[1:] = np.cumsum([len(r) for r in rows])
    mci = np.array([c for r in rows for c in r], dtype=np.int32)
    idx = torch.tensor(U, device=DEV)
    q, k, v = (x.index_select(0, idx).cpu().numpy() for x in (Q, K, V))
    ref = oracle.attention_f64(mrp, mci, q, k, v, scale)
    return ref[[loc[int(i)] for i in S]]


def test_wide_addressing_above_4gib(gpu, oracle):
    """Q, K, V of more than 4 GiB each (N = 9,000,000 rows, d = 256: gathers
    switch to 64-bit addresses): sampled rows, including the last ones and
    rows whose neighbours sit at the top of the arrays, against the oracle."""
    N, d = 9_000_000, 256
    assert N * d * 2 > 2 ** 32
    i = torch.arange(N, dtype=torch.int64, device=DEV)
    cols = torch.stack([i, (i * 7919 + 13) % N, N - 1 - i], dim=1)
    ci = cols.reshape(-1).to(torch.int32)
    rp = (torch.arange(N + 1, dtype=torch.int64, device=DEV) * 3).to(torch.int32)
    g = torch.Generator(device=DEV)
    g.manual_seed(7)
    Q, K, V = (torch.randn((N, d), generator=g, device=DEV, dtype=torch.float32).half()
               for _ in range(3))
    plan = gpu.Plan(rp, ci, N)
    O = gpu.run(plan, Q, K, V, scale=1 / 16)
    torch.cuda.synchronize()
    rng = np.random.default_rng(8)
    S = np.unique(np.concatenate([[0, 1, N // 2, N - 2, N - 1],
                                  rng.integers(0, N, size=120),
                                  N - 1 - rng.integers(0, 1000, size=40)]))
    ref = _sample_rows_reference(oracle, rp, ci, S, Q, K, V, 1 / 16)
    got = O.index_select(0, torch.tensor(S, device=DEV)).cpu().numpy()
    print(f"  {len(S)} sampled rows", flush=True)
    _assert_parity(got, ref)
    plan.close()
    del Q, K, V, O
    torch.cuda.empty_cache()
