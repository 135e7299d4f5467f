"""Plans whose row windows follow the graphs of a batch (f3s_plan_segments),
the component-aware layout that Section 4.2 leaves to future work.

The windows, the Binary Sparse Block arrays over them (Section 3.1) and the
work list (Section 3.2) are integers and must equal the oracle's bit for bit.
The forward over such a plan must meet the fp64 oracle at the bar of Table 5's
precision scheme (max-abs 5e-3, relative Frobenius 1e-3; bfloat16 inputs
1e-4): the windows only change which rows share a column list, never the
result's definition.
"""
import math

import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
MAX_ABS = 5e-3
REL_FRO = 1e-3


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _check(got, ref, max_abs=MAX_ABS, rel_fro=REL_FRO):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), "non-finite output"
    diff = got - ref
    ma = float(np.abs(diff).max()) if diff.size else 0.0
    nref = float(np.linalg.norm(ref))
    rf = float(np.linalg.norm(diff)) / nref if nref > 0 else float(np.linalg.norm(diff))
    print(f"  max_abs={ma:.3e} rel_fro={rf:.3e}", flush=True)
    assert ma <= max_abs and rf <= rel_fro, (ma, rf)


def _segment_plan(f3s, rp, ci, N, seg):
    return f3s.Plan.segments(_dev(rp), _dev(ci), N, seg)


def _check_layout(f3s, oracle, rp, ci, N, seg):
    """Plan of f3s_plan_segments against oracle.segment_windows + bsb +
    worklist, array by array."""
    print(f"segment plan N={N} nnz={int(rp[-1])} graphs={len(seg) - 1}", flush=True)
    plan = _segment_plan(f3s, rp, ci, N, seg)
    got = plan.export()
    wr = oracle.segment_windows(seg)
    ref = oracle.bsb(rp, ci, N, win_row=wr)
    info = plan.info
    assert info["n_windows"] == len(wr) - 1
    assert info["flags"] & 4
    assert np.array_equal(got["win_row"], wr)
    assert np.array_equal(got["blk_off"], ref["blk_off"])
    assert np.array_equal(got["cols"], ref["cols"])
    assert np.array_equal(got["mask"], ref["mask"])
    assert info["n_blocks"] == int(ref["blk_off"][-1])
    assert info["n_unique"] == int(ref["u"].sum())
    assert info["nnz"] == int(np.unpackbits(ref["mask"].view(np.uint8)).sum())
    items, merges = oracle.worklist(ref["nb"], ref["blk_off"], info["piece_blocks"],
                                    reorder=not (info["flags"] & 1))
    assert np.array_equal(got["items"], items)
    assert np.array_equal(got["merges"], merges)
    return plan


def _random_segments(rng, N, long_frac=0.3):
    """Graph sizes from 0 (empty graphs) to ~60 rows summing to N."""
    sizes = []
    while sum(sizes) < N:
        if rng.random() < 0.15:
            sizes.append(0)
        elif rng.random() < long_frac:
            sizes.append(int(rng.integers(17, 60)))
        else:
            sizes.append(int(rng.integers(1, 17)))
    sizes[-1] -= sum(sizes) - N
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)


def test_molecule_batch_layout(gpu, oracle):
    c = W.make_config(4, with_features=False)
    plan = _check_layout(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"], c["seg_ptr"])
    print(f"  {plan.info}", flush=True)
    fixed = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    # more, shorter windows, and fewer distinct columns per window in sum
    assert plan.info["n_windows"] > fixed.info["n_windows"]
    assert plan.info["n_unique"] < fixed.info["n_unique"]
    assert plan.info["max_blocks"] <= 3


@pytest.mark.parametrize("seed", range(8))
def test_random_patterns_layout(gpu, oracle, seed):
    rng = np.random.default_rng(2000 + seed)
    N = int(rng.integers(1, 400))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 60), empty_frac=0.2, dup_frac=0.3)
    _check_layout(gpu, oracle, rp, ci, N, _random_segments(rng, N))


def _size_class_pattern(rng, N=30000):
    """Graphs of 5, 12 and 13 rows (none fits beside its neighbour, so each is
    one window) holding 750, 3,600 and 11,700 entries: the one-wave (16 keys
    per lane), LDS-sort and column-bitmap paths of the plan build, at window
    row counts other than 16; then graphs of 20 and of 1 to 40 rows with 3
    entries per row."""
    deg = np.full(N, 3)
    deg[0:5], deg[5:17], deg[17:30] = 150, 300, 900
    rows = [rng.choice(N, size=int(k), replace=False) for k in deg]
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum(deg)
    ci = np.concatenate(rows).astype(np.int32)
    sizes = [5, 12, 13, 20]
    while sum(sizes) < N:
        sizes.append(int(rng.integers(1, 41)))
    sizes[-1] -= sum(sizes) - N
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    return rp, ci, seg


def test_window_size_classes_layout(gpu, oracle):
    rng = np.random.default_rng(31)
    rp, ci, seg = _size_class_pattern(rng)
    plan = _check_layout(gpu, oracle, rp, ci, len(rp) - 1, seg)
    assert plan.window_rows()[:5].tolist() == [0, 5, 17, 30, 46]
    assert plan.info["max_blocks"] > 600


@pytest.mark.parametrize("waves", ["1", "2", "4"])
def test_window_size_classes_forward_with_split_windows(gpu, oracle, waves, monkeypatch):
    """The heavy windows of odd row counts split into pieces (merge launch)
    and shared by one, two or four waves."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "16")
    rng = np.random.default_rng(32)
    rp, ci, seg = _size_class_pattern(rng, N=6000)
    N, d = len(rp) - 1, 64
    plan = _check_layout(gpu, oracle, rp, ci, N, seg)
    assert plan.info["n_split"] >= 3
    Q, K, V = (rng.standard_normal((N, d)).astype(np.float16) for _ in range(3))
    O = gpu.run(plan, _dev(Q), _dev(K), _dev(V), scale=0.125)
    torch.cuda.synchronize()
    _check(O.cpu().numpy(), oracle.attention_f64(rp, ci, Q, K, V, 0.125))


@pytest.mark.parametrize("d", [32, 128, 256])
@pytest.mark.parametrize("seed", range(3))
def test_random_patterns_forward(gpu, oracle, d, seed):
    rng = np.random.default_rng(2100 + 10 * seed + d)
    N = int(rng.integers(1, 600))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 70), empty_frac=0.1, dup_frac=0.2)
    seg = _random_segments(rng, N)
    plan = _segment_plan(gpu, rp, ci, N, seg)
    Q, K, V = (rng.standard_normal((N, d)).astype(np.float16) for _ in range(3))
    guard = torch.full((N + 8, d), float("nan"), dtype=torch.float32, device=DEV)
    O = gpu.run(plan, _dev(Q), _dev(K), _dev(V), scale=1 / math.sqrt(d), out=guard[:N])
    torch.cuda.synchronize()
    assert bool(torch.isnan(guard[N:]).all())          # nothing past the last row
    _check(O.cpu().numpy(), oracle.attention_f64(rp, ci, Q, K, V, 1 / math.sqrt(d)))


def test_molecule_batch_forward(gpu, oracle):
    c = W.make_config(4)
    plan = _segment_plan(gpu, c["row_ptr"], c["col_idx"], c["N"], c["seg_ptr"])
    O, lse = gpu.forward(plan, _dev(c["Q"]), _dev(c["K"]), _dev(c["V"]), scale=c["scale"],
                         lse=torch.empty(c["N"], dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
    ref, reflse = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                       c["scale"], want_lse=True)
    _check(O.cpu().numpy(), ref)
    assert np.abs(lse.cpu().numpy() - reflse).max() < 1e-3


def test_molecule_batch_forward_split_row(gpu, oracle, monkeypatch):
    """The split-row ablation instance (F3S_SPLIT_ROW=1) over windows aligned
    to the graphs: it reads each window's rows from the plan like the
    default kernel, and meets the oracle on every row."""
    monkeypatch.setenv("F3S_SPLIT_ROW", "1")
    c = W.make_config(4)
    plan = _segment_plan(gpu, c["row_ptr"], c["col_idx"], c["N"], c["seg_ptr"])
    assert plan.info["flags"] & 12 == 12
    O, lse = gpu.forward(plan, _dev(c["Q"]), _dev(c["K"]), _dev(c["V"]), scale=c["scale"])
    torch.cuda.synchronize()
    ref, reflse = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                       c["scale"], want_lse=True)
    _check(O.cpu().numpy(), ref)
    assert np.abs(lse.cpu().numpy() - reflse).max() < 1e-3


@pytest.mark.parametrize("order", ["item", "head"])
def test_molecule_batch_multi_head(gpu, oracle, order, monkeypatch):
    monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", "0" if order == "head" else str(1 << 40))
    c = W.make_config(4, with_features=False)
    N, H, d = c["N"], 3, 64
    rng = np.random.default_rng(41)
    Q, K, V = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(3))
    plan = _segment_plan(gpu, c["row_ptr"], c["col_idx"], N, c["seg_ptr"])
    O = gpu.run(plan, _dev(Q), _dev(K), _dev(V), scale=0.125)
    torch.cuda.synchronize()
    O = O.cpu().numpy()
    for h in range(H):
        _check(O[:, h], oracle.attention_f64(c["row_ptr"], c["col_idx"], Q[:, h], K[:, h],
                                             V[:, h], 0.125))


@pytest.mark.parametrize("dtype,out_dtype", [("bf16", torch.float32), ("fp8", torch.float16)])
def test_molecule_batch_precision_variants(gpu, oracle, dtype, out_dtype):
    c = W.make_config(4, dtype=dtype)
    plan = _segment_plan(gpu, c["row_ptr"], c["col_idx"], c["N"], c["seg_ptr"])
    if dtype == "bf16":
        q, kk, v = (_dev(c[x].view(np.int16)).view(torch.bfloat16) for x in ("Q", "K", "V"))
        ref = oracle.attention_bf16_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                        c["scale"])
        rel = 1e-4
    else:
        q, kk, v = (_dev(c[x]).view(torch.float8_e4m3fn) for x in ("Q", "K", "V"))
        ref = oracle.attention_e4m3_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                        c["scale"])
        rel = REL_FRO
    O, _ = gpu.forward_typed(plan, q, kk, v, out_dtype=out_dtype, scale=c["scale"])
    torch.cuda.synchronize()
    _check(O.float().cpu().numpy(), ref, rel_fro=rel)


def test_probe_and_trace_on_a_segment_plan(gpu):
    """The access-pattern probe writes every row of O and nothing past it;
    the traced forward equals the forward and records every work item."""
    c = W.make_config(4)
    N, d = c["N"], c["d"]
    plan = _segment_plan(gpu, c["row_ptr"], c["col_idx"], N, c["seg_ptr"])
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    guard = torch.full((N + 16, d), float("nan"), dtype=torch.float32, device=DEV)
    gpu.probe_gather(plan, q, kk, v, guard[:N])
    torch.cuda.synchronize()
    assert bool(torch.isfinite(guard[:N]).all()) and bool(torch.isnan(guard[N:]).all())
    ref = gpu.run(plan, q, kk, v, scale=c["scale"])
    O, rec = gpu.run_trace(plan, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    assert torch.equal(O, ref)
    r = rec.cpu().numpy().view(np.uint32)
    assert np.array_equal(r[:, 6], np.arange(plan.info["n_items"]))


def test_degenerate_segmentations(gpu, oracle):
    # one graph per row, one graph for everything, empty graphs around
    rng = np.random.default_rng(5)
    N = 100
    rp, ci = W.random_csr(rng, N, max_deg=30, empty_frac=0.3, dup_frac=0.2)
    for seg in (np.arange(N + 1), np.array([0, N]), np.array([0, 0, 0, 40, 40, N, N])):
        _check_layout(gpu, oracle, rp, ci, N, seg.astype(np.int32))
    # no rows
    z = np.zeros(1, dtype=np.int32)
    plan = gpu.Plan.segments(_dev(z), torch.empty(0, dtype=torch.int32, device=DEV), 0, [0])
    assert plan.info["n_windows"] == 0
    assert plan.window_rows().tolist() == [0]


def test_segment_plan_errors(gpu):
    rp = np.array([0, 1, 2, 3], dtype=np.int32)
    ci = np.array([0, 1, 2], dtype=np.int32)
    for seg in ([1, 3], [0, 2], [0, 2, 1, 3], [0, 4]):
        with pytest.raises(gpu.F3SError) as e:
            gpu.Plan.segments(_dev(rp), _dev(ci), 3, seg)
        assert e.value.code == 1           # F3S_ERR_INVALID_VALUE
    plan = gpu.Plan.segments(_dev(rp), _dev(ci), 3, [0, 1, 3])
    assert plan.window_rows().tolist() == [0, 3]


# ---- the backward pass over a plan with graph-aligned windows ---------------
# Gradient bar as for the 16-row plans: relative Frobenius <= 1e-3 per gradient
# and max-abs <= 5e-3 * max(1, max |reference|) (P and dS rounded to fp16).

def _check_grad(name, got, ref):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{name}: non-finite"
    diff = got - ref
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(diff)) / nref if nref > 0 else float(np.linalg.norm(diff))
    ma = float(np.abs(diff).max()) if diff.size else 0.0
    bound = 5e-3 * max(1.0, float(np.abs(ref).max()) if ref.size else 1.0)
    print(f"  {name}: rel_fro={rel:.2e} max_abs={ma:.2e} (bound {bound:.2e})", flush=True)
    assert rel <= 1e-3 and ma <= bound, (name, rel, ma)


def _grad_case(f3s, oracle, rp, ci, N, seg, Q, K, V, G, scale, dtype=torch.float16):
    plan = _segment_plan(f3s, rp, ci, N, seg)
    plan_t = plan.transpose()
    # A^T's plan has 16-row windows of its own, never a copy of the aligned plan
    assert not (plan_t.info["flags"] & 4)
    assert plan_t.info["n_windows"] == (N + 15) // 16
    conv = (lambda a: _dev(a)) if dtype == torch.float16 else \
        (lambda a: _dev(a.view(np.int16)).view(torch.bfloat16))
    q, k, v, g = conv(Q), conv(K), conv(V), conv(G)
    if dtype == torch.float16:
        O, lse = f3s.forward(plan, q, k, v, scale=scale)
    else:
        O, lse = f3s.forward_typed(plan, q, k, v, scale=scale, want_lse=True)
    dQ, dK, dV = f3s.backward(plan, plan_t, q, k, v, O, g, lse, scale=scale)
    torch.cuda.synchronize()
    if dtype == torch.float16:
        ref = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, scale)
    else:
        w = oracle.widen_bf16
        ref = oracle.attention_bwd_f64(rp, ci, w(Q), w(K), w(V), w(G), scale)
    for name, got, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
        _check_grad(name, got.cpu().numpy(), r)


def test_molecule_batch_gradients(gpu, oracle):
    c = W.make_config(4)
    G = np.random.default_rng(51).standard_normal(c["Q"].shape).astype(np.float16)
    _grad_case(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"], c["seg_ptr"], c["Q"],
               c["K"], c["V"], G, c["scale"])


@pytest.mark.parametrize("waves", ["1", "2", "4"])
def test_gradients_split_windows_of_odd_row_counts(gpu, oracle, waves, monkeypatch):
    """The heavy windows of 5, 12 and 13 rows split into pieces (dQ partials
    merged per window row), shared by one, two or four waves."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "16")
    rng = np.random.default_rng(52)
    rp, ci, seg = _size_class_pattern(rng, N=3000)
    N, d = len(rp) - 1, 64
    Q, K, V, G = (rng.standard_normal((N, d)).astype(np.float16) for _ in range(4))
    _grad_case(gpu, oracle, rp, ci, N, seg, Q, K, V, G, 0.125)


@pytest.mark.parametrize("seed", range(3))
def test_gradients_random_segmentations(gpu, oracle, seed):
    rng = np.random.default_rng(2200 + seed)
    N = int(rng.integers(1, 500))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 50), empty_frac=0.1, dup_frac=0.2)
    d = (32, 128, 256)[seed]
    Q, K, V, G = (rng.standard_normal((N, d)).astype(np.float16) for _ in range(4))
    _grad_case(gpu, oracle, rp, ci, N, _random_segments(rng, N), Q, K, V, G,
               1 / math.sqrt(d))


@pytest.mark.parametrize("order", ["item", "head"])
def test_molecule_batch_gradients_two_heads(gpu, oracle, order, monkeypatch):
    """Two heads sharing the aligned plan and its plan of A^T, in both head
    orders; each head's gradients against the oracle."""
    monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", "0" if order == "head" else str(1 << 40))
    c = W.make_config(4, with_features=False)
    N, H, d = c["N"], 2, 64
    rng = np.random.default_rng(54)
    Q, K, V, G = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(4))
    plan = _segment_plan(gpu, c["row_ptr"], c["col_idx"], N, c["seg_ptr"])
    plan_t = plan.transpose()
    q, k, v, g = (_dev(x) for x in (Q, K, V, G))
    O, lse = gpu.forward(plan, q, k, v, scale=0.125)
    dQ, dK, dV = gpu.backward(plan, plan_t, q, k, v, O, g, lse, scale=0.125)
    torch.cuda.synchronize()
    for h in range(H):
        ref = oracle.attention_bwd_f64(c["row_ptr"], c["col_idx"], Q[:, h], K[:, h],
                                       V[:, h], G[:, h], 0.125)
        for name, got, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
            _check_grad(f"{name}[h{h}]", got.cpu().numpy()[:, h], r)


def test_molecule_batch_gradients_bf16(gpu, oracle):
    c = W.make_config(4, dtype="bf16")
    G = W.to_bf16_bits(np.random.default_rng(53).standard_normal(c["Q"].shape,
                                                                 dtype=np.float32))
    _grad_case(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"], c["seg_ptr"], c["Q"],
               c["K"], c["V"], G, c["scale"], dtype=torch.bfloat16)
