"""Backward pass on the GPU against the fp64 oracle's gradients.

Tolerance for gradients (fp16 inputs; P and dS rounded to fp16 before the
products, unit roundoff 2^-11; P recomputed from an lse whose normaliser
summed fp16-rounded probabilities): relative Frobenius error <= 1e-3 per
gradient and max-abs error <= 5e-3 * max(1, max |reference|).  Measured:
rel-Fro ~2e-4 (the fp16 rounding of P and dS, 2^-11 relative, averaged).
bf16 inputs (the oracle gets the same bf16 values, widened exactly): P and
dS enter the products as two bf16 terms (~16 bits), so the same bar holds
with room to spare.
"""
import math

import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W
from _subproblem import rows_attending, rows_subproblem, sample_keys

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
REL_FRO = 1e-3
MAX_ABS_REL = 5e-3


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _check(name, got, ref):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{name}: non-finite"
    diff = got - ref
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(diff)) / nref if nref > 0 else float(np.linalg.norm(diff))
    ma = float(np.abs(diff).max()) if diff.size else 0.0
    bound = MAX_ABS_REL * max(1.0, float(np.abs(ref).max()) if ref.size else 1.0)
    print(f"  {name}: rel_fro={rel:.2e} max_abs={ma:.2e} (bound {bound:.2e})", flush=True)
    assert rel <= REL_FRO and ma <= bound, (name, rel, ma)


def _transpose_csr(rp, ci, N):
    rows = np.repeat(np.arange(N, dtype=np.int64), np.diff(rp))
    key = np.unique(ci.astype(np.int64) * N + rows)   # (col, row), deduplicated
    r2 = (key // N).astype(np.int64)
    c2 = (key % N).astype(np.int32)
    rp2 = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(np.bincount(r2, minlength=N), out=rp2[1:])
    return rp2.astype(np.int32), c2


def _grad_case(f3s, oracle, rp, ci, N, Q, K, V, G, scale):
    plan = f3s.Plan(_dev(rp), _dev(ci), N)
    plan_t = plan.transpose()
    q, k, v, g = _dev(Q), _dev(K), _dev(V), _dev(G)
    O, lse = f3s.forward(plan, q, k, v, scale=scale)
    dQ, dK, dV = f3s.backward(plan, plan_t, q, k, v, O, g, lse, scale=scale)
    torch.cuda.synchronize()
    H = Q.shape[1] if Q.ndim == 3 else 1
    for h in range(H):
        sl = (slice(None), h) if Q.ndim == 3 else (slice(None),)
        ref = oracle.attention_bwd_f64(rp, ci, Q[sl], K[sl], V[sl], G[sl], scale)
        for name, got, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
            _check(f"{name}[h{h}]", got.cpu().numpy()[sl], r)
    return plan, plan_t


def test_forward_lse_matches_oracle(gpu, oracle, monkeypatch):
    for piece in ("4", "1000000"):
        monkeypatch.setenv("F3S_PIECE_BLOCKS", piece)
        c = W.make_config(2)
        plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
        O, lse = gpu.forward(plan, _dev(c["Q"]), _dev(c["K"]), _dev(c["V"]), scale=c["scale"])
        torch.cuda.synchronize()
        refO, reflse = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                            c["scale"], want_lse=True)
        assert np.abs(lse.cpu().numpy() - reflse).max() < 2e-3
        assert np.abs(O.cpu().numpy() - refO).max() < 5e-3


def test_empty_rows_have_minus_inf_lse(gpu):
    rng = np.random.default_rng(1)
    N = 50
    rp, ci = W.random_csr(rng, N, max_deg=5, empty_frac=0.5)
    Q = _dev(rng.standard_normal((N, 32)).astype(np.float16))
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    _, lse = gpu.forward(plan, Q, Q, Q, scale=0.2)
    lse = lse.cpu().numpy()
    empty = np.diff(rp) == 0
    assert np.all(np.isneginf(lse[empty])) and np.all(np.isfinite(lse[~empty]))


@pytest.mark.parametrize("k", [1, 2, 4, 5, 3])
def test_transposed_plan_is_the_plan_of_the_transpose(gpu, oracle, k):
    """Small symmetric patterns are checked on the plan, large ones (configs 5
    and 3, above 8 M entries) on the sorted CSR of A^T; 5 is directed."""
    c = W.make_config(k, with_features=False)
    N = c["N"]
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), N)
    got = plan.transpose().export()
    rp2, ci2 = _transpose_csr(c["row_ptr"], c["col_idx"], N)
    ref = gpu.Plan(_dev(rp2), _dev(ci2), N).export()
    for key in ref:
        assert np.array_equal(got[key], ref[key]), key
    b = oracle.bsb(rp2, ci2, N)
    assert np.array_equal(got["cols"], b["cols"]) and np.array_equal(got["mask"], b["mask"])


# the symmetry check on the plan alone, or on the sorted rows of A^T (the
# default from 8 M entries on; forced here for small patterns)
SYMMETRY_PATHS = ["plan", "sorted"]


def _symmetry_path(monkeypatch, path):
    if path == "sorted":
        monkeypatch.setenv("F3S_SYMMETRY_SORT_FIRST", "0")
    else:
        monkeypatch.delenv("F3S_SYMMETRY_SORT_FIRST", raising=False)


@pytest.mark.parametrize("path", SYMMETRY_PATHS)
@pytest.mark.parametrize("seed", range(4))
def test_transposed_plan_of_asymmetric_patterns(gpu, oracle, seed, path, monkeypatch):
    """Random directed patterns with duplicates and empty rows: the plan of A^T
    built from a plan of A equals the oracle's layout of A^T."""
    _symmetry_path(monkeypatch, path)
    rng = np.random.default_rng(500 + seed)
    N = int(rng.integers(1, 400))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 70), empty_frac=0.2, dup_frac=0.3)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    got = plan.transpose().export()
    rp2, ci2 = _transpose_csr(rp, ci, N)
    b = oracle.bsb(rp2, ci2, N)
    for key in ("blk_off", "cols", "mask"):
        assert np.array_equal(got[key], b[key]), key


@pytest.mark.parametrize("N", [200, 3000, 70000, 17_000_000])
def test_transposed_plan_for_each_sort_depth(gpu, oracle, N):
    """Directed patterns whose node ids need one, two, three and four 8-bit
    digit passes of the column sort (the last pass writes A^T's columns in
    place, from either buffer pair)."""
    rng = np.random.default_rng(N)
    if N <= 100000:
        rp, ci = W.random_csr(rng, N, max_deg=min(N, 24), empty_frac=0.1, dup_frac=0.2)
    else:  # sparse: 0-2 entries per row, repeats possible
        rp = np.zeros(N + 1, dtype=np.int32)
        rp[1:] = np.cumsum(rng.integers(0, 3, size=N, dtype=np.int32))
        ci = rng.integers(0, N, size=int(rp[-1]), dtype=np.int32)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    got = plan.transpose().export()
    rp2, ci2 = _transpose_csr(rp, ci, N)
    b = oracle.bsb(rp2, ci2, N)
    for key in ("blk_off", "cols", "mask"):
        assert np.array_equal(got[key], b[key]), key


@pytest.mark.parametrize("path", SYMMETRY_PATHS)
@pytest.mark.parametrize("extra", [False, True])
def test_transposed_plan_of_symmetric_and_nearly_symmetric_patterns(gpu, oracle, extra,
                                                                    path, monkeypatch):
    """A symmetric pattern is its own transpose (the plan is copied); one
    directed entry more must be caught by the symmetry check."""
    _symmetry_path(monkeypatch, path)
    rng = np.random.default_rng(77)
    N = 500
    rp, ci = W.random_csr(rng, N, max_deg=40, empty_frac=0.1, dup_frac=0.2)
    rows = np.repeat(np.arange(N), np.diff(rp))
    a = set(zip(rows.tolist(), ci.tolist()))
    a |= {(c, r) for r, c in a}
    if extra:
        r0 = 123
        c0 = next(c for c in range(N - 1, -1, -1) if (r0, c) not in a)
        a.add((r0, c0))          # (c0, r0) stays absent
    pairs = sorted(a)
    rp_s = np.zeros(N + 1, dtype=np.int32)
    np.add.at(rp_s, np.array([p[0] for p in pairs]) + 1, 1)
    rp_s = np.cumsum(rp_s).astype(np.int32)
    ci_s = np.array([p[1] for p in pairs], dtype=np.int32)
    plan = gpu.Plan(_dev(rp_s), _dev(ci_s), N)
    got = plan.transpose().export()
    rp2, ci2 = _transpose_csr(rp_s, ci_s, N)
    b = oracle.bsb(rp2, ci2, N)
    for key in ("blk_off", "cols", "mask"):
        assert np.array_equal(got[key], b[key]), key
    same = all(np.array_equal(got[k], plan.export()[k]) for k in ("cols", "mask"))
    assert same == (not extra)
    # the library-allocated path (f3s_plan_transpose) gives the same plan
    L = gpu.load_library()
    h = L.f3s_plan_transpose(plan.handle)
    assert h
    alt = gpu.Plan._from_handle(h, DEV, N).export()
    for key in got:
        assert np.array_equal(got[key], alt[key]), key


def _bf16_dev(bits):
    return _dev(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)


def _grad_case_bf16(f3s, oracle, rp, ci, N, Qb, Kb, Vb, Gb, scale):
    """bf16 bit patterns in; forward (fp32 O, lse) and backward in bf16."""
    plan = f3s.Plan(_dev(rp), _dev(ci), N)
    plan_t = plan.transpose()
    q, k, v, g = (_bf16_dev(x) for x in (Qb, Kb, Vb, Gb))
    O, lse = f3s.forward_typed(plan, q, k, v, scale=scale, want_lse=True)
    dQ, dK, dV = f3s.backward(plan, plan_t, q, k, v, O, g, lse, scale=scale)
    torch.cuda.synchronize()
    H = Qb.shape[1] if Qb.ndim == 3 else 1
    wide = [oracle.widen_bf16(x) for x in (Qb, Kb, Vb, Gb)]
    for h in range(H):
        sl = (slice(None), h) if Qb.ndim == 3 else (slice(None),)
        ref = oracle.attention_bwd_f64(rp, ci, *(x[sl] for x in wide), scale)
        for name, got, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
            _check(f"bf16 {name}[h{h}]", got.cpu().numpy()[sl], r)


@pytest.mark.parametrize("d", [32, 64, 128, 160, 256])
@pytest.mark.parametrize("N", [17, 300])
def test_gradients_bf16_random_patterns(gpu, oracle, d, N):
    rng = np.random.default_rng(3 * d + N)
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 50), empty_frac=0.1, dup_frac=0.2)
    Qb, Kb, Vb, Gb = (W.to_bf16_bits(rng.standard_normal((N, d)).astype(np.float32))
                      for _ in range(4))
    _grad_case_bf16(gpu, oracle, rp, ci, N, Qb, Kb, Vb, Gb, 1.0 / math.sqrt(d))


@pytest.mark.parametrize("H,d", [(3, 64), (2, 256)])
def test_gradients_bf16_split_windows_and_heads(gpu, oracle, monkeypatch, H, d):
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")
    rng = np.random.default_rng(H * d)
    N = 700
    rp, ci = W.random_csr(rng, N, max_deg=200, empty_frac=0.05, dup_frac=0.1)
    Qb, Kb, Vb, Gb = (W.to_bf16_bits(rng.standard_normal((N, H, d)).astype(np.float32))
                      for _ in range(4))
    _grad_case_bf16(gpu, oracle, rp, ci, N, Qb, Kb, Vb, Gb, 1.0 / math.sqrt(d))


@pytest.mark.parametrize("k", [1, 4, 2, 5])
def test_gradients_bf16_workloads(gpu, oracle, k):
    c = W.make_config(k, dtype="bf16")
    print(f"workload {k} bf16 backward N={c['N']} d={c['d']}", flush=True)
    rng = np.random.default_rng(100 + k)
    Gb = W.to_bf16_bits(rng.standard_normal(c["Q"].shape).astype(np.float32))
    _grad_case_bf16(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"], c["Q"], c["K"], c["V"],
                    Gb, c["scale"])


def test_backward_rejects_mixed_or_other_types(gpu):
    rng = np.random.default_rng(5)
    N, d = 40, 64
    rp, ci = W.random_csr(rng, N, max_deg=10)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    plan_t = plan.transpose()
    q = _dev(rng.standard_normal((N, d)).astype(np.float16))
    O, lse = gpu.forward(plan, q, q, q)
    with pytest.raises(TypeError):
        gpu.backward(plan, plan_t, q, q, q, O, q.to(torch.bfloat16), lse)
    with pytest.raises(TypeError):
        qf = q.float()
        gpu.backward(plan, plan_t, qf, qf, qf, O, qf, lse)


def test_transpose_workspace_errors(gpu):
    rng = np.random.default_rng(9)
    N = 200
    rp, ci = W.random_csr(rng, N, max_deg=30)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    L = gpu.load_library()
    need = L.f3s_plan_transpose_workspace_bytes(plan.handle)
    assert need > 0 and L.f3s_plan_transpose_workspace_bytes(None) == 0
    ws = torch.empty(need + 512, dtype=torch.uint8, device=DEV)
    for ptr, size in ((ws.data_ptr(), need - 256), (ws.data_ptr() + 4, need), (None, need)):
        assert not L.f3s_plan_transpose_ws(plan.handle, ptr, size)
        assert L.f3s_last_error() == 1  # F3S_ERR_INVALID_VALUE


@pytest.mark.parametrize("waves", ["1", "2", "4"])
@pytest.mark.parametrize("d", [32, 64, 96, 128, 160, 192, 224, 256])
@pytest.mark.parametrize("N", [1, 17, 300])
def test_gradients_random_patterns(gpu, oracle, d, N, waves, monkeypatch):
    """Every feature size, with one wave per work item or two or four sharing it
    (forward and both backward passes; their partial sums combined in LDS)."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    rng = np.random.default_rng(d + 7 * N)
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 50), empty_frac=0.1, dup_frac=0.2)
    Q, K, V, G = (rng.standard_normal((N, d)).astype(np.float16) for _ in range(4))
    print(f"random N={N} d={d}", flush=True)
    _grad_case(gpu, oracle, rp, ci, N, Q, K, V, G, 1 / math.sqrt(d))


@pytest.mark.parametrize("k", [1, 4, 2, 5])
def test_gradients_workloads(gpu, oracle, k):
    c = W.make_config(k)
    rng = np.random.default_rng(11)
    G = rng.standard_normal(c["Q"].shape).astype(np.float16)
    print(f"workload {k} N={c['N']}", flush=True)
    _grad_case(gpu, oracle, c["row_ptr"], c["col_idx"], c["N"], c["Q"], c["K"], c["V"], G,
               c["scale"])


@pytest.mark.parametrize("k,H", [(2, 2), (4, 3), (5, 2)])
def test_gradients_workloads_several_heads(gpu, oracle, k, H):
    """Several heads of a workload in one backward call, every head against
    the oracle: the hub-heavy graph with split windows and window-major
    order, the molecule batch and the sequence workload head by head over
    their nearly uniform plans (with XCD ranges, and on the sequence
    workload two waves per item in the dQ pass)."""
    c = W.make_config(k, with_features=False)
    N, d = c["N"], 64
    rng = np.random.default_rng(40 + k)
    Q, K, V, G = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(4))
    print(f"workload {k} N={N} heads={H}", flush=True)
    _grad_case(gpu, oracle, c["row_ptr"], c["col_idx"], N, Q, K, V, G, 1 / math.sqrt(d))


@pytest.mark.parametrize("waves", ["1", "2", "4"])
@pytest.mark.parametrize("order", ["item", "head"])
@pytest.mark.parametrize("H,d", [(3, 64), (2, 160), (2, 256)])
def test_gradients_split_windows_and_heads(gpu, oracle, monkeypatch, H, d, order, waves):
    """Split windows in both plans; for d > 128 the dK/dV partials of one
    head fill a whole (double-width) partial row of the transposed plan.
    Both workgroup orders of the heads (window-major, the default at this
    size, and head by head, forced with a threshold of 0)."""
    if order == "head":
        monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", "0")
    else:
        monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", str(1 << 40))
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")
    rng = np.random.default_rng(12)
    N = 3000
    rows = [rng.choice(N, size=300, replace=False) if i < 20 else
            rng.choice(N, size=6, replace=False) for i in range(N)]
    rp = np.zeros(N + 1, dtype=np.int32)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32)
    Q, K, V, G = (rng.standard_normal((N, H, d)).astype(np.float16) for _ in range(4))
    plan, plan_t = _grad_case(gpu, oracle, rp, ci, N, Q, K, V, G, 0.125)
    assert plan.info["n_split"] > 0 and plan_t.info["n_split"] > 0


@pytest.mark.parametrize("dtype,d", [("f16", 128), ("bf16", 128), ("f16", 64), ("f16", 256)])
def test_gradients_million_node_workload_sampled(gpu, oracle, dtype, d):
    """The 1,048,576-node Chung-Lu workload (d = 128, and 64 and 256 for the
    feature-size sweep), whole backward on the GPU; the oracle runs on the
    sub-problem of 500 random keys and the 4 heaviest keys (hubs of about
    4,000 attending rows), every row attending to them with its full
    neighbour list: dQ is exact there on every one of those rows (about
    25,000), dK and dV on the sampled keys."""
    c = W.make_config(3, dtype=dtype, d=d)
    rp, ci, N, scale = c["row_ptr"], c["col_idx"], c["N"], c["scale"]
    rng = np.random.default_rng(31)
    g32 = rng.standard_normal(c["Q"].shape, dtype=np.float32)
    G = W.to_bf16_bits(g32) if dtype == "bf16" else g32.astype(np.float16)
    dev = _bf16_dev if dtype == "bf16" else _dev
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    plan_t = plan.transpose()
    q, k, v, g = (dev(x) for x in (c["Q"], c["K"], c["V"], G))
    if dtype == "bf16":
        O, lse = gpu.forward_typed(plan, q, k, v, scale=scale, want_lse=True)
    else:
        O, lse = gpu.forward(plan, q, k, v, scale=scale)
    dQ, dK, dV = gpu.backward(plan, plan_t, q, k, v, O, g, lse, scale=scale)
    torch.cuda.synchronize()
    del O, lse, q, k, v, g
    S = sample_keys(rp, ci, 500, 4, rng)
    R = np.union1d(S, rows_attending(rp, ci, S))
    mrp, mci, U = rows_subproblem(rp, ci, R)
    print(f"  {dtype}: {S.size} keys, {R.size} rows, sub-problem of {U.size} nodes and "
          f"{mci.size} entries", flush=True)
    sub = [x[U] for x in (c["Q"], c["K"], c["V"], G)]
    if dtype == "bf16":
        sub = [oracle.widen_bf16(x) for x in sub]
    ref = oracle.attention_bwd_f64(mrp, mci, *sub, scale)
    for name, got, r, rows in (("dQ", dQ, ref[0], R), ("dK", dK, ref[1], S),
                               ("dV", dV, ref[2], S)):
        sel = torch.from_numpy(rows).to(DEV)
        _check(f"{dtype} {name}", got.index_select(0, sel).cpu().numpy(),
               r[np.searchsorted(U, rows)])
    plan.close()
    plan_t.close()


@pytest.mark.parametrize("k,H", [(5, 1), (4, 1), (2, 1), (4, 4), (2, 2)])
def test_backward_xcd_ranges_order_gives_identical_gradients(gpu, k, H, monkeypatch):
    """Each XCD taking a consecutive range of the work list (with several
    heads, of one head's list, window-major or head by head) only reorders
    independent work items of both passes: bit-identical gradients."""
    c = W.make_config(k)
    rng = np.random.default_rng(70 + k)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    plan_t = plan.transpose()
    if H == 1:
        q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    else:
        shape = (c["N"], H, c["Q"].shape[1])
        q, kk, v = (_dev(rng.standard_normal(shape).astype(np.float16)) for _ in range(3))
    g = _dev(rng.standard_normal(tuple(q.shape)).astype(np.float16))
    O, lse = gpu.forward(plan, q, kk, v, scale=c["scale"])
    for head_major in ("0", "1000000000000"):
        monkeypatch.setenv("F3S_HEAD_MAJOR_BYTES", head_major)
        outs = []
        for chunks in ("0", "1"):
            monkeypatch.setenv("F3S_XCD_CHUNKS", chunks)
            outs.append(gpu.backward(plan, plan_t, q, kk, v, O, g, lse, scale=c["scale"]))
        torch.cuda.synchronize()
        for a, b in zip(*outs):
            assert torch.equal(a, b)


def test_backward_is_deterministic(gpu):
    c = W.make_config(2)
    rng = np.random.default_rng(13)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    plan_t = plan.transpose()
    q, k, v = _dev(c["Q"]), _dev(c["K"]), _dev(c["V"])
    g = _dev(rng.standard_normal(c["Q"].shape).astype(np.float16))
    O, lse = gpu.forward(plan, q, k, v)
    a = gpu.backward(plan, plan_t, q, k, v, O, g, lse)
    b = gpu.backward(plan, plan_t, q, k, v, O, g, lse)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_backward_argument_errors(gpu):
    c = W.make_config(1)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    other = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, k, v = _dev(c["Q"]), _dev(c["K"]), _dev(c["V"])
    O, lse = gpu.forward(plan, q, k, v)
    with pytest.raises(gpu.F3SError) as e:   # not the transpose of `plan`
        gpu.backward(plan, other, q, k, v, O, q, lse)
    assert e.value.code == 1
    plan_t = plan.transpose()
    big = torch.zeros((c["N"], 288), dtype=torch.float16, device=DEV)
    Ob = torch.zeros((c["N"], 288), dtype=torch.float32, device=DEV)
    with pytest.raises(gpu.F3SError) as e:   # d above 256
        gpu.backward(plan, plan_t, big, big, big, Ob, big, lse)
    assert e.value.code == 3


def test_backward_wide_addressing_above_4gib(gpu, oracle):
    """Gradients with Q, K, V, dO of more than 4 GiB each (N = 9,000,000,
    d = 256: 64-bit gathers in both passes).  Checked on sampled keys: the
    small oracle problem holds the sampled rows and every row attending to
    them (with their full neighbour lists), so dQ, dK and dV of the sampled
    rows are exact there."""
    N, d, scale = 9_000_000, 256, 1 / 16
    assert N * d * 2 > 2 ** 32
    i = torch.arange(N, dtype=torch.int64, device=DEV)
    ci = torch.stack([i, (i * 7919 + 13) % N, N - 1 - i], dim=1).reshape(-1).to(torch.int32)
    rp = (torch.arange(N + 1, dtype=torch.int64, device=DEV) * 3).to(torch.int32)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(9)
    Q, K, V, G = (torch.randn((N, d), generator=gen, device=DEV, dtype=torch.float32).half()
                  for _ in range(4))
    plan = gpu.Plan(rp, ci, N)
    plan_t = plan.transpose()
    O, lse = gpu.forward(plan, Q, K, V, scale=scale)
    dQ, dK, dV = gpu.backward(plan, plan_t, Q, K, V, O, G, lse, scale=scale)
    torch.cuda.synchronize()
    del O, lse
    rng = np.random.default_rng(10)
    S = np.unique(np.concatenate([[0, N - 1, N // 3], rng.integers(0, N, size=20),
                                  N - 1 - rng.integers(0, 500, size=10)]))
    St = torch.tensor(S, dtype=torch.int32, device=DEV)
    attending = (torch.isin(ci, St).nonzero().reshape(-1) // 3).cpu().numpy()
    R = sorted(set(S.tolist()) | set(attending.tolist()))
    rpn = rp.cpu().numpy().astype(np.int64)
    nb = {r: ci[int(rpn[r]):int(rpn[r + 1])].cpu().numpy() for r in R}
    U = sorted(set(R) | set(int(j) for a in nb.values() for j in a))
    loc = {u: k for k, u in enumerate(U)}
    rows = [[loc[int(j)] for j in nb[u]] if u in nb else [] for u in U]
    mrp = np.zeros(len(U) + 1, dtype=np.int32)
    mrp[1:] = np.cumsum([len(r) for r in rows])
    mci = np.array([c for r in rows for c in r], dtype=np.int32)
    idx = torch.tensor(U, device=DEV)
    q, k, v, gg = (x.index_select(0, idx).cpu().numpy() for x in (Q, K, V, G))
    gg[[loc[u] for u in U if u not in nb]] = 0    # rows outside R contribute nothing
    ref = oracle.attention_bwd_f64(mrp, mci, q, k, v, gg, scale)
    sel = torch.tensor(S, device=DEV)
    print(f"  {len(S)} sampled keys, {len(R)} rows in the small problem", flush=True)
    for name, got, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
        _check(name, got.index_select(0, sel).cpu().numpy(), r[[loc[int(s)] for s in S]])
    plan.close()
    plan_t.close()
    del Q, K, V, G, dQ, dK, dV
    torch.cuda.empty_cache()
