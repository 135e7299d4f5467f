"""Precision variants of the forward (bfloat16 and fp8 e4m3 inputs, fp16
output) on the GPU against the fp64 oracle.

Tolerances.  fp16 output adds one rounding of O (half an ulp: at most
2^-11 |O| relative) to the fp16 scheme's error, which stays inside the same
bar (max-abs 5e-3, relative Frobenius 1e-3) for N(0,1) inputs: the
probability error is <= 2^-11 * max|V| ~ 2.8e-3 and the output rounding
<= 2^-10 * |O| with |O| < 4 on all but a vanishing fraction of rows.  With
bfloat16 inputs the probabilities carry ~16 significant bits (two bf16
terms), so the error is fp32 accumulation only; the test asserts a relative
Frobenius error below 1e-4, ten times under the bar, which a single bf16
probability term (8 bits, ~2e-3) could not meet.  fp8 (e4m3) inputs are
widened to fp16 exactly before any product, so the fp16 scheme's bar applies
unchanged and the fp8 result equals the fp16 kernel's on the widened values.
"""
import ctypes
import math

import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
MAX_ABS = 5e-3
REL_FRO = 1e-3
BF16_REL_FRO = 1e-4


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _bf16_dev(bits):
    return _dev(bits.view(np.int16)).view(torch.bfloat16)


def _check(got, ref, max_abs=MAX_ABS, rel_fro=REL_FRO):
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), "non-finite output"
    diff = got - ref
    ma = float(np.abs(diff).max()) if diff.size else 0.0
    nref = float(np.linalg.norm(ref))
    rf = float(np.linalg.norm(diff)) / nref if nref > 0 else float(np.linalg.norm(diff))
    print(f"  max_abs={ma:.3e} rel_fro={rf:.3e}", flush=True)
    assert ma <= max_abs and rf <= rel_fro, (ma, rf)


@pytest.mark.parametrize("k", [1, 2, 4, 5, 3])
def test_bf16_inputs_workloads(gpu, oracle, k):
    c = W.make_config(k, dtype="bf16")
    print(f"workload {k} bf16 N={c['N']} d={c['d']}", flush=True)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, kk, v = (_bf16_dev(c[x]) for x in ("Q", "K", "V"))
    O, lse = gpu.forward_typed(plan, q, kk, v, scale=c["scale"], want_lse=True)
    torch.cuda.synchronize()
    ref, reflse = oracle.attention_bf16_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"],
                                            c["V"], c["scale"], want_lse=True)
    _check(O.cpu().numpy(), ref, rel_fro=BF16_REL_FRO)
    assert np.abs(lse.cpu().numpy() - reflse).max() < 1e-3


@pytest.mark.parametrize("d", [32, 64, 96, 128, 160, 192, 224, 256])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.float16])
def test_bf16_inputs_feature_sizes(gpu, oracle, d, out_dtype):
    rng = np.random.default_rng(d)
    N = 203
    rp, ci = W.random_csr(rng, N, max_deg=70, empty_frac=0.05, dup_frac=0.1)
    Q, K, V = (W.to_bf16_bits(rng.standard_normal((N, d), dtype=np.float32))
               for _ in range(3))
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    O, _ = gpu.forward_typed(plan, _bf16_dev(Q), _bf16_dev(K), _bf16_dev(V),
                             out_dtype=out_dtype, scale=1 / math.sqrt(d))
    torch.cuda.synchronize()
    ref = oracle.attention_bf16_f64(rp, ci, Q, K, V, 1 / math.sqrt(d))
    if out_dtype == torch.float32:
        _check(O.cpu().numpy(), ref, rel_fro=BF16_REL_FRO)
    else:
        _check(O.float().cpu().numpy(), ref)


@pytest.mark.parametrize("k", [1, 2, 4, 5, 3])
def test_f16_output_workloads(gpu, oracle, k):
    c = W.make_config(k)
    print(f"workload {k} fp16 out N={c['N']} d={c['d']}", flush=True)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    O16, _ = gpu.forward_typed(plan, q, kk, v, out_dtype=torch.float16, scale=c["scale"])
    O32, _ = gpu.forward_typed(plan, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    ref = oracle.attention_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                               c["scale"])
    _check(O16.float().cpu().numpy(), ref)
    # the fp16 output is the fp32 result rounded to nearest even, bit for bit
    assert torch.equal(O16, O32.half())


@pytest.mark.parametrize("in_dtype", [torch.float16, torch.bfloat16])
def test_f16_output_is_rounded_f32_output_with_split_windows_and_heads(
        gpu, monkeypatch, in_dtype):
    """Split windows (merge kernel) and head groups: fp16 O equals the fp32 O
    rounded, and bf16-input heads equal single-head runs bit for bit (one
    wave per work item for both, whatever the grid sizes)."""
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", "1")
    c = W.make_config(2, with_features=False)
    N, H, d = c["N"], 5, 64
    rng = np.random.default_rng(17)
    x = [torch.from_numpy(rng.standard_normal((N, H, d), dtype=np.float32)).to(in_dtype)
         for _ in range(3)]
    q, k, v = (t.to(DEV) for t in x)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), N)
    assert plan.info["n_split"] > 0
    O32, lse = gpu.forward_typed(plan, q, k, v, scale=0.125, want_lse=True)
    O16, lse16 = gpu.forward_typed(plan, q, k, v, out_dtype=torch.float16, scale=0.125,
                                   want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(O16, O32.half())
    assert torch.equal(lse, lse16)
    for h in (0, 4):
        Oh, _ = gpu.forward_typed(plan, q[:, h].contiguous(), k[:, h].contiguous(),
                                  v[:, h].contiguous(), scale=0.125)
        torch.cuda.synchronize()
        assert torch.equal(O32[:, h], Oh)


def test_typed_f16_f32_is_the_default_forward(gpu):
    c = W.make_config(2)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, k, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    a, la = gpu.forward(plan, q, k, v)
    b, lb = gpu.forward_typed(plan, q, k, v, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(la, lb)


def test_bf16_multi_head_matches_oracle(gpu, oracle):
    rng = np.random.default_rng(23)
    N, H, d = 500, 3, 64
    rp, ci = W.random_csr(rng, N, max_deg=40, empty_frac=0.05)
    X = [W.to_bf16_bits(rng.standard_normal((N, H, d), dtype=np.float32)) for _ in range(3)]
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    O, _ = gpu.forward_typed(plan, *(_bf16_dev(x) for x in X), scale=0.125)
    torch.cuda.synchronize()
    O = O.cpu().numpy()
    for h in range(H):
        ref = oracle.attention_bf16_f64(rp, ci, *(np.ascontiguousarray(x[:, h]) for x in X),
                                        0.125)
        _check(O[:, h], ref, rel_fro=BF16_REL_FRO)


def test_bf16_large_values_stay_exact(gpu, oracle):
    """Values far outside the fp16 range (bf16 has binary32's exponent): V
    rows of magnitude 1e6 and single-neighbour rows reproduce V exactly."""
    N, d = 64, 32
    rng = np.random.default_rng(29)
    rp = np.arange(N + 1, dtype=np.int32)
    ci = rng.integers(0, N, size=N).astype(np.int32)
    Q, K = (W.to_bf16_bits(rng.standard_normal((N, d), dtype=np.float32)) for _ in range(2))
    V = W.to_bf16_bits(1e6 * rng.standard_normal((N, d), dtype=np.float32))
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    O, _ = gpu.forward_typed(plan, _bf16_dev(Q), _bf16_dev(K), _bf16_dev(V), scale=0.2)
    torch.cuda.synchronize()
    assert np.array_equal(O.cpu().numpy().astype(np.float64),
                          oracle.widen_bf16(V)[ci])


def test_typed_argument_errors(gpu):
    c = W.make_config(1)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q = _dev(c["Q"])
    L = gpu.load_library()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    O = torch.empty((c["N"], 64), dtype=torch.float32, device=DEV)
    for ind, outd in ((2, 2), (7, 2), (0, 1), (0, 9), (-1, 2), (3, 3), (0, 3)):
        assert L.f3s_forward_typed(plan.handle, q.data_ptr(), q.data_ptr(), q.data_ptr(),
                                   ind, O.data_ptr(), outd, None, 1, 64, 0.1, s) == 3
    with pytest.raises(gpu.F3SError) as e:
        gpu.forward_typed(plan, q, q, q, out_dtype=torch.bfloat16)
    assert e.value.code == 3
    torch.cuda.synchronize()


def _fp8_dev(bits):
    return _dev(bits).view(torch.float8_e4m3fn)


@pytest.mark.parametrize("k", [1, 2, 4, 5, 3])
def test_fp8_inputs_workloads(gpu, oracle, k):
    c = W.make_config(k, dtype="fp8")
    print(f"workload {k} fp8 N={c['N']} d={c['d']}", flush=True)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, kk, v = (_fp8_dev(c[x]) for x in ("Q", "K", "V"))
    O, lse = gpu.forward_typed(plan, q, kk, v, scale=c["scale"], want_lse=True)
    torch.cuda.synchronize()
    ref, reflse = oracle.attention_e4m3_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"],
                                            c["V"], c["scale"], want_lse=True)
    _check(O.cpu().numpy(), ref)
    assert np.abs(lse.cpu().numpy() - reflse).max() < 2e-3


@pytest.mark.parametrize("d", [32, 64, 96, 128, 160, 192, 224, 256])
def test_fp8_equals_f16_on_widened_inputs(gpu, oracle, d):
    """e4m3 -> fp16 is exact and the fp8 kernel widens before any product,
    so its output must equal the fp16 kernel's on the widened inputs bit for
    bit (fp32 and fp16 outputs, split windows included)."""
    rng = np.random.default_rng(300 + d)
    N = 333
    rp, ci = W.random_csr(rng, N, max_deg=90, empty_frac=0.05, dup_frac=0.1)
    X = [W.to_e4m3_bits(2 * rng.standard_normal((N, d), dtype=np.float32)) for _ in range(3)]
    H = [oracle.widen_e4m3(x).astype(np.float16) for x in X]
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    for out_dtype in (torch.float32, torch.float16):
        a, la = gpu.forward_typed(plan, *(_fp8_dev(x) for x in X), out_dtype=out_dtype,
                                  scale=1 / math.sqrt(d), want_lse=True)
        b, lb = gpu.forward_typed(plan, *(_dev(h) for h in H), out_dtype=out_dtype,
                                  scale=1 / math.sqrt(d), want_lse=True)
        torch.cuda.synchronize()
        assert torch.equal(a, b) and torch.equal(la, lb)
    ref = oracle.attention_e4m3_f64(rp, ci, *X, 1 / math.sqrt(d))
    _check(a.float().cpu().numpy(), ref)


def test_fp8_multi_head_split_windows(gpu, oracle, monkeypatch):
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")
    c = W.make_config(2, with_features=False)
    N, H, d = c["N"], 3, 64
    rng = np.random.default_rng(31)
    X = [W.to_e4m3_bits(rng.standard_normal((N, H, d), dtype=np.float32)) for _ in range(3)]
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), N)
    assert plan.info["n_split"] > 0
    O, _ = gpu.forward_typed(plan, *(_fp8_dev(x) for x in X), scale=0.125)
    torch.cuda.synchronize()
    O = O.cpu().numpy()
    for h in range(H):
        ref = oracle.attention_e4m3_f64(c["row_ptr"], c["col_idx"],
                                        *(np.ascontiguousarray(x[:, h]) for x in X), 0.125)
        _check(O[:, h], ref)


def test_fp8_wide_addressing_above_4gib(gpu, oracle):
    """fp8 Q, K, V of more than 4 GiB each (N = 17,000,000, d = 256: one byte
    per element, so 64-bit gathers start above 16.7M rows), sampled rows
    against the oracle's e4m3 entry."""
    N, d, scale = 17_000_000, 256, 1 / 16
    assert N * d > 2 ** 32
    i = torch.arange(N, dtype=torch.int64, device=DEV)
    ci = torch.stack([i, (i * 7919 + 13) % N, N - 1 - i], dim=1).reshape(-1).to(torch.int32)
    rp = (torch.arange(N + 1, dtype=torch.int64, device=DEV) * 3).to(torch.int32)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(11)
    X = [torch.randn((N, d), generator=gen, device=DEV, dtype=torch.float32)
         .to(torch.float8_e4m3fn) for _ in range(3)]
    plan = gpu.Plan(rp, ci, N)
    O, _ = gpu.forward_typed(plan, *X, scale=scale)
    torch.cuda.synchronize()
    rng = np.random.default_rng(12)
    S = np.unique(np.concatenate([[0, N - 1], rng.integers(0, N, size=60),
                                  N - 1 - rng.integers(0, 300, size=20)]))
    rpn = rp.cpu().numpy().astype(np.int64)
    nb = {int(r): ci[int(rpn[r]):int(rpn[r + 1])].cpu().numpy() for r in S}
    U = sorted(set(int(s) for s in S) | set(int(j) for a in nb.values() for j in a))
    loc = {u: k for k, u in enumerate(U)}
    rows = [[loc[int(j)] for j in nb[u]] if u in nb else [] for u in U]
    mrp = np.zeros(len(U) + 1, dtype=np.int32)
    mrp[1:] = np.cumsum([len(r) for r in rows])
    mci = np.array([c for r in rows for c in r], dtype=np.int32)
    idx = torch.tensor(U, device=DEV)
    q, k, v = (x.view(torch.uint8).index_select(0, idx).cpu().numpy() for x in X)
    ref = oracle.attention_e4m3_f64(mrp, mci, q, k, v, scale)[[loc[int(s)] for s in S]]
    got = O.index_select(0, torch.tensor(S, device=DEV)).cpu().numpy()
    _check(got, ref)
    plan.close()
    del X, O
    torch.cuda.empty_cache()
