"""f3s_backward_noalloc (the backward pass for callers that cannot allocate:
its per-row records in the library's fixed device array) against
f3s_backward_typed with a caller-allocated record buffer, through the C ABI.

Both run the same kernels on the same inputs, so the gradients must be
bit-identical; two calls in a row, the second on a smaller pattern (the
array keeps the first call's records, which the second must not read), in
fp16 and bf16, and the size limit."""
import ctypes
import math

import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
F3S_OK, F3S_ERR_TOO_LARGE = 0, 6
DTYPE = {torch.float16: 0, torch.bfloat16: 1}


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _lib(gpu):
    L = gpu.load_library()
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    L.f3s_backward_noalloc.argtypes = ([vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp,
                                        i32, i32, ctypes.c_float, vp])
    L.f3s_backward_noalloc.restype = ctypes.c_int
    L.f3s_backward_noalloc_max_records.argtypes = []
    L.f3s_backward_noalloc_max_records.restype = ctypes.c_int64
    return L


def _case(gpu, rng, N, H, d, dtype, max_deg):
    rp, ci = W.random_csr(rng, N, max_deg=max_deg, empty_frac=0.05, dup_frac=0.1)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    plan_t = plan.transpose()
    shape = (N, H, d) if H > 1 else (N, d)
    q, k, v, g = (torch.randn(shape, device=DEV, dtype=torch.float32).to(dtype)
                  for _ in range(4))
    scale = 1.0 / math.sqrt(d)
    if dtype == torch.float16:
        O, lse = gpu.forward(plan, q, k, v, scale=scale)
    else:
        O, lse = gpu.forward_typed(plan, q, k, v, scale=scale, want_lse=True)
    return plan, plan_t, (q, k, v, g), O, lse, scale, H, d


def _noalloc(L, case):
    plan, plan_t, (q, k, v, g), O, lse, scale, H, d = case
    outs = [torch.full(q.shape, float("nan"), device=DEV) for _ in range(3)]
    stream = torch.cuda.current_stream(DEV).cuda_stream
    rc = L.f3s_backward_noalloc(plan.handle, plan_t.handle, q.data_ptr(), k.data_ptr(),
                                v.data_ptr(), DTYPE[q.dtype], O.data_ptr(), g.data_ptr(),
                                lse.data_ptr(), *(x.data_ptr() for x in outs), H, d, scale,
                                ctypes.c_void_p(stream))
    return rc, outs


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
def test_noalloc_backward_equals_backward(gpu, dtype):
    L = _lib(gpu)
    rng = np.random.default_rng(2024)
    # first call: 3000 rows, 2 heads, split windows; second: 257 rows, one head
    for N, H, d, max_deg in ((3000, 2, 64, 400), (257, 1, 128, 40)):
        print(f"noalloc {dtype} N={N} H={H} d={d}", flush=True)
        case = _case(gpu, rng, N, H, d, dtype, max_deg)
        plan, plan_t, (q, k, v, g), O, lse, scale, _, _ = case
        ref = gpu.backward(plan, plan_t, q, k, v, O, g, lse, scale=scale)
        rc, got = _noalloc(L, case)
        torch.cuda.synchronize()
        assert rc == F3S_OK, gpu.status_string(rc)
        for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
            assert torch.isfinite(a).all(), name
            assert torch.equal(a, b), name


def test_noalloc_backward_rejects_sizes_beyond_its_array(gpu):
    L = _lib(gpu)
    cap = L.f3s_backward_noalloc_max_records()
    assert cap == 1 << 21
    rng = np.random.default_rng(7)
    N, d = 64, 32
    H = cap // N + 1                       # N * H just above the capacity
    case = _case(gpu, rng, N, H, d, torch.float16, 10)
    rc, outs = _noalloc(L, case)
    torch.cuda.synchronize()
    assert rc == F3S_ERR_TOO_LARGE and L.f3s_last_error() == F3S_ERR_TOO_LARGE
    assert all(torch.isnan(x).all() for x in outs)   # nothing was launched
    # one head fewer fits and matches the allocating call
    H -= 1
    plan, plan_t = case[0], case[1]
    q, k, v, g = (x[:, :H].contiguous() for x in case[2])
    O, lse = gpu.forward(plan, q, k, v, scale=case[5])
    small = (plan, plan_t, (q, k, v, g), O, lse, case[5], H, d)
    rc, got = _noalloc(L, small)
    ref = gpu.backward(plan, plan_t, q, k, v, O, g, lse, scale=case[5])
    torch.cuda.synchronize()
    assert rc == F3S_OK
    for a, b in zip(got, ref):
        assert torch.equal(a, b)
