"""Out-of-memory handling of the plan builds: every device allocation of
f3s_plan and f3s_plan_transpose is made to fail in turn (from the host, with
F3S_ALLOC_LIMIT_BYTES), each call returns NULL with F3S_ERR_OUT_OF_MEMORY,
and repeating a failing call does not lower the device's free memory (each
allocation here is megabytes, so one leaked per call would show at once).
The library-allocating entry points are called through the C ABI, so torch's
caching allocator takes no part."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
F3S_ERR_OUT_OF_MEMORY = 4


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


TOL = 2 << 20    # bytes


def _free():
    torch.cuda.synchronize()
    return torch.cuda.mem_get_info(DEV)[0]


def _no_leak(call, reps=8):
    """call() once, then `reps` more times: free memory must not drop."""
    call()
    before = _free()
    for _ in range(reps):
        call()
    after = _free()
    assert before - after <= TOL, (before, after)


def test_every_plan_allocation_failing_leaks_nothing(gpu, monkeypatch):
    L = gpu.load_library()
    c = W.make_config(2, with_features=False)   # split windows: three allocations
    rp, ci, N = _dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"]
    ok = L.f3s_plan(rp.data_ptr(), ci.data_ptr(), N)
    assert ok
    info = gpu.PlanInfo()
    assert L.f3s_plan_info(ok, ctypes.byref(info)) == 0
    assert info.n_split > 0
    L.f3s_destroy(ok)
    # limits from nothing to above the largest allocation: each makes a later
    # allocation fail (the build's scratch, the plan's arrays, the partials)
    failures = 0
    for lim in (0, 1 << 20, 2 << 20, 4 << 20, 6 << 20, 8 << 20, 12 << 20, 1 << 30):
        monkeypatch.setenv("F3S_ALLOC_LIMIT_BYTES", str(lim))
        res = []

        def call():
            h = L.f3s_plan(rp.data_ptr(), ci.data_ptr(), N)
            res.append(bool(h))
            if h:
                L.f3s_destroy(h)
            else:
                assert L.f3s_last_error() == F3S_ERR_OUT_OF_MEMORY, lim
        _no_leak(call)
        failures += not res[0]
        print(f"  limit {lim}: plan {'built' if res[0] else 'out of memory'}", flush=True)
    assert failures >= 2 and res[-1]


@pytest.mark.parametrize("k", [5, 2])
def test_transpose_allocation_failing_leaks_nothing(gpu, monkeypatch, k):
    """A directed pattern (a new plan is built) and a symmetric one (the
    plan is copied)."""
    L = gpu.load_library()
    c = W.make_config(k, with_features=False)
    rp, ci, N = _dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"]
    src = L.f3s_plan(rp.data_ptr(), ci.data_ptr(), N)
    assert src
    failures = 0
    for lim in (0, 1 << 20, 8 << 20, 32 << 20, 1 << 30):
        monkeypatch.setenv("F3S_ALLOC_LIMIT_BYTES", str(lim))
        res = []

        def call():
            t = L.f3s_plan_transpose(src)
            res.append(bool(t))
            if t:
                L.f3s_destroy(t)
            else:
                assert L.f3s_last_error() == F3S_ERR_OUT_OF_MEMORY, lim
        _no_leak(call)
        failures += not res[0]
        print(f"  limit {lim}: transpose {'built' if res[0] else 'out of memory'}", flush=True)
    assert failures >= 1 and res[-1]
    L.f3s_destroy(src)


def test_segment_plan_allocation_failing_leaks_nothing(gpu, monkeypatch):
    """f3s_plan_segments (the molecule batch, windows aligned to its graphs):
    the window rows travel in the build's scratch and in the plan's arrays;
    every failing limit gives F3S_ERR_OUT_OF_MEMORY and leaks nothing."""
    L = gpu.load_library()
    c = W.make_config(4, with_features=False)
    rp, ci, N = _dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"]
    seg = np.ascontiguousarray(c["seg_ptr"], dtype=np.int32)
    sp = seg.ctypes.data_as(ctypes.c_void_p)
    failures = 0
    for lim in (0, 1 << 20, 2 << 20, 4 << 20, 1 << 30):
        monkeypatch.setenv("F3S_ALLOC_LIMIT_BYTES", str(lim))
        res = []

        def call():
            h = L.f3s_plan_segments(rp.data_ptr(), ci.data_ptr(), N, sp, seg.size - 1)
            res.append(bool(h))
            if h:
                L.f3s_destroy(h)
            else:
                assert L.f3s_last_error() == F3S_ERR_OUT_OF_MEMORY, lim
        _no_leak(call)
        failures += not res[0]
        print(f"  limit {lim}: plan {'built' if res[0] else 'out of memory'}", flush=True)
    assert failures >= 2 and res[-1]
