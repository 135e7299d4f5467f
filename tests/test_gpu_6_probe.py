"""The memory-system probe kernels (f3s_probe.h) that bench.py uses for its
measured bandwidth ceilings: the copy and write probes move exactly the bytes
they are given, the read probe leaves its sink alone (in practice), and the
access-pattern probe runs on every workload plan and on split windows
without touching memory outside O and the plan's own buffers."""
import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def test_stream_probes_move_the_given_bytes(gpu):
    n = (64 << 20) // 4 + 4 * 1000 + 4      # not a whole number of probe tiles
    src = torch.arange(n, dtype=torch.int32, device=DEV)
    guard = torch.full((n + 64,), -1, dtype=torch.int32, device=DEV)
    dst = guard[:n]
    gpu.probe_stream("copy", src, dst)
    torch.cuda.synchronize()
    assert torch.equal(dst, src) and bool((guard[n:] == -1).all())
    guard.fill_(-1)
    gpu.probe_stream("write", dst)
    torch.cuda.synchronize()
    assert bool((guard[n:] == -1).all()) and not bool((dst == -1).any())
    sink = torch.zeros(256, dtype=torch.int32, device=DEV)
    gpu.probe_stream("read", src, sink)
    torch.cuda.synchronize()
    with pytest.raises(ValueError):
        gpu.probe_stream("copy", src, dst[:-4])
    L = gpu.load_library()
    assert L.f3s_probe_read(src.data_ptr() + 4, 64, sink.data_ptr(), None) == 1
    assert L.f3s_probe_copy(src.data_ptr(), dst.data_ptr(), 20, None) == 1


@pytest.mark.parametrize("row_bytes", [16, 64, 128, 256, 1024])
def test_row_probe_reads_only_its_table(gpu, row_bytes):
    """f3s_probe_rows reads a table of rows * row_bytes bytes (its rows come
    from a hash taken modulo rows), changes neither the table nor, in
    practice, its sink, and reports the bytes it read; bad sizes are rejected
    before any launch."""
    rows = 1000
    table = torch.arange(rows * row_bytes // 4, dtype=torch.int32, device=DEV)
    sink = torch.zeros(256, dtype=torch.int32, device=DEV)
    for u in (1, 2, 4, 8, 16):
        nbytes = gpu.probe_rows(table, rows, row_bytes, sink, in_flight=u, workgroups=64,
                                rounds=3)
        assert nbytes == 64 * 3 * u * 4096
    torch.cuda.synchronize()
    assert not bool(sink.any())
    assert torch.equal(table, torch.arange(rows * row_bytes // 4, dtype=torch.int32,
                                           device=DEV))
    L = gpu.load_library()
    p, s = table.data_ptr(), sink.data_ptr()
    assert L.f3s_probe_rows(p, rows, 48, 8, 64, 1, s, None) == 3         # F3S_ERR_UNSUPPORTED
    assert L.f3s_probe_rows(p, rows, row_bytes, 3, 64, 1, s, None) == 3
    assert L.f3s_probe_rows(p, 0, row_bytes, 8, 64, 1, s, None) == 1     # F3S_ERR_INVALID_VALUE
    assert L.f3s_probe_rows(p, rows, row_bytes, 8, 0, 1, s, None) == 1
    assert L.f3s_probe_rows(p, rows, row_bytes, 8, 64, 0, s, None) == 1
    assert L.f3s_probe_rows(p + 4, rows, row_bytes, 8, 64, 1, s, None) == 1
    assert L.f3s_probe_rows(p, 1 << 32, row_bytes, 8, 64, 1, s, None) == 1
    with pytest.raises(ValueError):
        gpu.probe_rows(table, rows + 1, row_bytes, sink)


@pytest.mark.parametrize("k", [1, 2, 4, 5])
def test_pattern_probe_runs_on_the_workload_plans(gpu, k, monkeypatch):
    if k == 2:
        monkeypatch.setenv("F3S_PIECE_BLOCKS", "4")   # many split windows
    c = W.make_config(k)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    guard = torch.full((c["N"] + 16, c["d"]), -3.0, dtype=torch.float32, device=DEV)
    O = guard[: c["N"]]
    gpu.probe_gather(plan, q, kk, v, O)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(O).all())
    assert bool((guard[c["N"]:] == -3.0).all())
    # the same accesses loaded into LDS
    O.fill_(-3.0)
    gpu.probe_gather(plan, q, kk, v, O, lds=True)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(O).all())
    assert bool((guard[c["N"]:] == -3.0).all())
    # the operator still gives its result on the same plan afterwards
    O2 = gpu.run(plan, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    assert bool(torch.isfinite(O2).all())


@pytest.mark.parametrize("k,waves", [(1, "4"), (1, "1"), (2, "1"), (4, "1"), (5, "1")])
def test_traced_run_equals_run_and_records_every_workgroup(gpu, k, waves, monkeypatch):
    """f3s_run_trace writes exactly f3s_run's O (split windows and their
    merge included) and one record per workgroup: end after start, the
    workgroup's index, and compute-unit ids that name at most 256 CUs."""
    monkeypatch.setenv("F3S_WAVES_PER_ITEM", waves)
    c = W.make_config(k)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    ref = gpu.run(plan, q, kk, v, scale=c["scale"])
    O, rec = gpu.run_trace(plan, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    assert torch.equal(O, ref)
    r = rec.cpu().numpy().view(np.uint32).astype(np.uint64)
    n = plan.info["n_items"]
    assert r.shape == (n, 8)
    t0 = r[:, 0] | (r[:, 1] << np.uint64(32))
    t1 = r[:, 2] | (r[:, 3] << np.uint64(32))
    assert np.all(t1 >= t0) and np.all(t0 > 0)
    assert np.array_equal(r[:, 6], np.arange(n))
    import bench
    stats = bench.cu_balance(r.astype(np.uint32), gpu.wall_clock_khz(0))
    print(f"  {stats}", flush=True)
    assert 1 <= stats["cus"] <= 256
    assert gpu.wall_clock_khz(0) > 0


def test_lds_pattern_probe_argument_errors(gpu):
    """f3s_probe_gather_lds takes d = 32, 64 or 128 (its LDS areas) and
    refuses other feature sizes before any launch."""
    rng = np.random.default_rng(11)
    N = 64
    rp, ci = W.random_csr(rng, N, max_deg=8)
    plan = gpu.Plan(_dev(rp), _dev(ci), N)
    L = gpu.load_library()
    for d, want in ((256, 3), (96, 3), (48, 3)):
        q = torch.zeros((N, d), dtype=torch.float16, device=DEV)
        o = torch.zeros((N, d), dtype=torch.float32, device=DEV)
        assert L.f3s_probe_gather_lds(plan.handle, q.data_ptr(), q.data_ptr(), q.data_ptr(),
                                      o.data_ptr(), d, None) == want
    q = torch.zeros((N, 64), dtype=torch.float16, device=DEV)
    o = torch.zeros((N, 64), dtype=torch.float32, device=DEV)
    assert L.f3s_probe_gather_lds(plan.handle, q.data_ptr() + 4, q.data_ptr(), q.data_ptr(),
                                  o.data_ptr(), 64, None) == 1
    assert L.f3s_probe_gather_lds(None, q.data_ptr(), q.data_ptr(), q.data_ptr(),
                                  o.data_ptr(), 64, None) == 1
