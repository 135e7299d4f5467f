"""Benchmark of the fused 3S operator on one MI355X.

Default workload: the 1,048,576-node Chung-Lu graph (exponent 2.5, mean
degree 16, permuted ids, d = 128): the largest graph workload, on which the
HBM-bandwidth target is set.  One "step" is one f3s_run call (the whole
operator: block scores, mask, online softmax, value product, normalisation)
over device-resident inputs.

Prints ONE JSON line.  `value` is effective GFLOP/s = 4 * nnz * d / time,
with nnz the distinct (row, column) pairs.  `roofline` prices the fused
kernel against HBM bandwidth with the algorithmic bytes of one launch;
`cpu_baseline` times the fp64 oracle on a bounded row sample on the host.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MFMA_F16_PEAK_TFLOPS = 2500.0  # dense fp16 MFMA, published
METRIC = "ms per fused 3S call and effective GFLOP/s (4*nnz*d) at 1 MI355X"
COUNTERS_FILE = os.path.join(HERE, "profiles", "fused3s_cl25_d128_counters.json")
KERNEL_SOURCES = [os.path.join(HERE, "paper_2505_08098_amd", "csrc", f)
                  for f in ("fused3s.hip", "fused3s_kernel.h", "kernel_common.h",
                            "f3s_internal.h")]


def kernel_source_hash(root=None):
    """Hash of the fused kernel's source code with comments and whitespace
    removed (a comment edit does not invalidate measured counters).  Of the
    internal header only the part the kernel uses counts: the constants, the
    work item and the plan struct, i.e. everything before the launcher
    declarations."""
    import re
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        if root is not None:
            p = os.path.join(root, os.path.relpath(p, HERE))
        with open(p) as f:
            text = f.read()
        if p.endswith("f3s_internal.h"):
            text = text.split("// ---- plan kernels")[0]
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("".join(text.split()).encode())
    return h.hexdigest()[:16]


def algorithmic_bytes(info, d, heads=1, in_size=2, out_size=4):
    """Bytes one launch must move at minimum without cache reuse: Q read and
    O written once ((in_size + out_size)*N*d per head: 6*N*d for fp16 in,
    fp32 out), the K and V rows of every distinct (window, column) pair
    (2*in_size*d per pair and head), 64 B of column ids + 32 B of bitmap per
    block, 16 B per work item (plan data counted once: the heads of a window
    share it)."""
    return (heads * ((in_size + out_size) * info["N"] * d
                     + 2 * in_size * d * info["n_unique"])
            + 96 * info["n_blocks"] + 16 * info["n_items"])


def traffic_from_counters(d):
    """HBM bytes per launch measured by rocprofv3 counters, if they were taken
    on the current kernel source; otherwise None."""
    try:
        with open(COUNTERS_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash() or rec.get("d") != d:
        return None
    return rec.get("hbm_bytes_per_launch")


def library_switches():
    """The library's F3S_* environment switches (ablations and tuning) set for
    this run, as {"switches": {...}}, or {} when none is set: a line measured
    under an ablation says so."""
    sw = {k: v for k, v in sorted(os.environ.items()) if k.startswith("F3S_")}
    return {"switches": sw} if sw else {}


def host_threads():
    """Threads of the oracle baseline: every core this process may run on
    (its affinity mask), unless OMP_NUM_THREADS sets the host's CPU share
    lower.  Returns (threads, affinity core count)."""
    cores = len(os.sched_getaffinity(0))
    try:
        share = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        share = 0
    return (min(cores, share) if share > 0 else cores), cores


def cpu_baseline(c, O_gpu, sample_rows, threads=0):
    import numpy as np
    import oracle
    affinity = len(os.sched_getaffinity(0))
    if threads <= 0:
        threads, affinity = host_threads()
    r1 = min(c["N"], sample_rows)
    t0 = time.perf_counter()
    ref = oracle.attention_rows_f64(c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"],
                                    c["scale"], 0, r1, threads=threads)
    dt = time.perf_counter() - t0
    rp = c["row_ptr"]
    nnz_sample = 0
    ci = c["col_idx"]
    for lo in range(0, r1, 65536):
        hi = min(r1, lo + 65536)
        rows = np.repeat(np.arange(lo, hi), np.diff(rp[lo:hi + 1]))
        key = rows.astype(np.int64) * c["N"] + ci[rp[lo]:rp[hi]]
        nnz_sample += np.unique(key).size
    flops = 4.0 * nnz_sample * c["d"]
    got = O_gpu[:r1].astype(np.float64)
    diff = got - ref
    parity = dict(rows=r1, max_abs=float(np.abs(diff).max()),
                  rel_fro=float(np.linalg.norm(diff) / np.linalg.norm(ref)))
    return dict(value=flops / dt / 1e9, unit="GFLOP/s", cores=threads,
                affinity_cores=affinity, kind="oracle",
                sample=f"rows 0..{r1} of the same workload ({nnz_sample} nnz, "
                       f"{dt:.2f} s wall, fp64)",
                ms=dt * 1e3), parity


def plan_stats(plan):
    """The structure metrics of the paper's dataset tables for this pattern:
    blocks per row window (mean, coefficient of variation, deciles, max),
    distinct columns per window and non-zeros per 16x16 block."""
    import numpy as np
    info = plan.info
    nb = np.diff(plan.export()["blk_off"]).astype(np.float64)
    mean = float(nb.mean()) if nb.size else 0.0
    dec = np.percentile(nb, [10, 20, 30, 40, 50, 60, 70, 80, 90]) if nb.size else [0] * 9
    return {
        "windows": int(nb.size),
        "blocks_per_window": {
            "mean": round(mean, 3),
            "cv": round(float(nb.std() / mean), 4) if mean > 0 else 0.0,
            "deciles_p10_p90": [round(float(x), 1) for x in dec],
            "max": int(nb.max()) if nb.size else 0,
        },
        "unique_cols_per_window": round(info["n_unique"] / max(1, info["n_windows"]), 3),
        "nnz_per_block": round(info["nnz"] / max(1, info["n_blocks"]), 3),
        "block_fill": round(info["nnz"] / max(1, 256 * info["n_blocks"]), 4),
    }


# Table sizes (MB) of the random-row gather sweep: inside one XCD's 4 MB L2,
# above it, inside the 256 MB Infinity Cache, and far above it.
GATHER_SWEEP_MB = (2, 4, 8, 16, 32, 64, 128, 256, 1024, 4096)


def memory_ceilings(plan, Q, K, V, O, d, achieved_gbs, alg_bytes, stream, dev, reps=20,
                    kv_rows=0, row_bytes=0):
    """Bandwidth ceilings measured in this process with the library's probe
    kernels: a streaming read, copy and write over 4 GiB (16x the 256 MB
    Infinity Cache, so DRAM serves them); uniformly random gathers of whole
    rows of `row_bytes` (the workload's K/V row) from a table as large as K
    and V together (`kv_rows` rows) and from tables of GATHER_SWEEP_MB
    (f3s_probe_rows: the hardware's rate for gather-bound work with that
    working set); and the fused kernel's own access pattern on this plan
    without its arithmetic (f3s_probe_gather; its rate counts the same
    algorithmic bytes).  Streams: mean of `reps` timed calls after one
    untimed call; the gather probes: one HIP graph of `reps` calls (as the
    operator's steps are timed)."""
    import numpy as np
    import torch
    import paper_2505_08098_amd as f3s

    def timed(fn):
        fn()
        a = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
        b = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
        for k in range(reps):
            a[k].record(stream)
            fn()
            b[k].record(stream)
        torch.cuda.synchronize()
        return float(np.mean([x.elapsed_time(y) for x, y in zip(a, b)]))

    nbytes = 4 << 30
    out = {}
    buf = torch.empty(nbytes // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(buf)
    sink = torch.zeros(256, dtype=torch.int32, device=dev)
    f3s.probe_stream("write", buf, stream=stream)
    out["stream_read_GBs"] = round(nbytes / timed(
        lambda: f3s.probe_stream("read", buf, sink, stream=stream)) / 1e6, 1)
    out["stream_copy_GBs"] = round(2 * nbytes / timed(
        lambda: f3s.probe_stream("copy", buf, dst, stream=stream)) / 1e6, 1)
    out["stream_write_GBs"] = round(nbytes / timed(
        lambda: f3s.probe_stream("write", dst, stream=stream)) / 1e6, 1)
    if row_bytes in (16, 32, 64, 128, 256, 512, 1024):
        def rows_rate(n_rows):
            # on torch's current stream: the capturing stream inside graph_timed
            call = lambda: f3s.probe_rows(buf, n_rows, row_bytes, sink, in_flight=8,
                                          workgroups=2048, rounds=4)
            nb = 2048 * 4 * 8 * 4096
            return round(nb / graph_timed(call, reps, dev)[1] / 1e6, 1)
        out["random_rows_bytes"] = row_bytes
        out["random_rows_GBs_by_table_MB"] = {
            str(mb): rows_rate((mb << 20) // row_bytes) for mb in GATHER_SWEEP_MB}
        if 0 < kv_rows * row_bytes <= nbytes:
            out["random_rows_table_MB"] = round(kv_rows * row_bytes / 1e6, 1)
            out["random_rows_GBs"] = rows_rate(kv_rows)
            out["frac_of_random_rows"] = round(achieved_gbs / out["random_rows_GBs"], 4)
    del buf, dst, sink
    torch.cuda.empty_cache()
    out["stream_bytes"] = nbytes
    if Q is not None:
        # one HIP graph of `reps` probe calls, timed like the operator's steps
        ms = graph_timed(lambda: f3s.probe_gather(plan, Q, K, V, O), reps, dev)[1]
        out["pattern_gather_ms"] = round(ms, 5)
        out["pattern_gather_GBs"] = round(alg_bytes / ms / 1e6, 1)
        out["frac_of_pattern_gather"] = round(achieved_gbs / out["pattern_gather_GBs"], 4)
        if d <= 128 and Q.shape[0] * d * 2 <= 0xFFFFFFF0:
            # the same accesses into LDS, rows in flight bounded by the hardware only
            ms = graph_timed(lambda: f3s.probe_gather(plan, Q, K, V, O, lds=True), reps,
                             dev)[1]
            out["pattern_gather_lds_ms"] = round(ms, 5)
    out["frac_of_stream_read"] = round(achieved_gbs / out["stream_read_GBs"], 4)
    return out


def gather_sweep(dev, reps=10):
    """f3s_probe_rows over tables of GATHER_SWEEP_MB with 64-, 128- and
    256-byte rows, 1 to 16 rows in flight per thread and 2, 4 or 8 workgroups
    of 256 threads per CU (about 256 MB read per call, one HIP graph of
    `reps` calls each): what the memory system delivers to random row
    gathers, and whether more requests in flight raise it.  Then, at the
    ceilings' launch shape (8 rows in flight, 2,048 workgroups), rows of 128
    to 1024 bytes: whether longer contiguous rows (a K row and a V row side
    by side) are gathered at a higher byte rate."""
    import torch
    import paper_2505_08098_amd as f3s
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    buf = torch.empty((4 << 30) // 4, dtype=torch.int32, device=dev)
    sink = torch.zeros(256, dtype=torch.int32, device=dev)
    f3s.probe_stream("write", buf)
    rows = []
    for mb in GATHER_SWEEP_MB:
        for rb in (64, 128, 256):
            for per_cu in (2, 4, 8):
                for u in (1, 2, 4, 8, 16):
                    wg = per_cu * cus
                    rounds = max(1, (256 << 20) // (wg * u * 4096))
                    n = (mb << 20) // rb
                    call = lambda: f3s.probe_rows(buf, n, rb, sink, in_flight=u,
                                                  workgroups=wg, rounds=rounds)
                    ms = graph_timed(call, reps, dev)[1]
                    rows.append({"table_MB": mb, "row_bytes": rb, "workgroups_per_cu": per_cu,
                                 "in_flight": u,
                                 "GBs": round(wg * rounds * u * 4096 / ms / 1e6, 1)})
        print(f"gather sweep: {mb} MB done", file=sys.stderr, flush=True)
    by_size = []
    for mb in GATHER_SWEEP_MB:
        for rb in (128, 256, 512, 1024):
            n = (mb << 20) // rb
            call = lambda: f3s.probe_rows(buf, n, rb, sink, in_flight=8, workgroups=2048,
                                          rounds=4)
            ms = graph_timed(call, reps, dev)[1]
            by_size.append({"table_MB": mb, "row_bytes": rb,
                            "GBs": round(2048 * 4 * 8 * 4096 / ms / 1e6, 1)})
    print("gather sweep: row sizes done", file=sys.stderr, flush=True)
    print(json.dumps({"metric": "random whole-row gather rate (f3s_probe_rows)", "n_gpus": 1,
                      "cus": cus, "rows": rows, "row_sizes": by_size}), flush=True)


def dram_check(args, stream, dev, reps=10):
    """The operator on uniform_random_graph (8,388,608 nodes, 16 random
    neighbours + self, d = 128: K and V 17x the Infinity Cache, so the gathers
    are served by DRAM): ms per call and algorithmic GB/s, the bandwidth the
    kernel sustains from HBM itself.  Features: seeded N(0,1) fp16 drawn on
    the device."""
    import numpy as np
    import torch
    import paper_2505_08098_amd as f3s
    from paper_2505_08098_amd import workloads as W
    d = 128
    rp, ci = W.uniform_random_graph(args.seed)
    N = len(rp) - 1
    plan = f3s.Plan(torch.from_numpy(rp).to(dev), torch.from_numpy(ci).to(dev), N)
    del rp, ci
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    Q, K, V = (torch.randn((N, d), generator=gen, device=dev).half() for _ in range(3))
    O = torch.empty((N, d), dtype=torch.float32, device=dev)
    scale = 1.0 / math.sqrt(d)
    for _ in range(2):
        f3s.run(plan, Q, K, V, scale=scale, out=O, stream=stream)
    a = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
    b = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
    for k in range(reps):
        a[k].record(stream)
        f3s.run(plan, Q, K, V, scale=scale, out=O, stream=stream)
        b[k].record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([x.elapsed_time(y) for x, y in zip(a, b)]))
    info = plan.info
    nbytes = algorithmic_bytes(info, d)
    gbs = nbytes / ms / 1e6
    # the same accesses without arithmetic, and random 256-byte rows of K
    # (2.1 GB, 8x the Infinity Cache): the DRAM-side ceilings of this graph
    for _ in range(2):
        f3s.probe_gather(plan, Q, K, V, O, stream=stream)
    a0, b0 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record(stream)
    for _ in range(reps):
        f3s.probe_gather(plan, Q, K, V, O, stream=stream)
    b0.record(stream)
    torch.cuda.synchronize()
    ms_probe = a0.elapsed_time(b0) / reps
    # the same accesses into LDS with no limit on the rows in flight
    for _ in range(2):
        f3s.probe_gather(plan, Q, K, V, O, stream=stream, lds=True)
    a0.record(stream)
    for _ in range(reps):
        f3s.probe_gather(plan, Q, K, V, O, stream=stream, lds=True)
    b0.record(stream)
    torch.cuda.synchronize()
    ms_probe_lds = a0.elapsed_time(b0) / reps
    sink = torch.zeros(256, dtype=torch.int32, device=dev)
    rows_call = lambda: f3s.probe_rows(K, N, 2 * d, sink, in_flight=8, workgroups=2048,
                                       rounds=16, stream=stream)
    rows_call()
    a0.record(stream)
    for _ in range(reps):
        rows_call()
    b0.record(stream)
    torch.cuda.synchronize()
    rows_gbs = 2048 * 16 * 8 * 4096 / (a0.elapsed_time(b0) / reps) / 1e6
    out = {"workload": f"uniform random graph N={N}, 16 random neighbours + self, d={d}",
           "nnz": info["nnz"], "n_unique": info["n_unique"], "ms": round(ms, 4),
           "algorithmic_bytes": nbytes, "achieved_GBs": round(gbs, 1),
           "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
           "gflops_eff": round(4.0 * info["nnz"] * d / ms / 1e6, 1),
           "pattern_gather_ms": round(ms_probe, 4),
           "pattern_gather_GBs": round(nbytes / ms_probe / 1e6, 1),
           "pattern_gather_lds_ms": round(ms_probe_lds, 4),
           "random_rows_of_K_GBs": round(rows_gbs, 1)}
    plan.close()
    del Q, K, V, O
    torch.cuda.empty_cache()
    return out


def cu_balance(rec, khz):
    """Per compute unit busy time from f3s_run_trace records (one per
    workgroup): busy = the union of its workgroups' [start, end] intervals,
    end = its last workgroup's end, both in microseconds from the kernel's
    first start."""
    import numpy as np
    rec = rec.astype(np.uint64)
    t0 = rec[:, 0] | (rec[:, 1] << np.uint64(32))
    t1 = rec[:, 2] | (rec[:, 3] << np.uint64(32))
    hw, xcc = rec[:, 4], rec[:, 5]
    key = ((xcc & np.uint64(15)) << np.uint64(16)) | \
          (((hw >> np.uint64(13)) & np.uint64(7)) << np.uint64(8)) | \
          (((hw >> np.uint64(12)) & np.uint64(1)) << np.uint64(4)) | \
          ((hw >> np.uint64(8)) & np.uint64(15))
    base = t0.min()
    us = 1e3 / khz
    s = (t0 - base).astype(np.float64) * us
    e = (t1 - base).astype(np.float64) * us
    busy, end = [], []
    for k in np.unique(key):
        sel = key == k
        order = np.argsort(s[sel], kind="stable")
        ss, ee = s[sel][order], e[sel][order]
        tot, cur_s, cur_e = 0.0, ss[0], ee[0]
        for a, b in zip(ss[1:], ee[1:]):
            if a > cur_e:
                tot += cur_e - cur_s
                cur_s, cur_e = a, b
            else:
                cur_e = max(cur_e, b)
        busy.append(tot + cur_e - cur_s)
        end.append(ee.max())
    busy, end = np.array(busy), np.array(end)
    span = float(e.max())

    def st(x):
        return {"min": round(float(x.min()), 2), "mean": round(float(x.mean()), 2),
                "max": round(float(x.max()), 2)}
    dur = e - s
    q = np.percentile(dur, [10, 50, 90])
    return {"cus": int(busy.size), "workgroups": int(rec.shape[0]), "span_us": round(span, 2),
            "busy_us": st(busy), "end_us": st(end),
            "busy_frac_mean": round(float(busy.mean()) / span, 4),
            "idle_tail_us_mean": round(span - float(end.mean()), 2),
            "workgroup_us": {"mean": round(float(dur.mean()), 3), "p10": round(float(q[0]), 3),
                             "p50": round(float(q[1]), 3), "p90": round(float(q[2]), 3)},
            # workgroups resident on a CU at once, averaged over its busy time
            "resident_per_cu_mean": round(float(dur.sum()) / float(busy.sum()), 2)}


def bench_cu_trace(args, c, make_plan, Q, K, V, stream, dev):
    """Per-CU busy time of one traced forward call with the heavy-first work
    list and with the window-order work list (F3S_NO_REORDER=0 and 1), the
    load-balance comparison of the paper's row-window reordering ablation.
    The library's own choice is one of the two (`library_order`)."""
    import numpy as np
    import torch
    import paper_2505_08098_amd as f3s
    out = {"metric": "per-CU busy time of one fused 3S call (f3s_run_trace)",
           "n_gpus": 1, "config": {"workload": c["name"], "N": c["N"], "d": c["d"],
                                   "windows": "aligned to the graphs" if args.segments
                                   else "16 rows"},
           "wall_clock_khz": f3s.wall_clock_khz(0), "orders": {}}
    prev = os.environ.get("F3S_NO_REORDER")
    for order in ("heavy_first", "window_order"):
        os.environ["F3S_NO_REORDER"] = "1" if order == "window_order" else "0"
        plan = make_plan()
        for _ in range(args.warmup):
            f3s.run(plan, Q, K, V, scale=c["scale"], stream=stream)
        ms = []
        for _ in range(max(1, args.steps)):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            O, rec = f3s.run_trace(plan, Q, K, V, scale=c["scale"], stream=stream)
            b.record(stream)
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        r = cu_balance(rec.cpu().numpy().view(np.uint32), out["wall_clock_khz"])
        r["ms_mean"] = round(float(np.mean(ms)), 5)
        r["n_items"] = plan.info["n_items"]
        r["n_split"] = plan.info["n_split"]
        out["orders"][order] = r
        plan.close()
    if prev is None:
        os.environ.pop("F3S_NO_REORDER", None)
    else:
        os.environ["F3S_NO_REORDER"] = prev
    with make_plan() as plan:
        out["library_order"] = "window_order" if plan.info["flags"] & 1 else "heavy_first"
    print(json.dumps(out), flush=True)


def backward_bytes(info, info_t, d, heads=1):
    """Algorithmic bytes of one f3s_backward.  dQ pass over windows of A:
    Q, G and O rows of the window (delta = G.O is formed there) and their
    lse, the K and V rows of every distinct window column, dQ written and
    one (lse, delta) record per row written.  dK/dV pass over windows of
    A^T: K and V rows of the window, the Q and G rows and the (lse, delta)
    record of every distinct window column, dK and dV written.  Plan data:
    96 B per block, 16 B per item of both plans."""
    N = info["N"]
    dq = 2 * N * d + 2 * N * d + 4 * N * d + 4 * N + 4 * d * info["n_unique"] \
        + 4 * N * d + 8 * N
    dkdv = 4 * N * d + 4 * d * info_t["n_unique"] + 8 * info_t["n_unique"] + 8 * N * d
    plan_bytes = 96 * (info["n_blocks"] + info_t["n_blocks"]) + 16 * (
        info["n_items"] + info_t["n_items"])
    return heads * (dq + dkdv) + plan_bytes


def graph_timed(call, steps, dev):
    """`steps` calls captured in one HIP graph (the library launches onto
    the capturing stream; nothing in a call allocates or synchronises), one
    untimed replay, then one replay timed with events on its stream:
    returns (stream, ms per call), free of the host's per-launch latency."""
    import torch
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        call()                      # one eager call on the side stream first
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=side):
        for _ in range(steps):
            call()
    g.replay()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    cur = torch.cuda.current_stream(dev)
    a.record(cur)
    g.replay()
    b.record(cur)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    del g
    return cur, ms


def cold_mall_ms(args, call, stream, dev):
    """Mean ms of --cold-steps calls, each after writing a 1 GiB scrub buffer
    (4x the Infinity Cache), timed with events around the call only."""
    if args.cold_steps <= 0:
        return None
    import numpy as np
    import torch
    scrub = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    times = []
    for k in range(args.cold_steps):
        scrub.fill_(float(k))
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        call()
        b.record(stream)
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    del scrub
    return round(float(np.mean(times)), 5)


def copy_calibration(args, out, dev):
    """Three plain device copies of --copy-calib-mib MiB after the timed
    region: reference dispatches of known size for scaling HBM byte
    counters (FETCH_SIZE, WRITE_SIZE) taken over the same process."""
    if args.copy_calib_mib <= 0:
        return
    import torch
    n = args.copy_calib_mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    out["copy_calib_bytes"] = n * 4
    del src, dst


def bench_backward(args, c, plan, Q, K, V, stream, dev):
    import numpy as np
    import torch
    import paper_2505_08098_amd as f3s
    d, H = c["d"], args.heads
    plan_t = plan.transpose()
    transpose_ms = plan_t.info["build_ms"]
    warm = []
    for _ in range(5):         # warm: the transpose kernels' code is loaded
        pt = plan.transpose()  # build time measured by the library, as for plans
        warm.append(pt.info["build_ms"])
        pt.close()
    transpose_ms_warm = float(np.median(warm))
    rng = np.random.default_rng(np.random.SeedSequence(args.seed).spawn(4)[3])
    g32 = rng.standard_normal(tuple(Q.shape), dtype=np.float32)
    if Q.dtype == torch.bfloat16:
        from paper_2505_08098_amd import workloads as W
        G = torch.from_numpy(W.to_bf16_bits(g32)).to(dev).view(torch.int16).view(torch.bfloat16)
        O, lse = f3s.forward_typed(plan, Q, K, V, scale=c["scale"], want_lse=True,
                                   stream=stream)
    else:
        G = torch.from_numpy(g32.astype(np.float16)).to(dev)
        O, lse = f3s.forward(plan, Q, K, V, scale=c["scale"], stream=stream)
    grads = [None]

    def call():
        grads[0] = f3s.backward(plan, plan_t, Q, K, V, O, G, lse, scale=c["scale"])
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    for k in range(args.steps):
        starts[k].record(stream)
        call()
        ends[k].record(stream)
    torch.cuda.synchronize()
    per = np.array([a.elapsed_time(b) for a, b in zip(starts, ends)])
    ms_eager = float(per.mean())
    ms = ms_eager if args.no_graph else graph_timed(call, args.steps, dev)[1]
    info, info_t = plan.info, plan_t.info
    flops = 10.0 * info["nnz"] * d * H  # scores recomputed + 4 products
    nbytes = backward_bytes(info, info_t, d, H)
    out = {
        "metric": "ms per fused 3S backward call (dQ, dK, dV) and effective GFLOP/s "
                  "(10*nnz*d) at 1 MI355X",
        "value": round(flops / (ms * 1e-3) / 1e9, 2), "unit": "GFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": args.in_dtype, "data": "synthetic",
        "config": {"workload": c["name"], "N": c["N"], "nnz": info["nnz"], "d": d,
                   "windows": "aligned to the graphs" if args.segments else "16 rows",
                   "heads": H, "in_dtype": args.in_dtype, **library_switches()},
        "ms_eager_median": round(float(np.median(per)), 5),
        "ms_eager_per_call": round(ms_eager, 5),
        "timing": "eager calls, events around each" if args.no_graph else
                  "one HIP graph of the timed calls, events around its replay",
        "transpose_plan_ms": round(transpose_ms, 3),
        "transpose_plan_ms_warm": round(transpose_ms_warm, 3),
        "roofline": {"bound": "hbm", "achieved": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None, "algorithmic_bytes_per_call": nbytes,
                     "kernel": "k_bwd_dq + k_bwd_dkdv"},
        "cpu_baseline": None,
    }
    copy_calibration(args, out, dev)
    plan_t.close()
    plan.close()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--heads", type=int, default=1,
                    help="heads sharing the plan (Q, K, V of shape [N, heads, d]; "
                         "fresh seeded N(0,1) features)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="threads of the oracle baseline (default: every core of the "
                         "affinity mask, or OMP_NUM_THREADS if that is lower)")
    ap.add_argument("--cpu-rows", type=int, default=1 << 30,
                    help="rows of the workload in the oracle baseline sample")
    ap.add_argument("--backward", action="store_true",
                    help="time f3s_backward (dQ, dK, dV) instead of the forward call")
    ap.add_argument("--in-dtype", default="f16", choices=["f16", "bf16", "fp8"],
                    help="storage type of Q, K, V (bf16: f3s_forward_typed)")
    ap.add_argument("--out-dtype", default="f32", choices=["f32", "f16"],
                    help="type of O (f16: f3s_forward_typed)")
    ap.add_argument("--cold-steps", type=int, default=5,
                    help="after the timed region, calls timed one by one after a 1 GiB "
                         "scrub write each (L2 and the 256 MB Infinity Cache cold); "
                         "reported as ms_cold_mall, not in value")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager calls (events around each call, host latency "
                         "included on small workloads) instead of one HIP graph replay")
    ap.add_argument("--cu-trace", action="store_true",
                    help="per-CU busy time of one traced call, heavy-first and window-order "
                         "work lists (f3s_run_trace)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the probe kernels (streaming read/copy/write over 4 GiB "
                         "and the plan's access pattern without arithmetic)")
    ap.add_argument("--gather-sweep", action="store_true",
                    help="only the random-row gather rates by table size, row size, rows "
                         "in flight and workgroups per CU (one JSON line)")
    ap.add_argument("--d", type=int, default=None,
                    help="feature size instead of the workload's (a multiple of 32 up to "
                         "256; the paper's sweep is 64, 128, 256)")
    ap.add_argument("--segments", action="store_true",
                    help="row windows aligned to the graphs of the batch "
                         "(f3s_plan_segments; the batched-graph workload 4)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="after timing, run 3 plain device copies of this many MiB "
                         "(reference dispatches for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.backward and (args.in_dtype == "fp8" or args.out_dtype != "f32"):
        print(json.dumps({"error": "the backward pass takes fp16 or bf16 inputs and "
                                   "fp32 outputs"}))
        sys.exit(2)
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU: --gpus must be 1"}))
        sys.exit(2)
    if args.segments and args.workload != 4:
        print(json.dumps({"error": "--segments needs the batched-graph workload 4"}))
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2505_08098_amd as f3s
    from paper_2505_08098_amd import workloads as W

    f3s.load_library()
    dev = torch.device("cuda:0")
    if args.gather_sweep:
        return gather_sweep(dev)
    t0 = time.perf_counter()
    c = W.make_config(args.workload, seed=args.seed, dtype=args.in_dtype, d=args.d)
    gen_s = time.perf_counter() - t0
    N, d = c["N"], c["d"]
    H = args.heads
    if H > 1:
        rng = np.random.default_rng(np.random.SeedSequence(args.seed).spawn(3)[2])
        for key in ("Q", "K", "V"):
            x = rng.standard_normal((N, H, d), dtype=np.float32)
            c[key] = {"f16": lambda a: a.astype(np.float16), "bf16": W.to_bf16_bits,
                      "fp8": W.to_e4m3_bits}[args.in_dtype](x)
    rp = torch.from_numpy(c["row_ptr"]).to(dev)
    ci = torch.from_numpy(c["col_idx"]).to(dev)

    def to_dev(a):
        t = torch.from_numpy(a).to(dev)
        if args.in_dtype == "bf16":
            return t.view(torch.int16).view(torch.bfloat16)
        return t.view(torch.float8_e4m3fn) if args.in_dtype == "fp8" else t

    Q, K, V = to_dev(c["Q"]), to_dev(c["K"]), to_dev(c["V"])
    out_dt = torch.float32 if args.out_dtype == "f32" else torch.float16
    O = torch.empty(tuple(c["Q"].shape), dtype=out_dt, device=dev)
    typed = args.in_dtype != "f16" or args.out_dtype != "f32"

    def call():
        # on torch's current stream: the default stream, or the capturing
        # stream while a HIP graph is recorded
        if typed:
            f3s.forward_typed(plan, Q, K, V, out_dtype=out_dt, scale=c["scale"], out=O)
        else:
            f3s.run(plan, Q, K, V, scale=c["scale"], out=O)
    def make_plan():
        if args.segments:
            return f3s.Plan.segments(rp, ci, N, c["seg_ptr"])
        return f3s.Plan(rp, ci, N)
    torch.cuda.synchronize()
    plan = make_plan()
    info = plan.info
    # more builds of the same plan (median of 5): the first one in a process
    # also pays the one-time loading of the plan kernels' code
    warm = []
    for _ in range(5):
        plan2 = make_plan()
        warm.append(plan2.info["build_ms"])
        plan2.close()
    plan_ms_warm = sorted(warm)[len(warm) // 2]
    stream = torch.cuda.current_stream(dev)

    if args.backward:
        return bench_backward(args, c, plan, Q, K, V, stream, dev)
    if args.cu_trace:
        if typed or H != 1:
            print(json.dumps({"error": "--cu-trace times the one-head fp16 -> fp32 call"}))
            sys.exit(2)
        plan.close()
        return bench_cu_trace(args, c, make_plan, Q, K, V, stream, dev)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    # eager calls, events on the launch stream around each call (on the small
    # workloads these include the host's per-call latency)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        call()
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3 / args.steps
    per = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)])
    ms_eager = float(per.mean())
    if args.no_graph:
        ms = ms_eager
    else:
        stream, ms = graph_timed(call, args.steps, dev)
        # the graph's calls write the same O as the eager ones
        O_eager = O.clone()
        O.fill_(float("nan"))
        stream, _ = graph_timed(call, 1, dev)
        torch.cuda.synchronize()
        if not torch.equal(O, O_eager):
            print(json.dumps({"error": "graph replay differs from the eager call"}))
            sys.exit(1)
    cold = cold_mall_ms(args, call, stream, dev)

    flops_eff = 4.0 * info["nnz"] * d * H
    value = flops_eff / (ms * 1e-3) / 1e9
    alg_bytes = algorithmic_bytes(info, d, H, 1 if args.in_dtype == "fp8" else 2,
                                  4 if args.out_dtype == "f32" else 2)
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    issued = 1024.0 * d * H * info["n_blocks"]  # MFMA flops incl. zero padding
    traffic = traffic_from_counters(d) if H == 1 and not typed else None
    ceilings = None
    if not args.no_ceilings and args.workload == 3 and H == 1 and not typed:
        # the HBM-target workload also runs on a graph 8x larger that no cache holds
        dram = dram_check(args, stream, dev)
    else:
        dram = None
    if not args.no_ceilings:
        # the pattern probe reads what the fp16 -> fp32 single-head kernel reads
        plain = H == 1 and not typed and d in (32, 64, 128, 256)
        # (the probe writes meaningless values: it gets its own output buffer)
        ceilings = memory_ceilings(plan, Q if plain else None, K, V,
                                   torch.empty_like(O) if plain else None, d, achieved,
                                   alg_bytes, stream, dev, kv_rows=2 * N * H,
                                   row_bytes=d * (1 if args.in_dtype == "fp8" else 2))
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.in_dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{c['name']}: " + {
                1: "Erdos-Renyi N=1024, ~16 nbrs/row incl. self-loop",
                2: "Chung-Lu N=65536, exponent 2.1, mean degree 20, cap 4096, self-loops",
                3: "Chung-Lu N=1048576, exponent 2.5, mean degree 16, cap 4096, "
                   "self-loops, permuted ids",
                4: "4096 molecule-like graphs of 15-45 nodes, block-diagonal",
                5: "sequence L=32768, window 256 + 64 random keys per query",
            }[args.workload] + f", d={d}",
            "N": N, "nnz": info["nnz"], "d": d, "heads": H, "scale": c["scale"],
            "in_dtype": args.in_dtype, "out_dtype": args.out_dtype,
            "windows": "aligned to the graphs" if args.segments else "16 rows",
            "seed": args.seed,
            "parallelism": "single GPU",
            **library_switches(),
        },
        "ms_eager_per_call": round(ms_eager, 5),
        "timing": "eager calls, events around each" if args.no_graph else
                  "one HIP graph of the timed calls, events around its replay",
        "ms_eager_p10": round(float(np.percentile(per, 10)), 5),
        "ms_eager_median": round(float(np.median(per)), 5),
        "ms_eager_p90": round(float(np.percentile(per, 90)), 5),
        "wall_ms_per_step": round(wall_ms, 5),
        "ms_cold_mall": cold,
        "plan_ms": round(info["build_ms"], 3),
        "plan_ms_warm": round(plan_ms_warm, 3),
        "plan": {k: info[k] for k in ("n_windows", "n_unique", "n_blocks", "max_blocks",
                                      "piece_blocks", "n_items", "n_split", "n_pieces")},
        "plan_stats": plan_stats(plan),
        "launches_per_call": 1 + (info["n_split"] > 0),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "traffic_kind": "L2-to-fabric bytes per launch (rocprofv3 FETCH_SIZE + "
                            "WRITE_SIZE, scaled by a copy of known size): HBM reads "
                            "and writes plus Infinity-Cache hits",
            "algorithmic_bytes_per_launch": alg_bytes,
            "measured_ceilings": ceilings,
            "dram_scale_check": dram,
            "kernel": "k_fused3s<%d>" % d + (" %s->%s" % (args.in_dtype, args.out_dtype)
                                              if typed else "")
                      + (" x %d heads" % H if H > 1 else ""),
            "mfma_issued_frac": round(issued / (ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 5),
        },
        "gen_s": round(gen_s, 1),
    }
    copy_calibration(args, out, dev)
    if not args.no_cpu and (H > 1 or typed):
        # the oracle baseline is timed on the one-head fp16 -> fp32 workload
        out["cpu_baseline"] = None
    elif not args.no_cpu:
        torch.cuda.synchronize()
        O_host = O.cpu().numpy()
        base, parity = cpu_baseline(c, O_host, args.cpu_rows, args.cpu_threads)
        out["cpu_baseline"] = base
        out["parity_sample"] = parity
    else:
        out["cpu_baseline"] = None
    plan.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
