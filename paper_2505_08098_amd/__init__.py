"""Fused sparse attention (3S) on AMD MI355X: Python side of libf3s.so.

    import paper_2505_08098_amd as f3s
    plan = f3s.Plan(row_ptr, col_idx, N)          # device int32 CSR
    O = f3s.run(plan, Q, K, V, scale=1/d**0.5)    # fp16 in, fp32 out

The compute path is the HIP library only (see ``binding``); ``workloads``
holds the seeded synthetic inputs.
"""
from .binding import (F3SError, Plan, PlanInfo, backward, forward,  # noqa: F401
                      forward_typed, load_library, probe_gather, probe_rows, probe_stream,
                      run, run_raw, run_trace, status_string, wall_clock_khz)
