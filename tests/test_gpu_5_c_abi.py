"""The C ABI from a plain C program (tests/c_abi/f3s_c_driver.c, built by
__graft_entry__.build()): plan, info, run and the error paths without Python
or torch in the process; its output against the fp64 oracle."""
import math
import os
import subprocess

import numpy as np
import pytest

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "f3s_c_driver")


def _run_driver(tmp_path, rp, ci, Q, K, V, scale):
    N, d = Q.shape
    np.ascontiguousarray(rp, dtype=np.int32).tofile(tmp_path / "row_ptr.bin")
    np.ascontiguousarray(ci, dtype=np.int32).tofile(tmp_path / "col_idx.bin")
    for name, x in (("q", Q), ("k", K), ("v", V)):
        np.ascontiguousarray(x, dtype=np.float16).tofile(tmp_path / f"{name}.bin")
    res = subprocess.run([DRIVER, str(tmp_path), str(N), str(len(ci)), str(d), repr(scale)],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    O = np.fromfile(tmp_path / "o.bin", dtype=np.float32).reshape(N, d)
    O_seg = np.fromfile(tmp_path / "o_seg.bin", dtype=np.float32).reshape(N, d)
    info = dict(line.split(" ", 1) for line in (tmp_path / "info.txt").read_text().splitlines())
    return O, O_seg, info


@pytest.mark.parametrize("case", ["workload1", "random_ragged"])
def test_c_driver_matches_oracle(gpu, oracle, tmp_path, case):
    if not os.path.exists(DRIVER):
        pytest.fail("tests/c_abi/f3s_c_driver is not built (run __graft_entry__.build())")
    if case == "workload1":
        c = W.make_config(1)
        rp, ci, Q, K, V, scale = c["row_ptr"], c["col_idx"], c["Q"], c["K"], c["V"], c["scale"]
    else:
        rng = np.random.default_rng(44)
        N, d = 333, 96
        rp, ci = W.random_csr(rng, N, max_deg=40, empty_frac=0.1, dup_frac=0.2)
        Q, K, V = (rng.standard_normal((N, d)).astype(np.float16) for _ in range(3))
        scale = 1 / math.sqrt(d)
    O, O_seg, info = _run_driver(tmp_path, rp, ci, Q, K, V, scale)
    ref = oracle.attention_f64(rp, ci, Q, K, V, scale)
    for got in (O, O_seg):
        err = got.astype(np.float64) - ref
        rel = float(np.linalg.norm(err) / np.linalg.norm(ref))
        print(f"  {case}: max_abs={np.abs(err).max():.3e} rel_fro={rel:.3e}", flush=True)
        assert np.isfinite(got).all() and np.abs(err).max() <= 5e-3 and rel <= 1e-3
    print(f"  info={info}", flush=True)
    # graphs of 7 rows: two per window (14 rows), the last window the remainder
    N = Q.shape[0]
    wr = oracle.segment_windows(np.minimum(np.arange(0, N + 7, 7), N))
    assert info["seg_windows"] == (f"{len(wr) - 1} first {wr[0]} {wr[1]} {wr[2]} "
                                   f"last {wr[-1]}")
    assert info["seg_run"] == "F3S_OK"
    assert int(info["n_windows"]) == (Q.shape[0] + 15) // 16
    assert info["bad_d"] == "F3S_ERR_UNSUPPORTED"
    assert info["null_plan"] == "F3S_ERR_INVALID_VALUE last_error F3S_ERR_INVALID_VALUE"
    assert info["misaligned_out"] == "F3S_ERR_INVALID_VALUE"
    assert info["bad_csr"] == "null F3S_ERR_INVALID_CSR"
    assert info["ws_run"] == "F3S_OK same 1"          # f3s_plan_ws: identical result
    assert info["ws_short"] == "null F3S_ERR_INVALID_VALUE"
