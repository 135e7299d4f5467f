"""bench.py's host-side parts: the one-GPU refusal, the algorithmic-bytes
formula of the forward roofline, and the source hash that decides whether
the committed counter measurements still describe the kernel.  CPU only."""
import json
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_device_use():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, HIP_VISIBLE_DEVICES=""))
    assert r.returncode == 2
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    assert "one GPU" in json.loads(lines[0])["error"]


@pytest.mark.parametrize("d,heads", [(64, 1), (128, 3)])
def test_algorithmic_bytes_is_the_sum_over_windows(d, heads):
    # per 16-row window w with u_w distinct columns and b_w = ceil(u_w / 16)
    # blocks: Q rows 16*d*2, K and V rows 2*2*d*u_w, O rows 16*d*4 (per head),
    # 64 B of column ids and 32 B of bitmap per block, 16 B per work item
    rng = np.random.default_rng(7)
    T = 37
    N = 16 * T
    u = []
    for w in range(T):
        deg = rng.integers(0, 40, size=16)
        cols = np.concatenate([rng.integers(0, N, size=k) for k in deg])
        u.append(len(np.unique(cols)))
    u = np.array(u, dtype=np.int64)
    b = (u + 15) // 16
    per_window = heads * (16 * d * 2 + 4 * d * u + 16 * d * 4) + 96 * b + 16
    info = {"N": N, "n_unique": int(u.sum()), "n_blocks": int(b.sum()), "n_items": T}
    assert bench.algorithmic_bytes(info, d, heads) == int(per_window.sum())
    # fp8 in, fp16 out: 1-byte K/V/Q elements, 2-byte O elements
    per_window8 = heads * (16 * d * 1 + 2 * d * u + 16 * d * 2) + 96 * b + 16
    assert bench.algorithmic_bytes(info, d, heads, in_size=1, out_size=2) == \
        int(per_window8.sum())


@pytest.mark.parametrize("d,heads", [(64, 1), (128, 2)])
def test_backward_bytes_is_the_sum_over_both_passes(d, heads):
    # dQ pass, per 16-row window of A with u_w distinct columns (per head):
    # Q and G rows 2 * 16*d*2, O rows 16*d*4 (delta = G.O), lse 16*4, K and V
    # rows 2*2*d*u_w, dQ written 16*d*4, one 8-byte (lse, delta) record per
    # row written.  dK/dV pass, per window of A^T with v_w distinct columns:
    # K and V rows 2 * 16*d*2, Q and G rows 2*2*d*v_w plus an 8-byte record
    # per column, dK and dV written 2 * 16*d*4.  Plan data of both plans:
    # 96 B per block and 16 B per work item.
    rng = np.random.default_rng(9)
    T = 23
    N = 16 * T
    u = rng.integers(1, 200, size=T).astype(np.int64)
    v = rng.integers(1, 200, size=T).astype(np.int64)
    bu, bv = (u + 15) // 16, (v + 15) // 16
    per_w_dq = (16 * d * 2 * 2 + 16 * d * 4 + 16 * 4 + 4 * d * u + 16 * d * 4 + 16 * 8)
    per_w_dkdv = (16 * d * 2 * 2 + 4 * d * v + 8 * v + 2 * 16 * d * 4)
    want = heads * int(per_w_dq.sum() + per_w_dkdv.sum()) + \
        96 * int(bu.sum() + bv.sum()) + 16 * 2 * T
    info = {"N": N, "n_unique": int(u.sum()), "n_blocks": int(bu.sum()), "n_items": T}
    info_t = {"N": N, "n_unique": int(v.sum()), "n_blocks": int(bv.sum()), "n_items": T}
    assert bench.backward_bytes(info, info_t, d, heads) == want


def _copy_sources(tmp_path):
    for p in bench.KERNEL_SOURCES:
        dst = tmp_path / os.path.relpath(p, ROOT)
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(p, dst)
    return tmp_path


def test_source_hash_ignores_comments_and_whitespace(tmp_path):
    root = _copy_sources(tmp_path)
    base = bench.kernel_source_hash(str(root))
    assert base == bench.kernel_source_hash()
    k = root / "paper_2505_08098_amd" / "csrc" / "fused3s_kernel.h"
    text = k.read_text()
    k.write_text("// a comment line\n/* and a\n block */\n" + text.replace("\n", "\n\n", 5))
    assert bench.kernel_source_hash(str(root)) == base
    # the plan part of the internal header does not count either
    h = root / "paper_2505_08098_amd" / "csrc" / "f3s_internal.h"
    h.write_text(h.read_text() + "\nint unrelated_plan_helper(int);\n")
    assert bench.kernel_source_hash(str(root)) == base


def test_source_hash_changes_with_the_code(tmp_path):
    root = _copy_sources(tmp_path)
    base = bench.kernel_source_hash(str(root))
    k = root / "paper_2505_08098_amd" / "csrc" / "kernel_common.h"
    text = k.read_text()
    assert "__forceinline__" in text
    k.write_text(text.replace("__forceinline__", "inline", 1))
    assert bench.kernel_source_hash(str(root)) != base


def test_counters_are_used_only_for_their_feature_size():
    with open(bench.COUNTERS_FILE) as f:
        rec = json.load(f)
    other_d = 64 if rec.get("d") != 64 else 128
    assert bench.traffic_from_counters(other_d) is None
    got = bench.traffic_from_counters(rec.get("d"))
    if rec.get("kernel_source_hash") == bench.kernel_source_hash():
        assert got == rec.get("hbm_bytes_per_launch")
    else:
        assert got is None


def test_cu_balance_unions_intervals_per_cu():
    """bench.cu_balance: busy = union of each CU's workgroup intervals, end =
    its last end, from the first start (hand-worked records, 100 MHz)."""
    import numpy as np
    import bench
    rec = np.zeros((5, 8), dtype=np.uint32)
    rec[:, 0] = [100, 150, 100, 400, 450]          # starts (ticks)
    rec[:, 2] = [200, 300, 300, 500, 480]          # ends
    rec[:, 4] = [1 << 8, 1 << 8, 2 << 8, 2 << 8, 2 << 8]   # CU ids 1 and 2
    rec[:, 5] = [0, 0, 0, 0, 0]
    r = bench.cu_balance(rec, 100_000)             # 1 tick = 0.01 us
    assert r["cus"] == 2 and r["workgroups"] == 5
    assert r["span_us"] == 4.0
    assert r["busy_us"] == {"min": 2.0, "mean": 2.5, "max": 3.0}
    assert r["end_us"] == {"min": 2.0, "mean": 3.0, "max": 4.0}
    # the same CU id on another die is another CU
    rec[4, 5] = 3
    assert bench.cu_balance(rec, 100_000)["cus"] == 3


def test_library_switches_are_reported(monkeypatch):
    """A bench line measured under one of the library's F3S_* switches names
    it in its config; without any, the config carries no switches entry."""
    for k in [k for k in os.environ if k.startswith("F3S_")]:
        monkeypatch.delenv(k)
    assert bench.library_switches() == {}
    monkeypatch.setenv("F3S_SPLIT_ROW", "1")
    monkeypatch.setenv("F3S_PIECE_BLOCKS", "8")
    assert bench.library_switches() == {
        "switches": {"F3S_PIECE_BLOCKS": "8", "F3S_SPLIT_ROW": "1"}}
