"""The C-ABI library loads and exports every function include/f3s.h declares
(CPU only: no compute call is made)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(ROOT, "paper_2505_08098_amd", "libf3s.so")


def declared_functions():
    """Every function declared by a header under include/."""
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if h.endswith(".h"):
            text = re.sub(r"/\*.*?\*/", "", open(os.path.join(INCLUDE, h)).read(), flags=re.S)
            names |= set(re.findall(r"\b(f3s_[a-z_]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libf3s.so is not built (run __graft_entry__.build())")
    import torch  # noqa: F401  (same load order as the binding)
    return ctypes.CDLL(LIB)


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("f3s_plan", "f3s_plan_ws", "f3s_plan_workspace_bytes", "f3s_plan_transpose_ws",
              "f3s_plan_transpose_workspace_bytes", "f3s_run",
              "f3s_run_mh", "f3s_forward", "f3s_plan_transpose",
              "f3s_backward", "f3s_backward_typed", "f3s_destroy", "f3s_plan_info",
              "f3s_plan_export", "f3s_last_error", "f3s_status_string",
              "f3s_backward_noalloc", "f3s_backward_noalloc_max_records",
              "f3s_probe_read", "f3s_probe_copy", "f3s_probe_write", "f3s_probe_gather"):
        assert n in names


def test_workspace_bytes_rejects_negative_sizes(lib):
    lib.f3s_plan_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int64]
    lib.f3s_plan_workspace_bytes.restype = ctypes.c_size_t
    assert lib.f3s_plan_workspace_bytes(-1, 10) == 0
    assert lib.f3s_plan_workspace_bytes(10, -1) == 0
    # host-only: linear in the entries (column staging, 4 + 2 bytes per entry)
    a = lib.f3s_plan_workspace_bytes(1 << 20, 10_000_000)
    b = lib.f3s_plan_workspace_bytes(1 << 20, 20_000_000)
    assert 6 * 10_000_000 <= b - a <= 6 * 10_000_000 + 4096
    assert lib.f3s_plan_workspace_bytes(0, 0) > 0


def test_every_declared_symbol_is_exported(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_exports_are_c_symbols():
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if " T " in line)
    for n in declared_functions():
        assert n in exported, n


def test_status_strings_are_host_only(lib):
    lib.f3s_status_string.restype = ctypes.c_char_p
    lib.f3s_status_string.argtypes = [ctypes.c_int]
    assert lib.f3s_status_string(0) == b"F3S_OK"
    assert lib.f3s_status_string(2) == b"F3S_ERR_INVALID_CSR"
    assert lib.f3s_status_string(6) == b"F3S_ERR_TOO_LARGE"
    assert lib.f3s_status_string(99) == b"F3S_ERR_UNKNOWN"
    lib.f3s_last_error.restype = ctypes.c_int
    assert lib.f3s_last_error() == 0


def test_null_handles_are_rejected_without_a_device(lib):
    lib.f3s_destroy.argtypes = [ctypes.c_void_p]
    lib.f3s_destroy(None)  # no-op
    lib.f3s_plan_info.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    lib.f3s_plan_info.restype = ctypes.c_int
    assert lib.f3s_plan_info(None, None) == 1
    lib.f3s_run.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int32, ctypes.c_float,
                                                    ctypes.c_void_p]
    lib.f3s_run.restype = ctypes.c_int
    assert lib.f3s_run(None, None, None, None, None, 64, 1.0, None) == 1


def test_plain_c_program_builds_against_the_header():
    """A C11 translation unit including only include/f3s.h (and the HIP
    runtime API it names) compiles and links against libf3s.so (the GPU test
    runs the program)."""
    import sys
    sys.path.insert(0, ROOT)
    import __graft_entry__ as ge
    path = ge.build_c_driver()
    out = subprocess.run(["ldd", path], capture_output=True, text=True, check=True).stdout
    assert "libf3s.so" in out
