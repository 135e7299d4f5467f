"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU needed): every source is compiled with the sanitizers on
its host side (device code unchanged), linked into a separate library in a
temporary directory, and driven by tests/sanitize/host_abi_sanitize.c
through the C ABI (argument checks, scratch sizing over the int32 range,
status strings, plan builds failing for want of a device).  The run aborts
on any memory error, leak in the library or undefined behaviour."""
import concurrent.futures
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer"]


def test_library_host_code_under_asan_and_ubsan(tmp_path):
    import sys
    sys.path.insert(0, ROOT)
    from paper_2505_08098_amd import build as lib_build
    hipcc = lib_build.hipcc()
    clang = os.path.join(ROCM, "llvm", "bin", "clang")
    rt = glob.glob(os.path.join(ROCM, "llvm", "lib", "clang", "*", "lib", "linux",
                                "libclang_rt.asan-x86_64.so"))
    if not os.path.exists(clang) or not rt or shutil.which(hipcc) is None and \
            not os.path.exists(hipcc):
        pytest.skip("ROCm clang with the ASan runtime is not available")
    csrc = os.path.join(ROOT, "paper_2505_08098_amd", "csrc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", csrc]
    # each translation unit with its own device code object (no relocatable
    # device code), so a plain host link of the objects works
    cmds = [[hipcc, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *SAN, *inc,
             "-c", os.path.join(csrc, s), "-o", str(tmp_path / s.replace(".hip", ".o"))]
            for s in lib_build.SOURCES]
    with concurrent.futures.ThreadPoolExecutor(min(8, len(cmds))) as pool:
        for cmd, res in zip(cmds, pool.map(
                lambda c: subprocess.run(c, capture_output=True, text=True), cmds)):
            assert res.returncode == 0, res.stderr[-2000:]
    lib = tmp_path / "libf3s_san.so"
    objs = [c[-1] for c in cmds]
    subprocess.run([os.path.join(ROCM, "llvm", "bin", "clang++"), "-shared", "-fPIC",
                    "-fsanitize=address,undefined", "-shared-libasan", "-o", str(lib), *objs,
                    "-L", os.path.join(ROCM, "lib"), "-lamdhip64"], check=True)
    exe = tmp_path / "host_abi_sanitize"
    rtdir = os.path.dirname(rt[0])
    subprocess.run([clang, "-std=c11", "-g", "-fsanitize=address,undefined", "-shared-libasan",
                    "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", *inc, "-I",
                    os.path.join(ROCM, "include"),
                    os.path.join(ROOT, "tests", "sanitize", "host_abi_sanitize.c"), "-o",
                    str(exe), "-L", str(tmp_path), "-lf3s_san", "-L",
                    os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + str(tmp_path),
                    "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-Wl,-rpath," + rtdir],
                   check=True)
    # leaks inside the (uninstrumented) HIP runtime are not the library's
    supp = tmp_path / "lsan.supp"
    supp.write_text("leak:libamdhip64\nleak:libhsa-runtime64\nleak:libamd_comgr\n"
                    "leak:libdrm\nleak:libnuma\n")
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               LSAN_OPTIONS=f"suppressions={supp}",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               HIP_VISIBLE_DEVICES="-1")
    res = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr[-4000:]
    assert res.stdout.strip() == "ok"
