"""Build libf3s.so (HIP, gfx950) in-tree with hipcc.

The library is the product: the binding loads it and fails loudly when it is
missing.  Built here on the CPU (hipcc cross-compiles gfx950) and shipped as
a file next to this module.
"""
import concurrent.futures
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libf3s.so")
SOURCES = ["f3s_api.hip", "plan_kernels.hip", "fused3s.hip", "fused3s_bf16.hip",
           "fused3s_fp8.hip", "fused3s_ablation.hip", "fused3s_split_row.hip",
           "backward.hip", "backward_bf16.hip", "backward_noalloc.hip", "probe.hip",
           "transpose.hip", "worklist.hip", "radix.hip"]

# The plan and transposition sources are compiled as relocatable device code
# and linked into ONE device code object: the runtime loads a code object on
# its first kernel launch, about 0.3 ms each, which a first plan build in a
# process would otherwise pay once per source file.
RDC_SOURCES = {"plan_kernels.hip", "transpose.hip", "worklist.hip", "radix.hip"}

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # keep the compiler away from packed-fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def build(verbose=False, extra_flags=()):
    """Compile every source to an object (in parallel), then link."""
    obj_dir = os.path.join(HERE, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    cmds, objs = [], []
    for src in SOURCES:
        obj = os.path.join(obj_dir, src.replace(".hip", ".o"))
        objs.append(obj)
        rdc = ["-fgpu-rdc"] if src in RDC_SOURCES else []
        cmds.append([hipcc(), *HIPCC_FLAGS, *rdc, *extra_flags, *inc, "-c",
                     os.path.join(HERE, "csrc", src), "-o", obj])
    jobs = max(1, min(len(cmds), os.cpu_count() or 1))
    with concurrent.futures.ThreadPoolExecutor(jobs) as pool:
        for cmd, res in zip(cmds, pool.map(_run, cmds, [verbose] * len(cmds))):
            if res.returncode != 0:
                raise subprocess.CalledProcessError(res.returncode, cmd)
    link = [hipcc(), "--offload-arch=gfx950", "-fgpu-rdc", "--hip-link", "-shared", "-fPIC",
            "-o", LIB + ".tmp", *objs]
    _run(link, verbose, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def _run(cmd, verbose, check=False):
    if verbose:
        print(" ".join(cmd), flush=True)
    return subprocess.run(cmd, check=check)


if __name__ == "__main__":
    print(build(verbose=True))
