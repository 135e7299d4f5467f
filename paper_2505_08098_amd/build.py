"""Build libf3s.so (HIP, gfx950) in-tree with hipcc.

The library is the product: the binding loads it and fails loudly when it is
missing.  Built here on the CPU (hipcc cross-compiles gfx950) and shipped as
a file next to this module.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libf3s.so")
SOURCES = ["f3s_api.hip", "plan_kernels.hip", "fused3s.hip", "backward.hip"]

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
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
    srcs = [os.path.join(HERE, "csrc", s) for s in SOURCES]
    cmd = [hipcc(), *HIPCC_FLAGS, *extra_flags,
           "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(HERE, "csrc"),
           "-o", LIB + ".tmp", *srcs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
