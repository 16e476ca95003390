"""Build the HIP library ``paper_2202_06009_amd/libzoadam.so`` for gfx950.

Flags that the bit-exact contract depends on: -ffp-contract=off (no FMA
contraction), default correctly rounded binary32 division and square root,
no fast-math, denormals kept.  Packed-FP32 instructions are disabled.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libzoadam.so")
SOURCES = [os.path.join(HERE, "csrc", "zo_kernels.hip"), os.path.join(HERE, "csrc", "zo_adam.cpp")]
HEADERS = [os.path.join(ROOT, "include", "zo_adam.h"), os.path.join(HERE, "csrc", "zo_internal.h")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-fPIC", "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [HIPCC] + FLAGS + ["-shared", "-o", tmp, "-x", "hip"] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed:\n{out}")
    if verbose and out.strip():
        print(out)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
