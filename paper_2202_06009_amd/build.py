"""Build the HIP library ``paper_2202_06009_amd/libzoadam.so`` for gfx950.

Flags that the bit-exact contract depends on: -ffp-contract=off (no FMA
contraction), default correctly rounded binary32 division and square root,
no fast-math, denormals kept.  Packed-FP32 instructions are disabled.  The
translation units are compiled in parallel, then linked.
"""
import os
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libzoadam.so")
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("zo_kernels.hip", "zo_server.hip",
                                           "zo_kernels_ua.hip", "zo_adam.cpp")]
HEADERS = [os.path.join(ROOT, "include", "zo_adam.h"), os.path.join(CSRC, "zo_internal.h"),
           os.path.join(CSRC, "zo_device.h")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-fPIC", "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _filter(text):
    return "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)


def build(verbose: bool = False) -> str:
    with tempfile.TemporaryDirectory(prefix="zoadam_build_") as tmpd:
        objs, procs = [], []
        for src in SOURCES:
            obj = os.path.join(tmpd, os.path.basename(src) + ".o")
            cmd = [HIPCC] + FLAGS + ["-c", "-x", "hip", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
        errors = []
        for src, p in procs:
            out = _filter(p.communicate()[0])
            if p.returncode != 0:
                errors.append(f"{os.path.basename(src)}:\n{out}")
            elif verbose and out.strip():
                print(out)
        if errors:
            raise RuntimeError("hipcc failed:\n" + "\n".join(errors))
        tmp = LIB + ".tmp"
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{_filter(r.stdout + r.stderr)}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
