"""Build the CPU oracle (test infrastructure) into ``oracle/liboracle.so``.

Compiled with gcc at -O2, no fast-math and no FMA contraction, so that every
binary32 operation rounds exactly once, as the oracle's header requires.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False, src: str = None, out: str = None) -> str:
    """Compile `src` (default: the oracle's source) into `out` (default:
    oracle/liboracle.so); returns the library path."""
    src = src or os.path.join(HERE, "zo_oracle.c")
    out = out or LIB
    tmp = out + ".tmp"
    cmd = ["gcc", "-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fexcess-precision=standard", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
