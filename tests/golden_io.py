"""Read the hand-derived worked examples under tests/golden/.

A fixture is plain text: ``#`` comments, a ``[setup]`` and an ``[expect]``
section of ``key: values`` lines.  A value is a decimal number, a binary32
bit pattern ``f32:0x...`` or, for keys ending in ``_words``, a packed 64-bit
word ``0x...``.
"""
import os
import struct

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _value(tok):
    if tok.startswith("f32:"):
        return struct.unpack("<f", struct.pack("<I", int(tok[4:], 16)))[0]
    return float(tok)


def load(name):
    """(setup, expect) of fixture `name`: dicts of numpy arrays (float32, or
    uint64 for packed words; setup scalars as Python numbers)."""
    sections = {}
    cur = None
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            if line.startswith("[") and line.endswith("]"):
                cur = sections.setdefault(line[1:-1], {})
                continue
            key, _, rest = line.partition(":")
            toks = rest.split()
            if key.endswith("_words"):
                cur[key.strip()] = np.array([int(t, 16) for t in toks], np.uint64)
            else:
                cur[key.strip()] = np.array([_value(t) for t in toks], np.float32)
    setup, expect = sections["setup"], sections["expect"]
    for k in ("chunk", "world"):
        setup[k] = int(setup[k][0])
    for k in ("beta1", "eps", "gamma"):
        setup[k] = float(setup[k][0])
    setup["segments"] = [int(v) for v in setup["segments"]]
    return setup, expect


def names():
    return sorted(f for f in os.listdir(GOLDEN) if f.endswith(".txt"))
