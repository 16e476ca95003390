"""The hand-derived worked examples of tests/golden, recomputed exactly.

Independently of the oracle: one sync step of Algorithm 1 with Algorithm 2
and Equation 3 per chunk, written out over exact rationals (Python
``Fraction``) with every binary32 rounding applied explicitly (round to
nearest, ties to even; the square root correctly rounded).  Every expected
value of every fixture must come out bit for bit, so the fixtures' own
derivations are checked by a second route and the oracle's pin on them does
not rest on hand arithmetic alone.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import golden_io

F32 = np.float32


def rn32(q: Fraction) -> Fraction:
    """The binary32 value nearest to q (ties to the even significand)."""
    if q == 0:
        return Fraction(0)
    f = F32(float(q))
    best = f
    for cand in (np.nextafter(f, F32(-np.inf)), f, np.nextafter(f, F32(np.inf))):
        dc = abs(Fraction(float(cand)) - q)
        db = abs(Fraction(float(best)) - q)
        if dc < db or (dc == db and (int(cand.view(np.uint32)) & 1) == 0):
            best = cand
    return Fraction(float(best))


def sqrt32(q: Fraction) -> Fraction:
    """RN32 of the exact square root of q >= 0: the candidate c is the answer
    when q lies between the squares of the midpoints around it."""
    assert q >= 0
    if q == 0:
        return Fraction(0)
    c = F32(math.sqrt(float(q)))
    for _ in range(4):
        lo, hi = np.nextafter(c, F32(0)), np.nextafter(c, F32(np.inf))
        m_lo = (Fraction(float(lo)) + Fraction(float(c))) / 2
        m_hi = (Fraction(float(c)) + Fraction(float(hi))) / 2
        if q < m_lo * m_lo or (q == m_lo * m_lo and int(c.view(np.uint32)) & 1):
            c = lo
        elif q > m_hi * m_hi or (q == m_hi * m_hi and int(c.view(np.uint32)) & 1):
            c = hi
        else:
            return Fraction(float(c))
    raise AssertionError("square root did not settle")


def tree_abs(vals):
    """Balanced pairwise sum of |v| in index order, zero-padded to a power of
    two, each addition rounded to binary32."""
    n = 1
    while n < len(vals):
        n *= 2
    level = [abs(v) for v in vals] + [Fraction(0)] * (n - len(vals))
    while len(level) > 1:
        level = [rn32(level[i] + level[i + 1]) for i in range(0, len(level), 2)]
    return level[0]


def exact(v):
    return Fraction(float(v))


@pytest.mark.parametrize("name", golden_io.names())
def test_fixture_rederived_exactly(name):
    su, ex = golden_io.load(name)
    assert su["segments"] == [0, su["chunk"]]  # one chunk
    n, W = su["chunk"], su["world"]
    b1 = exact(F32(su["beta1"]))
    c1 = rn32(1 - b1)
    eps = exact(F32(su["eps"]))
    gamma = exact(F32(su["gamma"]))
    g = [exact(v) for v in su["g"]]
    x0 = [exact(v) for v in su["x0"]]
    v0 = [exact(v) for v in su["v0"]]
    # momentum and buffer lines (fresh momentum), from m = u = err = 0
    mn = [rn32(rn32(b1 * 0) + rn32(c1 * gj)) for gj in g]
    u = [rn32(0 + rn32(gamma * mj)) for mj in mn]
    a = [rn32(uj + 0) for uj in u]
    # worker half of Algorithm 2: Equation 3 on the chunk with error feedback
    s = rn32(tree_abs(a) / n)
    bits = [1 if aj >= 0 else 0 for aj in a]
    err = [rn32(aj - s) if b else rn32(aj + s) for aj, b in zip(a, bits)]
    own_word = sum(b << j for j, b in enumerate(bits))
    # server half: exact average of the W decompressed buffers, rounded once
    words = [own_word] + [int(w) for w in su["peer_words"]]
    scales = [s] + [exact(v) for v in su["peer_scales"]]
    avg = []
    for j in range(n):
        tot = sum((sc if (wd >> j) & 1 else -sc) for wd, sc in zip(words, scales))
        avg.append(rn32(tot / W))
    bsrv = [rn32(aj + 0) for aj in avg]
    sbar = rn32(tree_abs(bsrv) / n)
    sbits = [1 if bj >= 0 else 0 for bj in bsrv]
    serr = [rn32(bj - sbar) if sb else rn32(bj + sbar) for bj, sb in zip(bsrv, sbits)]
    srv_word = sum(b << j for j, b in enumerate(sbits))
    # sync lines of Algorithm 1: Gamma = gamma; m = ubar / Gamma; x from the anchor
    Gam = rn32(0 + gamma)
    ubar = [sbar if sb else -sbar for sb in sbits]
    m = [rn32(uj / Gam) for uj in ubar]
    x = [rn32(x0j - rn32(uj / sqrt32(rn32(vj + eps)))) for x0j, uj, vj in zip(x0, ubar, v0)]

    def same(got, key):
        want = [exact(v) for v in ex[key]]
        assert got == want, (key, [float(v) for v in got], [float(v) for v in want])

    same(a, "a")
    same([s], "own_scales")
    same(err, "err")
    same(avg, "avg")
    same([sbar], "srv_scales")
    same(serr, "srv_err")
    same(ubar, "ubar")
    same(m, "m")
    same(x, "x")
    assert [own_word] == [int(w) for w in ex["own_words"]]
    assert [srv_word] == [int(w) for w in ex["srv_words"]]


def test_exact_helpers():
    """rn32 and sqrt32 against cases with known answers."""
    assert rn32(Fraction(1) + Fraction(1, 2 ** 24)) == 1          # tie -> even
    assert rn32(Fraction(1) + Fraction(3, 2 ** 24)) == 1 + Fraction(1, 2 ** 22)  # tie -> even
    assert rn32(Fraction(1, 3)) == exact(F32(1) / F32(3))
    assert sqrt32(Fraction(1, 4)) == Fraction(1, 2)
    assert sqrt32(Fraction(2)) == exact(np.sqrt(F32(2)))
    r = np.random.default_rng(0)
    for v in r.uniform(1e-12, 10, 300).astype(F32):
        assert sqrt32(exact(v)) == exact(np.sqrt(v))
