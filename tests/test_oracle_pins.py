"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test ties one part of the oracle to something other than itself:
worked examples derived by hand from Equation 3 and Algorithm 2 (the
fixtures under tests/golden, one with a non-dyadic average), closed forms
and invariants of the compressor (contraction identities, error-feedback
telescoping), brute-force bit packing, an exact rational average, the
special case in which 0/1 Adam reduces to Adam (Equation 2, computed by an
independent binary64 implementation), and the consensus of workers after a
synchronisation.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import golden_io
import oracle as orc
from oracle.brute_adam import adam_fp64

F32 = np.float32
U = 2.0 ** -24  # unit roundoff of binary32


def rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------------------
# Worked examples (Equation 3 + Algorithm 2 + the sync lines of Algorithm 1),
# derived by hand: the fixtures under tests/golden, each with its derivation.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", golden_io.names())
def test_worked_examples(name):
    """The hand-derived examples of tests/golden (Equation 3, Algorithm 2,
    Algorithm 1's sync lines), part by part and as one step from g."""
    su, ex = golden_io.load(name)
    lay = orc.Layout.from_segments(su["segments"], su["chunk"])
    assert lay.nchunks == 1
    eq = np.testing.assert_array_equal
    # worker compress on a with zero error
    delta = np.zeros(lay.n, F32)
    words, scales = orc.ef_compress(lay, ex["a"], delta)
    eq(words, ex["own_words"])
    eq(scales, ex["own_scales"])
    eq(delta, ex["err"])
    # server over [own, peers]
    words_w = np.concatenate([words[None, :], su["peer_words"][:, None]], axis=0)
    scales_w = np.concatenate([scales[None, :], su["peer_scales"][:, None]], axis=0)
    assert words_w.shape[0] == su["world"]
    srv_err = np.zeros(lay.n, F32)
    sw, ss, avg = orc.server(lay, words_w, scales_w, srv_err, want_avg=True)
    eq(avg, ex["avg"])
    eq(sw, ex["srv_words"])
    eq(ss, ex["srv_scales"])
    eq(srv_err, ex["srv_err"])
    eq(orc.decompress(lay, sw, ss), ex["ubar"])
    # the whole step from the gradient
    w = orc.Worker(lay, su["x0"], beta1=su["beta1"], eps=su["eps"])
    w.v[:] = su["v0"]
    out = w.step(su["gamma"], su["g"], sync=True, var=False,
                 peer_words=su["peer_words"][:, None], peer_scales=su["peer_scales"][:, None])
    eq(out["own_words"], ex["own_words"])
    eq(out["srv_words"], ex["srv_words"])
    eq(out["srv_scales"], ex["srv_scales"])
    eq(w.err, ex["err"])
    eq(w.srv_err, ex["srv_err"])
    eq(w.m, ex["m"])
    eq(w.x, ex["x"])
    eq(w.anchor, w.x)
    eq(w.v, su["v0"])
    assert not w.u.any() and w.gamma_sum == 0


# ---------------------------------------------------------------------------
# The L1 tree
# ---------------------------------------------------------------------------

def test_tree_is_pairwise_in_index_order():
    big = float(2 ** 24)
    # pairwise: (1 + 1) + (1 + 2^24) = 2 + 2^24 (1 + 2^24 ties to even 2^24)
    assert orc.tree_abs_sum(np.array([1, 1, 1, big], F32)) == F32(big + 2)
    # left to right would give ((1 + 1) + 1) + 2^24 = 2^24 + 3 -> 2^24 + 4
    assert F32(F32(F32(1 + 1) + 1) + F32(big)) == F32(big + 4)
    # [2^24, 1, 1, 1]: (2^24 + 1) + (1 + 1) = 2^24 + 2
    assert orc.tree_abs_sum(np.array([big, 1, 1, 1], F32)) == F32(big + 2)
    # absolute values are summed
    assert orc.tree_abs_sum(np.array([-3, 1, -0.0, -4], F32)) == F32(8)
    # zero padding: n = 3 is the tree over [a0, a1, a2, 0]
    assert orc.tree_abs_sum(np.array([big, 1, 1], F32)) == F32(big)   # (2^24+1)+(1+0)
    assert orc.tree_abs_sum(np.array([1, 1, big], F32)) == F32(big + 2)


@pytest.mark.parametrize("n", [1, 2, 3, 7, 64, 100, 1000, 4096, 16383])
def test_tree_error_bound(n):
    """Pairwise summation: |T - sum| <= ceil(log2 n) * u * sum |a| (Higham)."""
    a = rng(n).standard_normal(n).astype(F32) * F32(1e-3)
    exact = math.fsum(abs(float(v)) for v in a)
    t = float(orc.tree_abs_sum(a))
    k = max(1, math.ceil(math.log2(n))) if n > 1 else 0
    assert abs(t - exact) <= k * U * exact * 1.0001 + 1e-45


# ---------------------------------------------------------------------------
# Equation 3 on a chunk: closed forms and invariants
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 2, 5, 64, 65, 1000, 2048])
def test_compressor_identities(n):
    r = rng(100 + n)
    a = (r.standard_normal(n) * 1e-3).astype(F32)
    s, bits = orc.compress_chunk(a)
    sigma = np.where(bits == 1, 1.0, -1.0)
    np.testing.assert_array_equal(bits, (a >= 0).astype(np.uint8))
    l1 = math.fsum(abs(float(v)) for v in a)
    # s = |a|_1 / n up to the tree's and the division's rounding
    k = max(1, math.ceil(math.log2(n))) if n > 1 else 0
    assert abs(float(s) - l1 / n) <= (k + 1) * U * (l1 / n) * 1.0001
    # the new error delta' = a - s sigma, each entry rounded once
    lay = orc.Layout.from_lengths([n])
    delta = np.zeros(n, F32)
    orc.ef_compress(lay, a, delta)
    ad = a.astype(np.float64)
    dd = delta.astype(np.float64)
    # C[a] + delta' = a up to one rounding of delta'
    assert np.all(np.abs(sigma * float(s) + dd - ad) <= U * np.abs(dd) + 1e-45)
    # <sigma, delta'> = |a|_1 - n s = 0 up to rounding
    assert abs(math.fsum(sigma * dd)) <= (k + 4) * U * l1
    # |delta'|^2 = |a|^2 - |a|_1^2 / n  (the contraction of Assumption 6)
    lhs = math.fsum(dd * dd)
    rhs = math.fsum(ad * ad) - l1 * l1 / n
    assert abs(lhs - rhs) <= 8 * (k + 4) * U * math.fsum(ad * ad) + 1e-30
    if n == 1:
        assert delta[0] == 0


@pytest.mark.parametrize("n", [1, 3, 64, 100, 2048])
def test_constant_magnitude_is_lossless(n):
    r = rng(7 * n)
    c = F32(2.0 ** -13)
    a = np.where(r.random(n) < 0.5, -c, c).astype(F32)
    lay = orc.Layout.from_lengths([n])
    delta = np.zeros(n, F32)
    words, scales = orc.ef_compress(lay, a, delta)
    assert scales[0] == c
    assert not delta.any()
    np.testing.assert_array_equal(orc.decompress(lay, words, scales), a)


def test_sign_of_zero_is_plus():
    s, bits = orc.compress_chunk(np.array([0.0, -0.0, -1.0, 1.0], F32))
    assert list(bits) == [1, 1, 0, 1]
    assert s == F32(0.5)


def test_single_chunk_is_equation3():
    """C = d on one segment: one magnitude |a|_1/d for the whole vector."""
    d = 3000
    a = (rng(5).standard_normal(d) * 0.01).astype(F32)
    lay = orc.Layout.from_segments([0, d], d)
    assert lay.nchunks == 1
    delta = np.zeros(d, F32)
    words, scales = orc.ef_compress(lay, a, delta)
    l1 = math.fsum(abs(float(v)) for v in a)
    assert abs(float(scales[0]) - l1 / d) <= 13 * U * l1 / d
    out = orc.decompress(lay, words, scales)
    np.testing.assert_array_equal(np.sign(out), np.where(a >= 0, 1, -1))


def test_error_feedback_telescopes():
    """sum_k C[z_k + delta_k] = sum_k z_k - delta_K with delta_0 = 0."""
    lay = orc.Layout.from_segments([0, 500, 1300], 256)
    r = rng(11)
    delta = np.zeros(lay.n, F32)
    sent = np.zeros(lay.n)
    total = np.zeros(lay.n)
    bound = np.zeros(lay.n)
    for _ in range(12):
        z = (r.standard_normal(lay.n) * 1e-2).astype(F32)
        before = delta.astype(np.float64).copy()
        words, scales = orc.ef_compress(lay, z, delta)
        c = orc.decompress(lay, words, scales).astype(np.float64)
        sent += c
        total += z
        # roundings of a = z + delta and of delta' = a -+ s
        bound += U * (np.abs(z.astype(np.float64) + before) + np.abs(delta.astype(np.float64)))
    resid = sent - (total - delta.astype(np.float64))
    assert np.all(np.abs(resid) <= 2 * bound + 1e-30)


# ---------------------------------------------------------------------------
# Packing
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 31, 32, 63, 64, 65, 128, 200])
def test_pack_layout_brute_force(n):
    bits = (rng(n).random(n) < 0.5).astype(np.uint8)
    words = orc.pack_chunk(bits)
    assert len(words) == (n + 63) // 64
    expect = [0] * len(words)
    for j in range(n):
        if bits[j]:
            expect[j // 64] |= 1 << (j % 64)
    assert [int(w) for w in words] == expect
    np.testing.assert_array_equal(orc.unpack_chunk(words, n), bits)
    if n % 64:
        assert int(words[-1]) >> (n % 64) == 0  # pad bits are zero


def test_pack_bit_positions():
    bits = np.zeros(130, np.uint8)
    bits[0] = bits[63] = bits[64] = bits[129] = 1
    w = orc.pack_chunk(bits)
    assert [int(x) for x in w] == [1 | (1 << 63), 1, 2]


def test_chunk_table_never_crosses_segments():
    seg = [0, 100, 100 + 4096, 100 + 4096 + 8, 20000]
    lay = orc.Layout.from_segments(seg, 1024)
    ends = set(seg[1:])
    pos = 0
    words = 0
    for c in range(lay.nchunks):
        assert lay.cstart[c] == pos and 1 <= lay.clen[c] <= 1024
        assert lay.cword[c] == words
        pos += lay.clen[c]
        words += (lay.clen[c] + 63) // 64
        # a chunk ends at a segment end or after exactly 1024 elements
        assert pos in ends or lay.clen[c] == 1024
        assert not any(lay.cstart[c] < e < pos for e in ends)
    assert pos == seg[-1] and lay.nwords == words
    assert lay.nchunks == 1 + 4 + 1 + 16  # 100 | 4096 | 8 | 15796


# ---------------------------------------------------------------------------
# Server average: exact rational reference
# ---------------------------------------------------------------------------

def rn32(q: Fraction) -> np.float32:
    """Round a rational to the nearest binary32, ties to even (exact)."""
    f = np.float32(float(q))
    best = f
    for cand in (np.nextafter(f, F32(-np.inf)), f, np.nextafter(f, F32(np.inf))):
        dc, db = abs(Fraction(float(cand)) - q), abs(Fraction(float(best)) - q)
        if dc < db or (dc == db and (cand.view(np.uint32) & 1) == 0):
            best = cand
    return best


@pytest.mark.parametrize("W", [1, 2, 3, 4, 5, 8, 16])
def test_server_average_is_exact_rounding(W):
    n = 200
    r = rng(1000 + W)
    lay = orc.Layout.from_lengths([n])
    words_w = np.stack([orc.pack_chunk((r.random(n) < 0.5).astype(np.uint8)) for _ in range(W)])
    scales_w = (r.uniform(0.5, 1.5, size=(W, 1)) * 3e-5).astype(F32)
    srv_err = np.zeros(n, F32)
    _, _, avg = orc.server(lay, words_w, scales_w, srv_err, want_avg=True)
    for j in range(n):
        tot = Fraction(0)
        for w in range(W):
            b = (int(words_w[w, j // 64]) >> (j % 64)) & 1
            tot += Fraction(float(scales_w[w, 0])) * (1 if b else -1)
        assert avg[j] == rn32(tot / W), (j, W)


def test_server_single_worker_and_equal_signs():
    n = 128
    r = rng(3)
    lay = orc.Layout.from_lengths([n])
    bits = (r.random(n) < 0.5).astype(np.uint8)
    own = orc.pack_chunk(bits)
    s = F32(3.0e-6)
    # W = 1: the average is the own decompressed value; recompressing a
    # constant-magnitude chunk of power-of-two length loses nothing
    srv_err = np.zeros(n, F32)
    sw, ss, avg = orc.server(lay, own[None], np.array([[s]], F32), srv_err, want_avg=True)
    np.testing.assert_array_equal(avg, np.where(bits == 1, s, -s).astype(F32))
    assert ss[0] == s and int(sw[0]) == int(own[0]) and int(sw[1]) == int(own[1])
    assert not srv_err.any()
    # all workers agree on the signs: avg = +-(sum S_w) / W
    W = 4
    sc = np.array([[1e-6], [2e-6], [3e-6], [1.5e-6]], F32)
    _, _, avg = orc.server(lay, np.repeat(own[None], W, 0), sc, np.zeros(n, F32), want_avg=True)
    mag = rn32(sum(Fraction(float(v)) for v in sc[:, 0]) / W)
    np.testing.assert_array_equal(avg, np.where(bits == 1, mag, -mag).astype(F32))


@pytest.mark.parametrize("W", [2, 3, 5, 7, 16])
def test_dense_average_is_exact_rounding(W):
    """The compression-off average of W dense buffers (worker-major [W][n]):
    the exact rational mean of the W values at each position, rounded once to
    binary32.  Worker values differ in sign, magnitude and position, so a
    wrong worker or element index changes the result."""
    n = 300
    r = rng(2000 + W)
    z = (r.standard_normal((W, n)) * r.choice([1e-8, 3e-7, 2e-6], size=(W, 1))).astype(F32)
    got = orc.dense_average(z)
    for j in range(n):
        want = rn32(sum(Fraction(float(z[w, j])) for w in range(W)) / W)
        assert got[j] == want, (j, W)
    # the same buffers in another worker order average to the same values
    np.testing.assert_array_equal(orc.dense_average(z[::-1].copy()), got)
    # one worker: the buffer itself
    np.testing.assert_array_equal(orc.dense_average(z[:1].copy()), z[0])


def test_dense_average_flags_inexact_sum():
    z = np.array([[1.0, 1.0], [2.0 ** -60, 0.0]], F32)
    with pytest.raises(orc.OracleError):
        orc.dense_average(z)


@pytest.mark.parametrize("W", [3, 5, 6, 7, 9, 11, 100, 127, 65535])
def test_binary64_quotient_by_w_rounds_once(W):
    """Both sides form the average as (float)(S / W) from the exact binary64
    sum S: two roundings.  For a binary64 S and an integer W the result is
    still RN32(S / W) -- if RN64(S / W) landed on a binary32 midpoint M while
    S / W != M, then |S - W M| >= ulp64(S) and |S / W - M| < ulp64(M) / 2
    would force 2^(e(S) - e(M) + 1) < W, while e(S) >= e(M) + floor(log2 W)
    -- checked here on sums right next to W times binary32 midpoints, where a
    double rounding would show."""
    r = rng(3000 + W)
    for _ in range(400):
        f = F32(r.uniform(0.5, 1.0) * 2.0 ** int(r.integers(-40, 40)))
        if r.random() < 0.5:
            f = -f
        mid = (Fraction(float(f)) + Fraction(float(np.nextafter(f, F32(np.inf))))) / 2
        s0 = float(mid * W)
        for k in range(-3, 4):
            s = s0
            for _ in range(abs(k)):
                s = float(np.nextafter(s, np.inf if k > 0 else -np.inf))
            got = F32(np.float64(s) / np.float64(W))
            assert got == rn32(Fraction(s) / W), (W, float(f), k)


def test_server_flags_inexact_sum():
    lay = orc.Layout.from_lengths([64])
    words_w = np.array([[0], [0xFFFFFFFFFFFFFFFF]], np.uint64)
    scales_w = np.array([[1.0], [2.0 ** -60]], F32)
    with pytest.raises(orc.OracleError):
        orc.server(lay, words_w, scales_w, np.zeros(64, F32))


def test_server_error_feedback_telescopes():
    """Server half: sum_k sbar_k sigma_k = sum_k avg_k - serr_K."""
    lay = orc.Layout.from_segments([0, 300, 812], 128)
    r = rng(21)
    W = 4
    srv_err = np.zeros(lay.n, F32)
    sent = np.zeros(lay.n)
    total = np.zeros(lay.n)
    bound = np.zeros(lay.n)
    for _ in range(8):
        words_w = r.integers(0, 2 ** 63, size=(W, lay.nwords), dtype=np.uint64)
        scales_w = (r.uniform(0.5, 1.5, size=(W, lay.nchunks)) * 1e-5).astype(F32)
        before = srv_err.astype(np.float64).copy()
        sw, ss, avg = orc.server(lay, words_w, scales_w, srv_err, want_avg=True)
        sent += orc.decompress(lay, sw, ss)
        total += avg
        bound += U * (np.abs(avg.astype(np.float64) + before) + np.abs(srv_err.astype(np.float64)))
    resid = sent - (total - srv_err.astype(np.float64))
    assert np.all(np.abs(resid) <= 2 * bound + 1e-30)


def test_server_ignores_pad_bits():
    lay = orc.Layout.from_segments([0, 100], 100)
    r = rng(4)
    W = 3
    words = r.integers(0, 2 ** 63, size=(W, lay.nwords), dtype=np.uint64)
    scales = (r.uniform(0.5, 1.5, size=(W, 1)) * 1e-4).astype(F32)
    e1 = np.zeros(100, F32)
    a1 = orc.server(lay, words, scales, e1, want_avg=True)
    masked = words.copy()
    masked[:, 1] &= np.uint64((1 << 36) - 1)
    e2 = np.zeros(100, F32)
    a2 = orc.server(lay, masked, scales, e2, want_avg=True)
    np.testing.assert_array_equal(a1[2], a2[2])
    np.testing.assert_array_equal(e1, e2)
    assert int(a1[0][1]) >> 36 == 0


# ---------------------------------------------------------------------------
# Algorithm 1 special cases
# ---------------------------------------------------------------------------

def _grads(n, steps, seed, sigma=1e-3):
    r = rng(seed)
    return [(r.standard_normal(n) * sigma).astype(F32) for _ in range(steps)]


def test_reduces_to_adam_when_every_step_syncs():
    """T_u = T_v = all steps, W = 1, compression off  ==>  Adam (Equation 2)."""
    n, T = 4096, 20
    x0 = (rng(1).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 2)
    gammas = [F32(1e-4)] * T
    ref = adam_fp64(x0, grads, gammas)
    w = orc.Worker(orc.Layout.from_segments([0, n], 1024), x0)
    for t in range(T):
        w.step(gammas[t], grads[t], sync=True, var=True, compress=False)
        x, m, v = ref[t]
        np.testing.assert_allclose(w.v, v, rtol=2e-6, atol=0)
        # momentum entries near zero come from cancellation: the floor is
        # relative to the tensor's magnitude (binary32 rounding of the terms)
        np.testing.assert_allclose(w.m, m, rtol=1e-6, atol=1e-6 * np.abs(m).max())
        np.testing.assert_allclose(w.x, x, rtol=1e-6, atol=1e-7)
        np.testing.assert_array_equal(w.anchor, w.x)
        assert not w.u.any() and w.gamma_sum == 0


def test_reduces_to_adam_without_sync():
    """T_u empty, T_v = all steps: the local lines are Adam on the model."""
    n, T = 2048, 15
    x0 = (rng(3).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 4)
    gammas = [F32(1e-4 * (1 + t)) for t in range(T)]
    ref = adam_fp64(x0, grads, gammas)
    w = orc.Worker(orc.Layout.from_segments([0, n], 512), x0)
    for t in range(T):
        w.step(gammas[t], grads[t], sync=False, var=True)
        x, m, v = ref[t]
        np.testing.assert_allclose(w.m, m, rtol=1e-6, atol=1e-6 * np.abs(m).max())
        np.testing.assert_allclose(w.v, v, rtol=2e-6, atol=0)
        np.testing.assert_allclose(w.x, x, rtol=1e-6, atol=1e-7)
    # the anchor never moves without a sync; u holds sum gamma m
    np.testing.assert_array_equal(w.anchor, x0)
    u_ref = sum(float(g) * ref[t][1] for t, g in enumerate(gammas))
    np.testing.assert_allclose(w.u, u_ref, rtol=1e-5, atol=1e-6 * np.abs(u_ref).max())
    assert w.gamma_sum == pytest.approx(sum(float(g) for g in gammas), rel=1e-6)


def test_unit_chunks_make_compression_lossless():
    """Chunk length 1: every scale is |a|, so compressing loses nothing and the
    run equals the uncompressed run bit for bit (W = 1)."""
    n, T = 512, 12
    x0 = (rng(5).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 6)
    lay1 = orc.Layout.from_segments([0, n], 1)
    a = orc.Worker(lay1, x0)
    b = orc.Worker(lay1, x0)
    sync = [t % 3 == 2 for t in range(T)]
    var = [t < 4 for t in range(T)]
    for t in range(T):
        a.step(F32(1e-4), grads[t], sync[t], var[t], compress=True)
        b.step(F32(1e-4), grads[t], sync[t], var[t], compress=False)
        for k in ("x", "m", "v", "u", "anchor"):
            np.testing.assert_array_equal(getattr(a, k), getattr(b, k))
        assert not a.err.any() and not a.srv_err.any()


def test_literal_momentum_index_freezes_momentum():
    """Literal reading of the model/buffer lines (old momentum) with a sync at
    every step: u = gamma m_t, ubar = u, m_{t+1} = ubar / gamma = m_t = 0."""
    n, T = 256, 6
    x0 = (rng(8).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 9)
    lay = orc.Layout.from_segments([0, n], 64)
    lit = orc.Worker(lay, x0, literal_momentum=True)
    fresh = orc.Worker(lay, x0)
    for t in range(T):
        lit.step(F32(1e-4), grads[t], True, True, compress=False)
        fresh.step(F32(1e-4), grads[t], True, True, compress=False)
        assert not lit.m.any()
        np.testing.assert_array_equal(lit.x, x0)
    assert np.abs(fresh.x - x0).max() > 0


def test_variance_frozen_outside_tv_and_bounded():
    """v is bit-unchanged at t not in T_v, and v <= (1 - b2^k) max gbar^2 after
    k updates (the bound behind the paper's variance lemma)."""
    n, T = 1000, 12
    x0 = np.zeros(n, F32)
    grads = _grads(n, T, 10)
    gbars = _grads(n, T, 11)
    tv = {0, 1, 3, 7}
    w = orc.Worker(orc.Layout.from_segments([0, n], 256), x0)
    k = 0
    gmax = 0.0
    for t in range(T):
        before = w.v.copy()
        w.step(F32(1e-4), grads[t], t % 2 == 1, t in tv, gbar=gbars[t], peer_words=None)
        if t in tv:
            k += 1
            gmax = max(gmax, float(np.max(gbars[t].astype(np.float64) ** 2)))
        else:
            np.testing.assert_array_equal(w.v.view(np.uint32), before.view(np.uint32))
        b2 = float(F32(0.999))
        assert np.all(w.v <= (1 - b2 ** k) * gmax * (1 + 1e-5))


def test_sync_with_frozen_variance_is_linear():
    """With v frozen, W = 1 and no compression, the synced model equals the
    model the local lines would have produced (x_{t'} - u / sqrt(v + eps)), and
    the momentum becomes the Gamma-weighted mean of the interval's momenta."""
    n = 1024
    x0 = (rng(12).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, 6, 13)
    gammas = [F32(1e-4), F32(2e-4), F32(3e-4), F32(1.5e-4), F32(1e-4), F32(5e-5)]
    lay = orc.Layout.from_segments([0, n], 256)
    w = orc.Worker(lay, x0)
    w.step(gammas[0], grads[0], sync=True, var=True, compress=False)   # v set, synced
    anchor = w.x.copy()
    local = orc.Worker(lay, x0)
    local.x[:], local.m[:], local.v[:] = w.x, w.m, w.v
    moms, gs = [], []
    for t in range(1, 6):
        last = t == 5
        local.step(gammas[t], grads[t], sync=False, var=False)
        moms.append(local.m.astype(np.float64).copy())
        gs.append(float(gammas[t]))
        w.step(gammas[t], grads[t], sync=last, var=False, compress=False)
    np.testing.assert_array_equal(w.anchor, w.x)
    assert not np.array_equal(w.x, anchor)
    # model: synced == local, up to the local path's per-step roundings
    scale = np.abs(local.x.astype(np.float64) - anchor).max()
    assert np.abs(w.x.astype(np.float64) - local.x).max() <= 1e-5 * scale + 4 * U * 0.1
    # momentum: ubar / Gamma == sum gamma_h m_h / sum gamma_h
    mean = sum(g * m for g, m in zip(gs, moms)) / sum(gs)
    np.testing.assert_allclose(w.m, mean, rtol=1e-5, atol=1e-6 * np.abs(mean).max())


def test_workers_reach_consensus_and_single_gpu_formulation_matches():
    """W real workers with their own gradients and a real server: after every
    sync all workers hold bit-identical x and m (the paper's consensus at sync
    steps).  Worker 0 run alone, fed the other workers' packed buffers as
    inputs, follows the identical trajectory."""
    W, T = 4, 9
    seg = [0, 700, 1024 + 700]
    lay = orc.Layout.from_segments(seg, 256)
    x0 = (rng(14).standard_normal(lay.n) * 0.02).astype(F32)
    workers = [orc.Worker(lay, x0) for _ in range(W)]
    solo = orc.Worker(lay, x0)
    server_err = np.zeros(lay.n, F32)
    grads = [_grads(lay.n, T, 100 + w) for w in range(W)]
    gbars = _grads(lay.n, T, 99)
    tu = {1, 3, 4, 8}
    tv = {0, 1, 2, 5}
    for t in range(T):
        gamma = F32(1e-4 * (1 + 0.1 * t))
        for w in range(W):
            workers[w].half_step(gamma, grads[w][t])
        if t in tu:
            sent = [wk.compress() for wk in workers]
            words_w = np.stack([s[0] for s in sent])
            scales_w = np.stack([s[1] for s in sent])
            sw, ss, _ = orc.server(lay, words_w, scales_w, server_err)
            for wk in workers:
                wk.sync(sw, ss)
            out = solo.step(gamma, grads[0][t], True, t in tv, gbar=gbars[t],
                            peer_words=words_w[1:], peer_scales=scales_w[1:])
            assert np.array_equal(out["own_words"], words_w[0])
            np.testing.assert_array_equal(out["srv_words"], sw)
            for wk in workers[1:]:
                np.testing.assert_array_equal(wk.x, workers[0].x)
                np.testing.assert_array_equal(wk.m, workers[0].m)
        else:
            solo.step(gamma, grads[0][t], False, t in tv, gbar=gbars[t])
        if t in tv:
            for wk in workers:
                wk.variance(gbars[t])
        for k in ("x", "m", "v", "u", "err", "anchor"):
            np.testing.assert_array_equal(getattr(solo, k), getattr(workers[0], k))
        np.testing.assert_array_equal(solo.srv_err, server_err)
