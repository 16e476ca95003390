"""Pins of the oracle's Algorithm 4 (the frozen-variance framework with
compressed gradients; 1-bit Adam when T_v is a prefix of the steps) against
what the paper and the mathematics fix: Equation 2 computed by an independent
binary64 implementation when nothing is compressed or compression is lossless,
the listing's own special cases (a zero first step, a frozen variance), and
the error-feedback telescoping of the compressed gradients.
"""
import numpy as np

import oracle as orc
from oracle.brute_adam import adam_eq2_fp64

F32 = np.float32


def rng(seed):
    return np.random.default_rng(seed)


def _grads(n, T, seed, scale=1e-3):
    r = rng(seed)
    return [(r.standard_normal(n) * scale).astype(F32) for _ in range(T)]


def _close_to(w, ref):
    x, m, v = ref
    np.testing.assert_allclose(w.v, v, rtol=2e-6, atol=0)
    np.testing.assert_allclose(w.m, m, rtol=1e-6, atol=1e-6 * np.abs(m).max())
    np.testing.assert_allclose(w.x, x, rtol=1e-6, atol=1e-7)


def test_full_precision_steps_are_equation2():
    """T_v = every step, one worker: Algorithm 4 is Equation 2 as printed."""
    n, T = 4096, 20
    x0 = (rng(1).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 2)
    gammas = [F32(1e-4 * (1 + 0.1 * t)) for t in range(T)]
    ref = adam_eq2_fp64(x0, grads, gammas)
    w = orc.FVWorker(orc.Layout.from_segments([0, n], 1024), x0)
    for t in range(T):
        assert w.step(gammas[t], grads[t], full=True) == {}
        _close_to(w, ref[t])


def test_first_step_leaves_the_model():
    """The model line uses m_t, and m_0 = 0: step 0 does not move x."""
    n = 1000
    x0 = (rng(3).standard_normal(n) * 0.02).astype(F32)
    g = _grads(n, 1, 4)[0]
    for full in (True, False):
        w = orc.FVWorker(orc.Layout.from_segments([0, 1000], 256), x0)
        w.step(F32(1e-3), g, full=full)
        np.testing.assert_array_equal(w.x, x0)
        assert w.m.any()


def test_one_bit_adam_with_lossless_compression_is_equation2_with_frozen_variance():
    """1-bit Adam (T_v = the first T0 steps) with unit chunks, one worker:
    every scale is |a|, so compressing loses nothing, the compressed average
    is the gradient itself and the run is Equation 2 with v frozen after T0."""
    n, T, T0 = 512, 14, 4
    x0 = (rng(5).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 6)
    gammas = [F32(1e-4)] * T
    ref = adam_eq2_fp64(x0, grads, gammas, update_v=lambda t: t < T0)
    w = orc.FVWorker(orc.Layout.from_segments([0, n], 1), x0)
    for t in range(T):
        out = w.step(gammas[t], grads[t], full=t < T0)
        _close_to(w, ref[t])
        if t >= T0:
            assert not w.err.any() and not w.srv_err.any()
            got = orc.decompress(w.layout, out["srv_words"], out["srv_scales"])
            np.testing.assert_array_equal(got, grads[t])


def test_variance_is_frozen_outside_tv():
    """With real chunks and W = 4, v changes at the T_v steps only."""
    segs = [0, 3000, 3500, 8192]
    lay = orc.Layout.from_segments(segs, 256)
    n, T = lay.n, 10
    tv = {0, 1, 2, 6}
    x0 = (rng(7).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 8)
    r = rng(9)
    w = orc.FVWorker(lay, x0)
    for t in range(T):
        v_before = w.v.copy()
        m_before = w.m.copy()
        pw = r.integers(0, 2 ** 63, size=(3, lay.nwords), dtype=np.int64).astype(np.uint64)
        ps = (r.random((3, lay.nchunks)) * 1e-3).astype(F32)
        w.step(F32(1e-4), grads[t], full=t in tv, peer_words=pw, peer_scales=ps)
        if t in tv:
            assert not np.array_equal(w.v, v_before)
        else:
            np.testing.assert_array_equal(w.v, v_before)
        assert not np.array_equal(w.m, m_before)


def test_compressed_step_uses_the_server_average():
    """A compressed step: m_{t+1} = b1 m_t + (1 - b1) gbar with gbar the
    server's decompressed output, and x_{t+1} = x_t - gamma m_t / sqrt(v_t + eps),
    checked in binary64 from the outputs (W = 5, ragged chunks)."""
    segs = [0, 2000, 2004, 6000]
    lay = orc.Layout.from_segments(segs, 512)
    n, T = lay.n, 6
    x0 = (rng(11).standard_normal(n) * 0.02).astype(F32)
    grads = _grads(n, T, 12)
    r = rng(13)
    w = orc.FVWorker(lay, x0)
    b1, e = float(F32(0.9)), float(F32(1e-8))
    for t in range(T):
        x_b, m_b, v_b = w.x.astype(np.float64), w.m.astype(np.float64), w.v.astype(np.float64)
        full = t < 2
        pw = r.integers(0, 2 ** 63, size=(4, lay.nwords), dtype=np.int64).astype(np.uint64)
        ps = (r.random((4, lay.nchunks)) * 1e-3).astype(F32)
        gam = F32(2e-4)
        out = w.step(gam, grads[t], full=full, peer_words=pw, peer_scales=ps)
        gbar = grads[t] if full else orc.decompress(lay, out["srv_words"], out["srv_scales"])
        m_ref = b1 * m_b + (1.0 - b1) * gbar.astype(np.float64)
        x_ref = x_b - float(gam) * m_b / np.sqrt(v_b + e)
        np.testing.assert_allclose(w.m, m_ref, rtol=1e-6, atol=1e-6 * np.abs(m_ref).max())
        np.testing.assert_allclose(w.x, x_ref, rtol=1e-6, atol=1e-7)


def test_compressed_gradients_telescope():
    """One worker, K compressed steps: the gradients the optimizer applied sum
    to the true gradients minus the final worker and server errors,
    sum_k gbar_k = sum_k g_k - delta_K - delta_bar_K (up to binary32 rounding)."""
    lay = orc.Layout.from_segments([0, 4096, 5000], 256)
    n, K = lay.n, 12
    grads = _grads(n, K, 14)
    w = orc.FVWorker(lay, np.zeros(n, F32))
    applied = np.zeros(n)
    mag = np.zeros(n)
    for k in range(K):
        out = w.step(F32(1e-4), grads[k], full=False)
        gb = orc.decompress(lay, out["srv_words"], out["srv_scales"]).astype(np.float64)
        applied += gb
        mag += np.abs(gb) + np.abs(grads[k])
    want = sum(g.astype(np.float64) for g in grads) - w.err - w.srv_err
    np.testing.assert_allclose(applied, want, rtol=0, atol=float(8 * 2.0 ** -24 * mag.max()))
