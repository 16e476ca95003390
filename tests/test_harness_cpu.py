"""Host pieces of the test harness that the GPU tests rely on."""
import numpy as np
import pytest

import harness


def test_bfloat16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -1.0 - 2 ** -8,
                  3.0e-39, 2.0 ** -126 * 1.5], np.float32)
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -1.0, 3.0e-39, 2.0 ** -126 * 1.5],
                    np.float32)
    got = harness.round_to(x, "bf16")
    # every result is a bfloat16 value (low 16 bits zero)
    assert not (got.view(np.uint32) & 0xFFFF).any()
    np.testing.assert_array_equal(got[:5], want[:5])
    # the subnormal and the normal with 1 extra bit round to their neighbours
    assert abs(float(got[5]) - 3.0e-39) <= 2.0 ** -133
    assert got[6] == np.float32(2.0 ** -126 * 1.5)


def test_float16_rounding_matches_numpy():
    r = np.random.default_rng(0)
    x = (r.standard_normal(10000) * 1e-4).astype(np.float32)
    np.testing.assert_array_equal(harness.round_to(x, "f16"),
                                  x.astype(np.float16).astype(np.float32))
    assert harness.round_to(x, "f32") is not None


def _small_wl(world=5, chunk=100, segs=(1000, 128, 124, 4, 3000), T=6, algorithm=None):
    from synth import configs as C
    extra = {"algorithm": algorithm} if algorithm else {}
    tu = [] if algorithm else [1, 2, 4, 5]
    return C.Workload(name="harness-cpu", seg_off=C.offsets(list(segs)), world=world,
                      chunk=chunk, steps=T, tv=[0, 1, 3], tu=tu,
                      gammas=[1e-4 * (1 + 0.25 * t) for t in range(T)], sigma_g=1e-3,
                      extra=extra)


def test_sample_holds_every_ragged_chunk_and_both_segment_ends():
    import oracle as orc
    from synth import configs as C
    for name in ("bert-large", "gpt2-1.5b"):
        wl = C.get(name)
        lay = orc.Layout.from_segments(wl.seg_off, wl.chunk)
        ids = harness.sample_chunks(lay, wl.seg_off)
        assert np.all(np.diff(ids) > 0)
        got = set(ids.tolist())
        seg = np.searchsorted(wl.seg_off, lay.cstart, side="right") - 1
        for s in range(wl.nseg):
            cs = np.flatnonzero(seg == s)
            if len(cs):
                assert cs[0] in got and cs[-1] in got
        assert all(int(c) in got for c in np.flatnonzero(lay.clen != wl.chunk))
        assert lay.clen[ids].sum() >= 0.02 * wl.n
        # the stride part: no gap between chosen chunks longer than 50 (+ the chosen ends)
        assert np.diff(ids).max() <= 51


@pytest.mark.parametrize("algorithm", [None, "frozen-variance"])
def test_threaded_oracle_equals_one_run(algorithm):
    """The oracle split into pieces on threads computes what one run over the
    same chunks computes: every state and output after every step, bitwise."""
    wl = _small_wl(algorithm=algorithm)
    import oracle as orc
    lay = orc.Layout.from_segments(wl.seg_off, wl.chunk)
    ids = np.array([0, 1, 2, 5, 9, 10, 11, lay.nchunks - 2, lay.nchunks - 1])
    one = harness.OracleRun(wl, ids)
    par = harness.ParallelOracle(wl, ids, parts=3)
    assert len(par.runs) == 3
    try:
        keys = ("x", "m", "v", "err", "srv_err") + (() if algorithm else ("u", "anchor"))
        for t in range(wl.steps):
            a, b = one.step(t), par.step(t)
            assert a.keys() == b.keys()
            for k in a:
                assert np.array_equal(a[k], b[k]), (t, k)
            for k in keys:
                assert np.array_equal(one.state(k).view(np.uint32), par.state(k).view(np.uint32))
        assert par.ranges == one.ranges and par.wranges == one.wranges
    finally:
        par.close()


def test_sampled_oracle_equals_full_run_on_its_chunks():
    """The oracle on a sample of chunks reproduces, on those chunks, what the
    run over the whole shard computes (every computation is chunk-local)."""
    wl = _small_wl(world=3, chunk=64, segs=(640, 64, 60, 4, 700))
    full = harness.OracleRun(wl)
    ids = np.array([0, 3, 4, 12, full.full.nchunks - 1])
    part = harness.ParallelOracle(wl, ids, parts=2)
    el, wd = harness.gather_index(part)
    try:
        for t in range(wl.steps):
            out_f, out_p = full.step(t), part.step(t)
            for k in ("x", "m", "v", "u", "err", "srv_err", "anchor"):
                assert np.array_equal(full.state(k)[el], part.state(k)), (t, k)
            if out_f:
                assert np.array_equal(out_f["own_words"][wd], out_p["own_words"])
                assert np.array_equal(out_f["srv_words"][wd], out_p["srv_words"])
                assert np.array_equal(out_f["srv_scales"][ids], out_p["srv_scales"])
    finally:
        part.close()
