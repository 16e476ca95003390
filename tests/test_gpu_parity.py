"""GPU parity: the HIP library against the CPU oracle, bit for bit.

Every state (x, m, v, u, worker error, server error, anchor), the own packed
signs and scales and the server packed signs and scales are compared after
every step of a run.  The contract allows a relative error of 1e-6 on the
binary32 states; the kernels are built to reproduce the oracle's rounding
exactly, so these tests demand equality (with -0 == +0), which implies it.
"""
import numpy as np
import pytest

from synth import configs as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(autouse=True)
def _free_memory(torch_cuda):
    yield
    import gc
    gc.collect()
    torch_cuda.cuda.empty_cache()


def _log(msg):
    print(msg, flush=True)


def _assert_clean(report, inexact):
    for t, bad in enumerate(report):
        assert not bad, f"mismatch after step {t - 1}: {bad}"
    assert inexact == 0


# ---------------------------------------------------------------------------
# the binary32 division and square root the kernels use
# ---------------------------------------------------------------------------

def test_device_div_sqrt_are_correctly_rounded(torch_cuda):
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    r = np.random.default_rng(0)
    n = 1 << 24
    # random finite bit patterns (both signs, all exponents incl. denormals)
    a = r.integers(0, 0x7F800000, size=n, dtype=np.uint32).view(np.float32).copy()
    b = r.integers(0, 0x7F800000, size=n, dtype=np.uint32).view(np.float32).copy()
    b[r.random(n) < 0.5] *= -1
    # values like the optimizer's: v + eps around 1e-8 .. 1e-2, ubar ~ 1e-8
    a[: n // 4] = (r.random(n // 4) * 1e-2 + 1e-8).astype(np.float32)
    b[: n // 4] = (r.standard_normal(n // 4) * 1e-4).astype(np.float32)
    ta, tb = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    tq, tr = torch.empty_like(ta), torch.empty_like(ta)
    zo.zo_diag_divsqrt(ta, tb, tq, tr)
    torch.cuda.synchronize()
    with np.errstate(all="ignore"):
        q_ref = a / b
        r_ref = np.sqrt(a)
    q, rr = tq.cpu().numpy(), tr.cpu().numpy()
    assert np.array_equal(q.view(np.uint32), q_ref.view(np.uint32))
    assert np.array_equal(rr.view(np.uint32), r_ref.view(np.uint32))


# ---------------------------------------------------------------------------
# Tiny workload, whole shard, both readings of its schedule
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("defer", [False, True], ids=["eager", "defer"])
@pytest.mark.parametrize("name", ["tiny", "tiny-alt"])
@pytest.mark.parametrize("fused", [True, False])
def test_tiny_full_shard(torch_cuda, name, fused, defer):
    """defer: the reconstruction leaves x in the anchor and u implicit; the
    logical state (x from wherever it lives, u as zeros) must still match."""
    import harness
    report, inexact = harness.run_parity(C.get(name), fused=fused, log=_log, defer=defer)
    _assert_clean(report, inexact)
    assert len(report) == C.get(name).steps + 1


# ---------------------------------------------------------------------------
# small ragged layouts: every kernel geometry, ragged tails, empty segments
# ---------------------------------------------------------------------------

def _small(name, segs, chunk, world, steps=8, tu=None, tv=None, sigma=1e-3, gammas=None):
    T = steps
    return C.Workload(
        name=name, seg_off=C.offsets(segs), world=world, chunk=chunk, steps=T,
        tv=tv if tv is not None else [0, 1, 2, 5],
        tu=tu if tu is not None else [t for t in range(T) if t % 3 != 0],
        gammas=gammas or [1e-4 * (1 + 0.25 * t) for t in range(T)], sigma_g=sigma)


SMALL = [
    # (segments, chunk, W).  The chunk sets the compress geometry: L lanes per
    # chunk (several chunks per 256-thread workgroup while L < 256) and V
    # blocks of 4L elements per lane (V > 1 only at L = 1024); and the
    # server's: LD lanes per chunk (one packed dword each) and G worker groups
    # of 8 (rounded up to a power of two while LD < 64).  Comments: L/V, LD/G.
    ([100, 4, 36, 0, 260], 4, 3),            # L1 V1, LD1 G1
    ([96, 12, 8, 40], 8, 2),                 # L2 V1, LD1 G1
    ([132, 16, 0, 64], 16, 5),               # L4 V1, LD1 G1; an empty segment
    ([200, 32, 4], 28, 1),                   # L8 V1, LD1 G1; chunk not a power of two
    ([1000, 64, 60], 64, 4),                 # L16 V1, LD2 G1
    ([1000, 128, 124, 4], 100, 8),           # L32 V1, LD4 G1
    ([3000, 256, 252], 256, 16),             # L64 V1, LD8 G2
    ([5000, 512, 4, 508], 500, 3),           # L128 V1, LD16 G1
    ([9000, 1024, 1020, 8], 1024, 4),        # L256 V1, LD32 G1
    ([20000, 2048, 4], 2048, 2),             # L512 V1, LD64 G1
    ([12000, 2500, 4000], 3000, 7),          # L1024 V1 (750 lanes used), LD128 G1
    ([40000, 8192, 8188], 8192, 4),          # L1024 V2, LD256 G1
    ([70000, 16384, 16380, 4], 16384, 3),    # L1024 V4, LD512 G1
    ([5000, 1000, 96], 1024, 9),             # LD32 G2, the second group partial
    ([3000, 1024, 1020, 8], 1024, 40),       # LD32 G8: groups 5..7 past the last worker
    ([20000, 16384, 4], 16384, 100),         # LD512 G13 at the GPT-2 chunk, the last of 4 workers
    ([6000, 2048, 2044], 2048, 20),          # LD64 G3, the last of 4 workers
    ([8192, 4096, 100], 4096, 72),           # LD128 G9
    ([8192, 8192, 8000], 8192, 88),          # LD256 G11 (three waves per SIMD)
    ([32768, 16384, 12], 16384, 120),        # LD512 G15 (three waves per SIMD)
    ([3000, 500, 12], 256, 128),             # half tables: LD8 G16
    ([700, 64, 36], 32, 64),                 # half tables: LD1 G8
    ([5000, 1000], 1024, 300),               # tables beyond the LDS budget: plain server
]


@pytest.mark.parametrize("segs,chunk,world", SMALL, ids=[f"C{c}-W{w}" for _, c, w in SMALL])
def test_small_layouts_full_shard(torch_cuda, segs, chunk, world):
    import harness
    wl = _small(f"small-C{chunk}", segs, chunk, world)
    report, inexact = harness.run_parity(wl, log=_log)
    _assert_clean(report, inexact)


@pytest.mark.parametrize("defer", [False, True], ids=["eager", "defer"])
def test_single_worker_every_step_syncs(torch_cuda, defer):
    """W = 1 with a sync and a variance update at every step (the setting in
    which the method reduces to Adam) -- exercises the fused variance line in
    the reconstruction at every step; deferred, every compress after the
    first reads u as the implicit zero and the model stays in the anchor."""
    import harness
    T = 10
    wl = _small("w1-adam", [8192, 4096, 1000], 1024, 1, steps=T, tu=list(range(T)),
                tv=list(range(T)))
    report, inexact = harness.run_parity(wl, log=_log, defer=defer)
    _assert_clean(report, inexact)


@pytest.mark.parametrize("segs,chunk,world", [SMALL[0], SMALL[6], SMALL[10]],
                         ids=["C4-W3", "C256-W16", "C3000-W7"])
def test_small_layouts_deferred_writes(torch_cuda, segs, chunk, world):
    """Runs of local steps after deferred syncs, a sync right after a sync
    (steps 1-2 and 4-5), and the unfused path."""
    import harness
    T = 9
    wl = _small(f"defer-C{chunk}", segs, chunk, world, steps=T, tu=[1, 2, 4, 5, 8],
                tv=[0, 2, 3, 5])
    for fused in (True, False):
        report, inexact = harness.run_parity(wl, log=_log, defer=True, fused=fused)
        _assert_clean(report, inexact)


def test_materialize_after_deferred_sync(torch_cuda):
    """zo_materialize writes x and u out at any point between steps and the
    run continues bit for bit."""
    import harness
    torch = torch_cuda
    T = 8
    wl = _small("materialize", [5000, 1000, 96], 1024, 5, steps=T, tu=[1, 2, 5],
                tv=[0, 3])
    report, inexact = harness.run_parity(wl, log=_log, defer=True, materialize_at=(1, 3, 5))
    _assert_clean(report, inexact)
    run = harness.GpuRun(wl, defer=True)
    zo = run.zo
    n = wl.n
    try:
        for t in range(3):
            run.step(t)
        # after the sync at step 2: the model in the anchor, u = +0
        xp, mode, _ = zo.zo_state_location(run.opt.h)
        assert xp == run.state["anchor"].data_ptr() and mode == zo.U_ZERO
        run.opt.materialize()
        xp, mode, _ = zo.zo_state_location(run.opt.h)
        assert xp == run.state["x"].data_ptr() and mode == zo.U_IN_BUFFER
        torch.cuda.synchronize()
        assert torch.equal(run.state["x"][:n].view(torch.int32),
                           run.state["anchor"][:n].view(torch.int32))
        assert torch.equal(run.state["u"][:n].view(torch.int32),
                           torch.zeros(n, dtype=torch.int32, device="cuda"))
        # one more sync, then the first local step after it: u = +0 + gamma_3 m
        run.step(3)
        run2 = harness.GpuRun(wl, defer=True)
        try:
            for t in range(4):
                run2.step(t)
            xp, mode, gam = zo.zo_state_location(run2.opt.h)
            assert mode == zo.U_GAMMA_M and gam == wl.gamma(3)
            assert xp == run2.state["x"].data_ptr()
            run2.opt.materialize()
            torch.cuda.synchronize()
            want = (run2.state["m"][:n] * torch.tensor(gam, device="cuda")) + 0.0
            assert torch.equal(run2.state["u"][:n].view(torch.int32), want.view(torch.int32))
            assert zo.zo_state_location(run2.opt.h)[1] == zo.U_IN_BUFFER
        finally:
            run2.close()
    finally:
        run.close()


def test_local_steps_only(torch_cuda):
    import harness
    T = 12
    wl = _small("local-only", [50000, 4096], 2048, 4, steps=T, tu=[], tv=[0, 3, 7])
    report, inexact = harness.run_parity(wl, log=_log)
    _assert_clean(report, inexact)


# ---------------------------------------------------------------------------
# the paper-shaped workloads at full size
# ---------------------------------------------------------------------------

def _sample(wl):
    """Every ragged chunk, both ends of every segment and every 50th other chunk
    (at least 2% of the shard)."""
    import harness
    import oracle as orc
    lay = orc.Layout.from_segments(wl.seg_off, wl.chunk)
    ids = harness.sample_chunks(lay, wl.seg_off)
    ragged = lay.clen != wl.chunk
    assert ragged[ids].sum() == ragged.sum()
    assert lay.clen[ids].sum() >= 0.02 * wl.n
    return ids


def test_gpt2_sampled_deferred_writes(torch_cuda):
    """The GPT-2-1.5B shard in the mode and launch shapes the benchmark times
    (deferred sync writes, fused calls, single server at W = 128)."""
    import harness
    import dataclasses
    T = 8
    # the benchmark's alternation: a local step, then a sync step, each with
    # the variance update
    wl = dataclasses.replace(C.get("gpt2-1.5b"), name="gpt2-1.5b-alternating", steps=T,
                             tu=list(range(1, T, 2)), tv=list(range(T)),
                             gammas=[1e-4] * T)
    report, inexact = harness.run_parity(wl, chunk_ids=_sample(wl), log=_log, defer=True)
    _assert_clean(report, inexact)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["bert-large", "gpt2-1.5b"])
def test_workload_sampled(torch_cuda, name):
    """BERT-Large and GPT-2-1.5B over their whole schedules, the oracle on a
    sample of chunks; the computation is chunk-local, so the sample's values
    are exactly the full run's."""
    import harness
    wl = C.get(name)
    report, inexact = harness.run_parity(wl, chunk_ids=_sample(wl), log=_log)
    _assert_clean(report, inexact)


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name", ["resnet50", "bert-base"])
def test_workload_full_shard(torch_cuda, name):
    """ResNet-50 and BERT-Base with the oracle over the whole shard (every
    element, word and scale compared after every step of the workload's
    schedule), not a sample of chunks."""
    import harness
    wl = C.get(name)
    _log(f"{name}: full shard, {wl.n} params, W={wl.world}, {wl.steps} steps")
    report, inexact = harness.run_parity(wl, log=_log)
    _assert_clean(report, inexact)


def test_largest_world(torch_cuda):
    """W = 65536, the largest worker count the library takes (the plain server:
    its tables would not fit in LDS), on a small ragged shard."""
    import harness
    wl = _small("w65536", [2048, 100], 1024, 65536, steps=3, tu=[1, 2], tv=[0])
    report, inexact = harness.run_parity(wl, log=_log)
    _assert_clean(report, inexact)
