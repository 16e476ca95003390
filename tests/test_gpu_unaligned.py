"""GPU parity for compression chunk lengths that are not a multiple of 4.

A chunk then need not start on a 16-byte boundary and its last float4 may be
partial, so the chunk kernels take their unaligned forms (element accesses,
the tail past the chunk masked) and the server its plain form.  Every state,
packed word and scale is compared with the oracle after every step, bit for
bit (-0 == +0).  The unit chunk length makes Equation 3 lossless (the scale
of a one-element chunk is its magnitude), so with one worker the run must
equal the oracle's run with compression off, bit for bit.
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


def _wl(name, segs, chunk, world, steps=8, tu=None, tv=None, algorithm=None):
    T = steps
    extra = {"algorithm": algorithm} if algorithm else {}
    return C.Workload(
        name=name, seg_off=C.offsets(segs), world=world, chunk=chunk, steps=T,
        tv=tv if tv is not None else [0, 1, 2, 5],
        tu=([] if algorithm else (tu if tu is not None else [t for t in range(T) if t % 3 != 0])),
        gammas=[1e-4 * (1 + 0.25 * t) for t in range(T)], sigma_g=1e-3, extra=extra)


UNALIGNED = [
    # (segments, chunk, W): compress geometry L lanes / V blocks per lane
    ([100, 4, 36, 0, 260], 1, 3),            # L1: one element per chunk
    ([96, 12, 8, 40], 2, 2),                 # L1
    ([132, 16, 0, 64], 3, 5),                # L1, an empty segment
    ([200, 32, 4], 5, 1),                    # L2
    ([1000, 64, 60], 7, 4),                  # L2
    ([1000, 128, 124, 4], 63, 8),            # L16
    ([3000, 256, 252], 65, 16),              # L32
    ([5000, 512, 4, 508], 99, 3),            # L32
    ([9000, 1024, 1020, 8], 1023, 4),        # L256
    ([20000, 2048, 4], 2047, 2),             # L512
    ([12000, 2500, 4000], 2999, 7),          # L1024 V1
    ([40000, 8192, 8188], 8191, 4),          # L1024 V2
    ([70000, 16384, 16380, 4], 16383, 3),    # L1024 V4
    ([5000, 1000, 96], 1021, 40),            # five worker groups
    ([20000, 3000], 4093, 128),              # W = 128
]


@pytest.mark.parametrize("segs,chunk,world", UNALIGNED,
                         ids=[f"C{c}-W{w}" for _, c, w in UNALIGNED])
def test_unaligned_layouts(torch_cuda, segs, chunk, world):
    import harness
    wl = _wl(f"ua-C{chunk}", segs, chunk, world)
    report, inexact = harness.run_parity(wl, log=_log)
    _assert_clean(report, inexact)


@pytest.mark.parametrize("segs,chunk,world", [UNALIGNED[1], UNALIGNED[7], UNALIGNED[12]],
                         ids=["C2-W2", "C99-W3", "C16383-W3"])
def test_unaligned_deferred_and_unfused(torch_cuda, segs, chunk, world):
    """Local steps after deferred syncs (the momentum rebuilt from the server
    copy over the chunk grid), a sync right after a sync, zo_read_state and
    the unfused path, at unaligned chunks."""
    import harness
    wl = _wl(f"ua-defer-C{chunk}", segs, chunk, world, steps=9, tu=[1, 2, 4, 5, 8],
             tv=[0, 2, 3, 5])
    for fused in (True, False):
        report, inexact = harness.run_parity(wl, log=_log, defer=True, fused=fused,
                                             materialize_at=(5,))
        _assert_clean(report, inexact)


@pytest.mark.parametrize("segs,chunk,world", [UNALIGNED[0], UNALIGNED[10]],
                         ids=["C1-W3", "C2999-W7"])
def test_unaligned_one_bit_adam(torch_cuda, segs, chunk, world):
    """Algorithm 4 (compressed gradients, the full-precision step in the
    middle): the compress of g and the server-output step at unaligned chunks."""
    import harness
    wl = _wl(f"ua-fv-C{chunk}", segs, chunk, world, tv=[0, 1, 4], algorithm="frozen-variance")
    report, inexact = harness.run_parity(wl, log=_log)
    _assert_clean(report, inexact)


def test_unaligned_bf16_gradients(torch_cuda):
    import harness
    wl = _wl("ua-bf16", [12000, 2500, 4000], 2999, 7)
    report, inexact = harness.run_parity(wl, log=_log, defer=True, grad_dtype="bf16")
    _assert_clean(report, inexact)


@pytest.mark.parametrize("defer", [False, True], ids=["eager", "defer"])
def test_unit_chunks_single_worker_equal_compression_off(torch_cuda, defer):
    """Chunk length 1 makes Equation 3 lossless: s = |a| and the error stays
    +-0, and with W = 1 the server's average of the one worker is its own
    value, which recompresses losslessly too.  So the library's run equals the
    oracle's run with compression off (the sync lines applied to u itself),
    bit for bit with -0 == +0, after every step; both errors stay zero."""
    import harness
    import oracle as orc
    torch = torch_cuda
    T = 10
    wl = _wl("unit-chunks", [4096, 1000, 2000], 1, 1, steps=T, tu=[1, 2, 4, 5, 7, 9],
             tv=[0, 1, 3, 4, 6])
    grun = harness.GpuRun(wl, defer=defer)
    orun = harness.OracleRun(wl)      # only for the inputs (gradients, x0)
    ref = orc.Worker(orc.Layout.from_segments(wl.seg_off, 1), orun.state("x"), wl.beta1,
                     wl.beta2, wl.eps)
    n = wl.n
    try:
        for t in range(T):
            sync, var = harness.steps_kind(wl, t)
            grun.step(t)
            g = orun.grad(t)
            ref.step(wl.gamma(t), g, sync, var, gbar=orun.gbar(t) if var else None,
                     compress=False)
            torch.cuda.synchronize()
            for k in ("x", "m", "v", "u", "anchor"):
                gpu = grun.opt.current(k)[:n].cpu().numpy()
                bad = int(np.count_nonzero(~(gpu == getattr(ref, k))))
                assert bad == 0, (t, k, bad)
            for k in ("err", "srv_err"):
                assert not grun.state[k][:n].any().item(), (t, k)
        assert grun.opt.inexact_chunks() == 0
    finally:
        grun.close()
