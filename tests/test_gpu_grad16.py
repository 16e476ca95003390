"""16-bit gradient inputs (binary16 and bfloat16, as in the paper's FP16
training): the library widens them exactly to binary32, so a run fed the
16-bit gradients must equal, bit for bit, the oracle fed the same values in
binary32."""
import dataclasses

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


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("fused,defer", [(True, True), (False, False)], ids=["fused-defer",
                                                                             "unfused-eager"])
def test_tiny(torch_cuda, dtype, fused, defer):
    import harness
    report, inexact = harness.run_parity(C.get("tiny"), fused=fused, defer=defer, log=_log,
                                         grad_dtype=dtype)
    _assert_clean(report, inexact)


def _small(name, segs, chunk, world, T=8):
    return C.Workload(name=name, seg_off=C.offsets(segs), world=world, chunk=chunk, steps=T,
                      tv=[0, 1, 2, 5], tu=[1, 2, 4, 7],
                      gammas=[1e-4 * (1 + 0.25 * t) for t in range(T)], sigma_g=1e-3)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("segs,chunk,world", [([100, 4, 36, 0, 260], 4, 3),
                                              ([12000, 2500, 4000], 3000, 7),
                                              ([70000, 16384, 16380, 4], 16384, 3)],
                         ids=["C4", "C3000", "C16384"])
def test_small_layouts(torch_cuda, dtype, segs, chunk, world):
    import harness
    wl = _small(f"g16-C{chunk}", segs, chunk, world)
    report, inexact = harness.run_parity(wl, defer=True, log=_log, grad_dtype=dtype)
    _assert_clean(report, inexact)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_one_bit_adam(torch_cuda, dtype):
    import harness
    report, inexact = harness.run_parity(C.get("tiny-1bit"), log=_log, grad_dtype=dtype)
    _assert_clean(report, inexact)


def test_gpt2_sampled_bf16(torch_cuda):
    """The GPT-2-1.5B shard with bfloat16 gradients in the benchmark's
    alternation (local step, sync step, both with the variance update)."""
    import harness
    import oracle as orc
    T = 6
    wl = dataclasses.replace(C.get("gpt2-1.5b"), name="gpt2-1.5b-alternating", steps=T,
                             tu=list(range(1, T, 2)), tv=list(range(T)), gammas=[1e-4] * T)
    lay = orc.Layout.from_segments(wl.seg_off, wl.chunk)
    ids = harness.sample_chunks(lay, wl.seg_off)
    report, inexact = harness.run_parity(wl, chunk_ids=ids, log=_log, defer=True,
                                         grad_dtype="bf16")
    _assert_clean(report, inexact)


def test_alignment_of_16bit_gradients(torch_cuda):
    """16-bit gradients need 8-byte alignment (four elements), binary32 16."""
    import harness
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    wl = _small("g16-align", [4096, 1000], 1024, 4)
    for dtype, ok_off, bad_off in (("bf16", 4, 2), ("f32", 4, 2)):
        run = harness.GpuRun(wl, grad_dtype=dtype)
        try:
            run.fill_inputs(0)
            buf = run.g_in.new_zeros(wl.n + 8)
            with pytest.raises(zo.ZoError) as e:
                run.opt.local_step(0, 1e-4, buf[bad_off:bad_off + wl.n], None)
            assert e.value.status == zo.ZO_EALIGN
            if dtype == "bf16":
                run.opt.local_step(0, 1e-4, buf[ok_off:ok_off + wl.n], None)
                assert run.opt.next_step == 0  # t = 0 is in T_v: the variance is still due
            torch.cuda.synchronize()
        finally:
            run.close()
