"""zo_adam_init_static, the entry point for callers that cannot allocate,
against zo_adam_init through the C ABI: two static handles in a row (the
second on a smaller shard, reusing the static scratch the first left behind),
each run step by step beside a handle from zo_adam_init on the same inputs
(the first with deferred sync writes, the second at a chunk length that is not
a multiple of 4);
every state, packed word and scale must be equal after every step (-0 == +0),
and so must the chunk table read back from the device."""
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


def _wl(name, segs, chunk, world, T, tu, tv):
    return C.Workload(name=name, seg_off=C.offsets(segs), world=world, chunk=chunk, steps=T,
                      tv=list(tv), tu=list(tu), gammas=[1e-4 * (1 + 0.25 * t) for t in range(T)],
                      sigma_g=1e-3)


def _same(a, b):
    return int(np.count_nonzero(~(a == b)))


def _run_pair(torch, wl, defer):
    import harness
    ref = harness.GpuRun(wl, defer=defer)                  # zo_adam_init
    sta = harness.GpuRun(wl, defer=defer, static=True)     # zo_adam_init_static
    n = wl.n
    try:
        assert sta.opt.chunk_table() == ref.opt.chunk_table()
        for t in range(wl.steps):
            ref.step(t)
            sta.step(t)
            torch.cuda.synchronize()
            for k in ref.keys:
                a = ref.opt.current(k)[:n].cpu().numpy()
                b = sta.opt.current(k)[:n].cpu().numpy()
                assert _same(a, b) == 0, (wl.name, t, k)
            for name in ("packed", "scales", "srv_packed", "srv_scales"):
                a = getattr(ref, name).cpu().numpy()
                b = getattr(sta, name).cpu().numpy()
                assert _same(a, b) == 0, (wl.name, t, name)
            print(f"{wl.name} step {t}: static handle equal", flush=True)
        assert sta.opt.inexact_chunks() == ref.opt.inexact_chunks() == 0
    finally:
        sta.close()
        ref.close()


def test_static_handle_equals_allocating_handle(torch_cuda):
    torch = torch_cuda
    first = _wl("static-first", [20000, 3000, 7000, 4], 1024, 8, 7, tu=[1, 2, 4, 6],
                tv=[0, 1, 3])
    second = _wl("static-second", [3000, 1000], 99, 4, 5, tu=[0, 2, 3], tv=[0, 4])  # unaligned
    assert second.n < first.n
    _run_pair(torch, first, defer=True)
    _run_pair(torch, second, defer=False)


def test_static_handle_limits(torch_cuda):
    """One live static handle per device; a configuration beyond the static
    scratch is rejected with ZO_ESCRATCH before anything is enqueued."""
    import harness
    import paper_2202_06009_amd as zo
    wl = _wl("static-limit", [4096, 1000], 1024, 4, 3, tu=[1], tv=[0])
    one = harness.GpuRun(wl, static=True)
    try:
        with pytest.raises(zo.ZoError) as e:
            harness.GpuRun(wl, static=True)
        assert e.value.status == zo.ZO_ESTATE
    finally:
        one.close()
    # 4 Mi elements in chunks of 16: 262,144 chunks, 21 bytes each > 4 MiB
    big = _wl("static-too-big", [1 << 22], 16, 4, 2, tu=[1], tv=[0])
    with pytest.raises(zo.ZoError) as e:
        harness.GpuRun(big, static=True)
    assert e.value.status == zo.ZO_ESCRATCH
    # the slot is free again
    again = harness.GpuRun(wl, static=True)
    again.close()
