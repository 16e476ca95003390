"""GPU edge cases: call order, argument errors, an empty shard, zero-gradient
segments, a shard of more than 2^31 parameters, the server restricted to a
chunk range, pad bits on input, the exact-sum condition, run-to-run
determinism."""
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


def _wl(segs=(4096, 1000, 3000), chunk=1024, world=4, T=6, tu=(1, 3, 4), tv=(0, 1, 4)):
    return C.Workload(name="edge", seg_off=C.offsets(list(segs)), world=world, chunk=chunk,
                      steps=T, tv=list(tv), tu=list(tu), gammas=[1e-4] * T, sigma_g=1e-3)


def test_call_order_is_enforced(torch_cuda):
    import harness
    import paper_2202_06009_amd as zo
    wl = _wl(tv=(0, 4))
    run = harness.GpuRun(wl)
    o = run.opt
    g, gb = run.g, run.gb
    run.fill_inputs(0)
    run.gb.copy_(run.g)
    try:
        with pytest.raises(zo.ZoError) as e:       # wrong step index
            o.local_step(1, 1e-4, g)
        assert e.value.status == zo.ZO_ESTATE
        with pytest.raises(zo.ZoError) as e:       # compress at a non-sync step
            o.compress_pack_ef(0, 1e-4, g, run.packed[0], run.scales[0])
        assert e.value.status == zo.ZO_ESTATE
        with pytest.raises(zo.ZoError) as e:       # gamma must be > 0
            o.local_step(0, 0.0, g)
        assert e.value.status == zo.ZO_EINVAL
        # a full-length gradient at an address that is not 16-byte aligned
        g_off = torch_cuda.empty(g.numel() + 1, dtype=g.dtype, device=g.device)[1:]
        g_off.copy_(g)
        with pytest.raises(zo.ZoError) as e:
            o.local_step(0, 1e-4, g_off)
        assert e.value.status == zo.ZO_EALIGN
        # the binding checks element types and sizes before the C ABI (which
        # takes bare pointers) is called
        for bad in (g[:-4], g.double(), g.half()):
            with pytest.raises(ValueError):
                o.local_step(0, 1e-4, bad)
        with pytest.raises(ValueError):
            o.compress_pack_ef(0, 1e-4, g, run.packed[0][:-1], run.scales[0])
        with pytest.raises(ValueError):
            o.unpack_average(0, run.packed[:-1], run.scales, run.srv_packed, run.srv_scales)
        with pytest.raises(ValueError):
            o.sync_update(0, run.srv_packed, run.srv_scales.double(), None)
        assert o.next_step == 0
        o.local_step(0, 1e-4, g)                   # t = 0 in T_v: variance still due
        with pytest.raises(zo.ZoError) as e:
            o.local_step(1, 1e-4, g)
        assert e.value.status == zo.ZO_ESTATE
        o.variance_update(0, gb)
        assert o.next_step == 1
        with pytest.raises(zo.ZoError) as e:       # gbar at a sync step's local half
            o.local_step(1, 1e-4, g, gb)
        assert e.value.status == zo.ZO_EINVAL
        with pytest.raises(zo.ZoError) as e:       # sync before the server half
            o.compress_pack_ef(1, 1e-4, g, run.packed[0], run.scales[0])
            o.sync_update(1, run.srv_packed, run.srv_scales, gb)
        assert e.value.status == zo.ZO_ESTATE
        o.unpack_average(1, run.packed, run.scales, run.srv_packed, run.srv_scales)
        with pytest.raises(zo.ZoError) as e:       # server half twice
            o.unpack_average(1, run.packed, run.scales, run.srv_packed, run.srv_scales)
        assert e.value.status == zo.ZO_ESTATE
        with pytest.raises(zo.ZoError) as e:       # gbar at a step not in T_v
            o.sync_update(1, run.srv_packed, run.srv_scales, gb)
        assert e.value.status == zo.ZO_EINVAL
        o.sync_update(1, run.srv_packed, run.srv_scales, None)
        assert o.next_step == 2 and o.gamma_sum == 0.0
        torch_cuda.cuda.synchronize()
    finally:
        run.close()


def test_empty_shard(torch_cuda):
    import harness
    wl = _wl(segs=(0,), chunk=64, world=2, T=3, tu=(1,), tv=(0,))
    run = harness.GpuRun(wl)
    try:
        assert run.opt.num_chunks == 0 and run.opt.packed_words == 0
        for t in range(3):
            run.step(t)
        torch_cuda.cuda.synchronize()
        assert run.opt.next_step == 3
    finally:
        run.close()


@pytest.mark.timeout(600)
def test_shard_beyond_2_31_elements(torch_cuda):
    """2,167,001,004 parameters in three segments, so element indices, packed
    bit indices and float4 indices pass 2^31 (the 64-bit index arithmetic of
    every kernel), in the benchmark's alternation of a local and a sync step
    with the variance update and deferred sync writes, W = 4.  Sampled: both
    ends of every segment, a stride, the chunks around element 2^31 and the
    ragged last chunk; every state and packed output after every step."""
    import harness
    import oracle as orc
    T = 4
    wl = C.Workload(name="beyond-2^31", seg_off=C.offsets([1_500_000_000, 667_000_004, 1000]),
                    world=4, chunk=16384, steps=T, tv=list(range(T)), tu=[1, 3],
                    gammas=[1e-4] * T, sigma_g=1e-3)
    assert wl.n > 2 ** 31
    lay = orc.Layout.from_segments(wl.seg_off, wl.chunk)
    ids = set(harness.sample_chunks(lay, wl.seg_off).tolist())
    b = int(np.searchsorted(lay.cstart, 2 ** 31, side="right")) - 1  # holds element 2^31
    ids.update(range(b - 2, min(b + 3, lay.nchunks)))
    ids.add(lay.nchunks - 1)
    ids = np.array(sorted(ids), dtype=np.int64)
    print(f"{wl.name}: d={wl.n}, {len(ids)} chunks sampled (chunk {b} holds element 2^31)",
          flush=True)
    report, inexact = harness.run_parity(wl, chunk_ids=ids, log=lambda m: print(m, flush=True),
                                         defer=True)
    for t, bad in enumerate(report):
        assert not bad, f"mismatch after step {t - 1}: {bad}"
    assert inexact == 0


@pytest.mark.parametrize("defer", [False, True], ids=["eager", "defer"])
def test_zero_gradient_segments(torch_cuda, defer):
    """Parameters whose gradient is exactly zero for the whole run (untouched
    embedding rows, frozen tensors): a segment of +0 and one of -0 gradients
    (and averaged gradients) next to a normal one, W = 3.  Up to the first
    sync their momentum and buffer stay zero, so that sync compresses exact
    zeros (scale 0, every sign +1: sign(+0) = sign(-0) = +1) and the server
    average there is the peers' alone; afterwards their momentum is the
    reconstructed average.  Every state and output against the oracle fed the
    same zeros, after every step."""
    import harness
    zero, negzero = (0, 4096), (7096, 8096)
    wl = _wl(segs=(4096, 3000, 1000), chunk=1024, world=3, T=8, tu=(1, 3, 4, 7),
             tv=(0, 1, 2, 5))
    grun = harness.GpuRun(wl, defer=defer)
    orun = harness.OracleRun(wl)
    fill = grun.fill_inputs

    def fill_zero(t):
        fill(t)
        for buf in (grun.g, grun.gb):  # binary32: these are the tensors handed over
            buf[zero[0]:zero[1]] = 0.0
            buf[negzero[0]:negzero[1]] = -0.0

    def zeroed(f):
        def h(t):
            a = np.array(f(t), dtype=np.float32, copy=True)
            a[zero[0]:zero[1]] = 0.0
            a[negzero[0]:negzero[1]] = -0.0
            return a
        return h

    grun.fill_inputs = fill_zero
    orun.grad, orun.gbar = zeroed(orun.grad), zeroed(orun.gbar)
    cmp_ = harness.Comparator(grun, orun)
    try:
        assert not cmp_.check(-1, None)
        for t in range(wl.steps):
            grun.step(t)
            out = orun.step(t)
            bad = cmp_.check(t, out)
            assert not bad, f"step {t}: {bad}"
            if t == min(wl.tu):
                # the +0 segment's four chunks: scale 0, all 64 words all ones
                own_s = grun.scales[0][:4].cpu().numpy()
                assert (own_s == 0).all(), own_s
                assert (grun.packed[0][:4 * 16].cpu().numpy() == -1).all()
                assert not orun.worker.err[zero[0]:zero[1]].any()
        assert grun.opt.inexact_chunks() == 0
    finally:
        cmp_.close()
        grun.close()


@pytest.mark.parametrize("chunk,world", [(1024, 8), (1021, 8), (4096, 128)],
                         ids=["C1024-W8", "C1021-W8", "C4096-W128"])
def test_server_range_matches_single_server(torch_cuda, chunk, world):
    """The server half restricted to a chunk range (one GPU's share in a
    sharded run) computes, on that range, exactly what the single server
    computes there: the lookup-table server, the plain server at a chunk
    length that is not a multiple of 4, and 16 worker groups."""
    import harness
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    wl = _wl(segs=(20000, 3000, 7000), chunk=chunk, world=world, T=4, tu=(0, 1, 2, 3), tv=(0,))
    full = harness.GpuRun(wl)
    _, ln, word, nw = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    c0, c1 = len(ln) // 4, 3 * len(ln) // 4 + 1  # an inner range, ragged chunks included
    part = harness.GpuRun(wl, srv_range=(c0, c1))
    try:
        rng_ = part.opt.server_range()
        assert rng_["chunk0"] == c0 and rng_["nchunks"] == c1 - c0
        w0, nwr = rng_["word0"], rng_["nwords"]
        e0, ne = rng_["elem0"], rng_["nelems"]
        W = wl.world
        for t in range(wl.steps):
            full.fill_inputs(t)
            full.opt.compress_pack_ef(t, wl.gamma(t), full.g, full.packed[0], full.scales[0])
            full.opt.unpack_average(t, full.packed, full.scales, full.srv_packed, full.srv_scales)
            # the share: packed inputs restricted to the range, slot-major
            part.fill_inputs(t)
            part.opt.compress_pack_ef(t, wl.gamma(t), part.g, part.packed[0], part.scales[0])
            rp = part.packed[:, w0:w0 + nwr].contiguous()
            rs = part.scales[:, c0:c1].contiguous()
            part.opt.unpack_average(t, rp, rs, part.srv_packed, part.srv_scales)
            torch.cuda.synchronize()
            assert torch.equal(part.srv_packed[w0:w0 + nwr], full.srv_packed[w0:w0 + nwr])
            assert torch.equal(part.srv_scales[c0:c1], full.srv_scales[c0:c1])
            assert torch.equal(part.state["srv_err"][:ne], full.state["srv_err"][e0:e0 + ne])
            full.opt.sync_update(t, full.srv_packed, full.srv_scales,
                                 full.gb if t in wl.tv else None)
            # the range's GPU cannot reconstruct alone; give it the full result
            part.srv_packed.copy_(full.srv_packed)
            part.srv_scales.copy_(full.srv_scales)
            part.opt.sync_update(t, part.srv_packed, part.srv_scales,
                                 part.gb if t in wl.tv else None)
        assert W == world
    finally:
        full.close()
        part.close()


def test_pad_bits_of_inputs_are_ignored(torch_cuda):
    """Two runs whose peer words differ only in pad bits (all clear versus all
    set) produce identical results."""
    import harness
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    wl = _wl(segs=(1000, 36, 4), chunk=100, world=5, T=2, tu=(0, 1), tv=(0,))
    _, ln, word, nw = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    mask = np.full(nw, np.uint64(0xFFFFFFFFFFFFFFFF), dtype=np.uint64)
    for c in range(len(ln)):
        rem = ln[c] % 64
        if rem:
            mask[word[c] + (ln[c] + 63) // 64 - 1] = np.uint64((1 << rem) - 1)
    data = torch.from_numpy(mask.view(np.int64)).cuda()
    runs = [harness.GpuRun(wl), harness.GpuRun(wl)]
    try:
        for t in range(wl.steps):
            for i, r in enumerate(runs):
                r.fill_inputs(t)
                if i == 0:
                    r.packed[1:] &= data
                else:
                    r.packed[1:] |= ~data
                gb = r.gb if t in wl.tv else None
                r.opt.compress_pack_ef(t, wl.gamma(t), r.g, r.packed[0], r.scales[0])
                r.opt.unpack_average(t, r.packed, r.scales, r.srv_packed, r.srv_scales)
                r.opt.sync_update(t, r.srv_packed, r.srv_scales, gb)
            torch.cuda.synchronize()
            for k in runs[0].state:
                assert torch.equal(runs[0].state[k], runs[1].state[k]), k
            assert torch.equal(runs[0].srv_packed, runs[1].srv_packed)
            # and the outputs' own pad bits are zero
            own = runs[0].packed[0].cpu().numpy().view(np.uint64)
            assert not np.any(own & ~mask)
            srv = runs[0].srv_packed.cpu().numpy().view(np.uint64)
            assert not np.any(srv & ~mask)
    finally:
        for r in runs:
            r.close()


def test_inexact_scales_are_counted(torch_cuda):
    import harness
    torch = torch_cuda
    wl = _wl(segs=(4096,), chunk=1024, world=4, T=2, tu=(0, 1), tv=())
    run = harness.GpuRun(wl)
    try:
        run.fill_inputs(0)
        run.opt.compress_pack_ef(0, wl.gamma(0), run.g, run.packed[0], run.scales[0])
        run.scales[1, 2] = 1.0e6        # 2^19 next to scales ~1e-8: span > 53 bits
        run.opt.unpack_average(0, run.packed, run.scales, run.srv_packed, run.srv_scales)
        assert run.opt.inexact_chunks() == 1
        # the flag stays set through later syncs whose scales are fine
        run.opt.sync_update(0, run.srv_packed, run.srv_scales, None)
        run.fill_inputs(1)
        run.opt.compress_pack_ef(1, wl.gamma(1), run.g, run.packed[0], run.scales[0])
        run.opt.unpack_average(1, run.packed, run.scales, run.srv_packed, run.srv_scales)
        assert run.opt.inexact_chunks() == 1
        torch.cuda.synchronize()
    finally:
        run.close()


def test_runs_are_deterministic(torch_cuda):
    import harness
    torch = torch_cuda
    wl = _wl(segs=(30000, 2000), chunk=2048, world=16, T=5, tu=(0, 2, 4), tv=(0, 1))
    a, b = harness.GpuRun(wl), harness.GpuRun(wl)
    try:
        for t in range(wl.steps):
            a.step(t)
            b.step(t)
        torch.cuda.synchronize()
        for k in a.state:
            assert torch.equal(a.state[k], b.state[k]), k
        assert torch.equal(a.srv_packed, b.srv_packed)
        assert torch.equal(a.packed[0], b.packed[0])
    finally:
        a.close()
        b.close()


def test_diag_stream_mix(torch_cuda):
    """The stream-mix diagnostic computes dst[w] = (sum of sources in order) + w."""
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    n = (1 << 20) + 12
    r = np.random.default_rng(7)
    host = [r.standard_normal(n).astype(np.float32) for _ in range(5)]
    src = [torch.from_numpy(h).cuda() for h in host]
    dst = [torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(4)]
    zo.zo_diag_stream(src, dst)
    torch.cuda.synchronize()
    acc = np.zeros(n, np.float32)
    for h in host:
        acc = (acc + h).astype(np.float32)
    for w in range(4):
        ref = (acc + np.float32(w)).astype(np.float32)
        assert np.array_equal(dst[w].cpu().numpy(), ref)
    # in place: sources 1 and 3 are rewritten from the sum of the old values,
    # next to three write-only arrays
    dst = [src[1], torch.empty_like(src[0]), src[3], torch.empty_like(src[0]),
           torch.empty_like(src[0])]
    zo.zo_diag_stream(src, dst)
    torch.cuda.synchronize()
    for w in range(5):
        ref = (acc + np.float32(w)).astype(np.float32)
        assert np.array_equal(dst[w].cpu().numpy(), ref), w


def test_server_pattern_diagnostic_keeps_the_error(torch_cuda):
    """zo_diag_server_pattern (the server's accesses without its arithmetic)
    rewrites the server error with exactly the bits it held, including -0 and
    a NaN payload, on a ragged layout; chunks of at most 1024 elements are
    rejected."""
    import paper_2202_06009_amd as zo
    torch = torch_cuda
    dev = torch.device("cuda", 0)
    seg = C.offsets([5000, 3 * 2048 + 100, 12])
    d, W = seg[-1], 5
    state = {k: torch.zeros(d, dtype=torch.float32, device=dev)
             for k in ("x", "m", "v", "u", "err", "srv_err", "anchor")}
    opt = zo.ZoAdam(beta1=0.9, beta2=0.999, eps=1e-8, world=W, chunk=2048, seg_off=seg,
                    tv=[], tu=[0], state=state)
    try:
        rng = np.random.default_rng(7)
        bits = rng.integers(0, 2**32, size=d, dtype=np.uint64).astype(np.uint32)
        bits[:8] = [0x80000000, 0x7fc01234, 0xff800000, 0, 1, 0x80000001, 0x3f800000, 0xbf800000]
        state["srv_err"].copy_(torch.from_numpy(bits.view(np.int32)).to(dev).view(torch.float32))
        before = state["srv_err"].view(torch.int32).clone()
        packed = torch.from_numpy(rng.integers(-2**62, 2**62, size=(W, opt.nwords),
                                               dtype=np.int64)).to(dev)
        opt.diag_server_pattern(packed)
        torch.cuda.synchronize()
        assert torch.equal(state["srv_err"].view(torch.int32), before)
    finally:
        opt.close()
    narrow = zo.ZoAdam(beta1=0.9, beta2=0.999, eps=1e-8, world=W, chunk=1024, seg_off=seg,
                       tv=[], tu=[0], state=state)
    try:
        with pytest.raises(zo.ZoError) as e:
            narrow.diag_server_pattern(
                torch.zeros((W, narrow.nwords), dtype=torch.int64, device=dev))
        assert e.value.status == zo.ZO_EINVAL
    finally:
        narrow.close()
