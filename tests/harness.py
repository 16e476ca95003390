"""Drive the HIP library and the CPU oracle through the same synthetic
workload, step by step, and compare them.

The GPU side generates every input on the device (synth device fills); the
oracle side generates the same values on the host (synth host fills, bit
identical) for either the whole shard or a sample of chunks.  Every
computation of the method is local to a chunk, so the oracle run on a sample
of chunks reproduces exactly what a full run computes on those chunks.
"""
import numpy as np

import oracle as orc
import synth
from synth import configs as C


def round_to(values, grad_dtype):
    """Binary32 values rounded to nearest-even in the 16-bit gradient type
    (and back, exactly): what the GPU side receives, converted on the device
    by torch, and what the oracle is fed."""
    a = np.ascontiguousarray(values, dtype=np.float32)
    if grad_dtype == "f32":
        return a
    if grad_dtype == "f16":
        return a.astype(np.float16).astype(np.float32)
    b = a.view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)


def steps_kind(wl, t):
    """(sync, var): Algorithm 1 -- t in T_u, t in T_v.  Algorithm 4 -- a
    compressed step is t outside T_v, a full-precision step t in T_v."""
    if wl.algorithm == "frozen-variance":
        full = t in set(wl.tv)
        return (not full), full
    return (t in set(wl.tu)), (t in set(wl.tv))


# ---------------------------------------------------------------------------
# chunk sampling
# ---------------------------------------------------------------------------

def sample_chunks(lay, seg_off, budget_elems, stride_chunks=None):
    """Chunks to check at scale: the first and the last chunk of segments
    (every ragged tail is a last chunk), taken alternately from both ends of
    the model until the element budget is spent, plus every
    `stride_chunks`-th chunk."""
    seg_off = np.asarray(seg_off, dtype=np.int64)
    seg = np.searchsorted(seg_off, lay.cstart, side="right") - 1
    firsts = {}
    lasts = {}
    for c, sg in enumerate(seg):
        firsts.setdefault(int(sg), c)
        lasts[int(sg)] = c
    segs = sorted(firsts)
    order = []
    lo, hi = 0, len(segs) - 1
    while lo <= hi:
        order.append(segs[lo])
        if hi != lo:
            order.append(segs[hi])
        lo, hi = lo + 1, hi - 1
    chosen, total = set(), 0
    for sg in order:
        for c in (firsts[sg], lasts[sg]):
            if c in chosen:
                continue
            if chosen and total + int(lay.clen[c]) > budget_elems:
                continue
            chosen.add(c)
            total += int(lay.clen[c])
    if stride_chunks:
        chosen.update(range(stride_chunks // 2, lay.nchunks, stride_chunks))
    return np.array(sorted(chosen), dtype=np.int64)


# ---------------------------------------------------------------------------
# oracle run (full shard or a sample of chunks)
# ---------------------------------------------------------------------------

class OracleRun:
    def __init__(self, wl, chunk_ids=None, literal=False, grad_dtype="f32"):
        self.wl = wl
        self.grad_dtype = grad_dtype
        self.full = orc.Layout.from_segments(wl.seg_off, wl.chunk)
        if chunk_ids is None:
            chunk_ids = np.arange(self.full.nchunks, dtype=np.int64)
        self.ids = np.asarray(chunk_ids, dtype=np.int64)
        self.lay = orc.Layout.from_lengths(self.full.clen[self.ids])
        self.ranges = [(int(self.full.cstart[c]), int(self.full.clen[c])) for c in self.ids]
        self.wranges = [(int(self.full.cword[c]), int((self.full.clen[c] + 63) // 64))
                        for c in self.ids]
        x0 = self.gather_normal(C.STREAM_X, 0, wl.sigma_x)
        if wl.algorithm == "frozen-variance":
            self.worker = orc.FVWorker(self.lay, x0, wl.beta1, wl.beta2, wl.eps)
        else:
            self.worker = orc.Worker(self.lay, x0, wl.beta1, wl.beta2, wl.eps,
                                     literal_momentum=literal)

    def gather_normal(self, stream, step, sigma, per_mille=0, factor=1.0):
        k = synth.key(0, stream, step)
        ks = C.ksigma(sigma)
        if len(self.ranges) == 1 or self.lay.n == self.full.n:
            return synth.normal_host(self.full.n, 0, k, ks, per_mille, factor) \
                if self.lay.n == self.full.n else \
                synth.normal_host(self.ranges[0][1], self.ranges[0][0], k, ks, per_mille, factor)
        return np.concatenate([synth.normal_host(l, s, k, ks, per_mille, factor)
                               for s, l in self.ranges])

    def grad(self, t):
        wl = self.wl
        return round_to(self.gather_normal(C.STREAM_G, t, wl.sigma_g, wl.outlier_per_mille,
                                           wl.outlier_factor), self.grad_dtype)

    def gbar(self, t):
        wl = self.wl
        return round_to(self.gather_normal(C.STREAM_GBAR, t, wl.sigma_g, wl.outlier_per_mille,
                                           wl.outlier_factor), self.grad_dtype)

    def peers(self, t):
        wl = self.wl
        W = wl.world
        base = wl.peer_scale_base(t)
        words = np.zeros((W - 1, self.lay.nwords), np.uint64)
        scales = np.zeros((W - 1, self.lay.nchunks), np.float32)
        for w in range(1, W):
            kb = synth.key(w, C.STREAM_BITS, t)
            ks = synth.key(w, C.STREAM_SCALES, t)
            if self.lay.n == self.full.n:
                words[w - 1] = synth.bits_host(self.full.nwords, 0, kb)
                scales[w - 1] = synth.scales_host(self.full.nchunks, 0, ks, base)
            else:
                words[w - 1] = np.concatenate([synth.bits_host(nw, w0, kb)
                                               for w0, nw in self.wranges])
                scales[w - 1] = np.concatenate([synth.scales_host(1, int(c), ks, base)
                                                for c in self.ids])
        return words, scales

    def step(self, t):
        sync, var = steps_kind(self.wl, t)
        g = self.grad(t)
        gb = self.gbar(t) if var else None
        pw = ps = None
        if sync and self.wl.world > 1:
            pw, ps = self.peers(t)
        if self.wl.algorithm == "frozen-variance":
            return self.worker.step(self.wl.gamma(t), g, var, gbar=gb, peer_words=pw,
                                    peer_scales=ps)
        return self.worker.step(self.wl.gamma(t), g, sync, var, gbar=gb, peer_words=pw,
                                peer_scales=ps)


# ---------------------------------------------------------------------------
# GPU run
# ---------------------------------------------------------------------------

class GpuRun:
    STATE = ("x", "m", "v", "u", "err", "srv_err", "anchor")
    FV_STATE = ("x", "m", "v", "err", "srv_err")

    def __init__(self, wl, device="cuda", fused=True, srv_range=(0, -1), defer=False,
                 grad_dtype="f32"):
        import torch
        import paper_2202_06009_amd as zo
        self.torch, self.zo, self.wl, self.fused = torch, zo, wl, fused
        self.grad_dtype = grad_dtype
        self.gdt = {"f32": None, "f16": torch.float16, "bf16": torch.bfloat16}[grad_dtype]
        self.fv = wl.algorithm == "frozen-variance"
        self.keys = self.FV_STATE if self.fv else self.STATE
        n = wl.n
        f32 = dict(dtype=torch.float32, device=device)
        start, ln, word, nw = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
        self.nchunks, self.nwords = len(ln), nw
        self.state = {k: torch.empty(max(n, 4), **f32) for k in self.keys}
        self.g = torch.empty(max(n, 4), **f32)
        self.gb = torch.empty(max(n, 4), **f32)
        W = wl.world
        self.packed = torch.zeros((W, max(nw, 1)), dtype=torch.int64, device=device)
        self.scales = torch.zeros((W, max(self.nchunks, 1)), **f32)
        self.srv_packed = torch.zeros(max(nw, 1), dtype=torch.int64, device=device)
        self.srv_scales = torch.zeros(max(self.nchunks, 1), **f32)
        if n:
            synth.normal_dev(self.state["x"][:n], 0, synth.key(0, C.STREAM_X, 0),
                             C.ksigma(wl.sigma_x))
        self.opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=W,
                             chunk=wl.chunk, seg_off=wl.seg_off, tv=wl.tv, tu=wl.tu,
                             state=self.state, srv_chunk_begin=srv_range[0],
                             srv_chunk_end=srv_range[1], defer_sync_writes=defer,
                             algorithm=wl.algorithm, grad_dtype=grad_dtype)

    def fill_inputs(self, t):
        wl = self.wl
        n = wl.n
        sync, var = steps_kind(wl, t)
        if n:
            synth.normal_dev(self.g[:n], 0, synth.key(0, C.STREAM_G, t), C.ksigma(wl.sigma_g),
                             wl.outlier_per_mille, wl.outlier_factor)
            if var:
                synth.normal_dev(self.gb[:n], 0, synth.key(0, C.STREAM_GBAR, t),
                                 C.ksigma(wl.sigma_g), wl.outlier_per_mille, wl.outlier_factor)
        if self.gdt is not None:
            self.g_in, self.gb_in = self.g.to(self.gdt), self.gb.to(self.gdt)
        else:
            self.g_in, self.gb_in = self.g, self.gb
        if sync and self.nwords:
            base = wl.peer_scale_base(t)
            for w in range(1, wl.world):
                synth.bits_dev(self.packed[w], 0, synth.key(w, C.STREAM_BITS, t))
                synth.scales_dev(self.scales[w], 0, synth.key(w, C.STREAM_SCALES, t), base)

    def step(self, t, avg_debug=None):
        wl = self.wl
        sync, var = steps_kind(wl, t)
        self.fill_inputs(t)
        g = self.g_in
        gb = self.gb_in if var else None
        o = self.opt
        gam = wl.gamma(t)
        if self.fv:
            if var:
                o.fullprec_step(t, gam, gb)
                return
            o.compress_pack_ef(t, gam, g, self.packed[0], self.scales[0])
            o.unpack_average(t, self.packed, self.scales, self.srv_packed, self.srv_scales,
                             avg_debug)
            o.sync_update(t, self.srv_packed, self.srv_scales, None)
            return
        if not sync:
            o.local_step(t, gam, g, gb)
            return
        if self.fused:
            o.compress_pack_ef(t, gam, g, self.packed[0], self.scales[0])
        else:
            o.local_step(t, gam, g, None)
            o.compress_pack_ef(t, gam, None, self.packed[0], self.scales[0])
        o.unpack_average(t, self.packed, self.scales, self.srv_packed, self.srv_scales,
                         avg_debug)
        if self.fused:
            o.sync_update(t, self.srv_packed, self.srv_scales, gb)
        else:
            o.sync_update(t, self.srv_packed, self.srv_scales, None)
            if var:
                o.variance_update(t, gb)

    def close(self):
        self.opt.close()


# ---------------------------------------------------------------------------
# comparison
# ---------------------------------------------------------------------------

def gather_index(orun):
    """Global element and word indices of the oracle run's chunks."""
    el = np.concatenate([np.arange(s, s + l) for s, l in orun.ranges]) if orun.ranges \
        else np.zeros(0, np.int64)
    wd = np.concatenate([np.arange(w, w + k) for w, k in orun.wranges]) if orun.wranges \
        else np.zeros(0, np.int64)
    return el, wd


class Comparator:
    def __init__(self, grun, orun):
        import torch
        self.torch = torch
        self.grun, self.orun = grun, orun
        el, wd = gather_index(orun)
        self.full = orun.lay.n == orun.full.n
        dev = grun.g.device
        self.el = torch.as_tensor(el, device=dev)
        self.wd = torch.as_tensor(wd, device=dev)
        self.ch = torch.as_tensor(orun.ids, device=dev)

    def fetch(self, t, kind="elem"):
        if self.full:
            n = self.orun.full.n if kind == "elem" else (
                self.orun.full.nwords if kind == "word" else self.orun.full.nchunks)
            return t[:n].cpu().numpy()
        idx = {"elem": self.el, "word": self.wd, "chunk": self.ch}[kind]
        return t.index_select(0, idx).cpu().numpy()

    def check(self, t, out):
        """Compare every state after step t; returns a dict of mismatch counts
        (floats: -0 == +0; packed words: exact)."""
        bad = {}
        w = self.orun.worker
        self.torch.cuda.synchronize()
        for k in self.grun.keys:
            gpu = self.fetch(self.grun.opt.current(k))
            ref = getattr(w, k)
            if k == "srv_err" and not self.full:
                pass  # the server range is the whole shard: same indices as elements
            nbad = int(np.count_nonzero(~(gpu == ref)))
            if nbad:
                bad[k] = nbad
        if out:
            pw = self.fetch(self.grun.packed[0], "word").view(np.uint64)
            if not np.array_equal(pw, out["own_words"]):
                bad["own_words"] = int(np.count_nonzero(pw != out["own_words"]))
            ps = self.fetch(self.grun.scales[0], "chunk")
            if not np.array_equal(ps, out["own_scales"]):
                bad["own_scales"] = int(np.count_nonzero(ps != out["own_scales"]))
            sw = self.fetch(self.grun.srv_packed, "word").view(np.uint64)
            ref_sw = out["srv_words"]
            if not np.array_equal(sw, ref_sw):
                bad["srv_words"] = int(np.count_nonzero(sw != ref_sw))
            ss = self.fetch(self.grun.srv_scales, "chunk")
            if not np.array_equal(ss, out["srv_scales"]):
                bad["srv_scales"] = int(np.count_nonzero(ss != out["srv_scales"]))
        return bad


def run_parity(wl, steps=None, chunk_ids=None, fused=True, log=None, defer=False,
               materialize_at=(), grad_dtype="f32"):
    """Run both sides for `steps` steps; return per-step mismatch dicts.
    defer: deferred sync writes (the logical state is compared);
    materialize_at: steps after which the deferred writes are forced out;
    grad_dtype: element type of the gradients handed to the library."""
    grun = GpuRun(wl, fused=fused, defer=defer, grad_dtype=grad_dtype)
    orun = OracleRun(wl, chunk_ids, grad_dtype=grad_dtype)
    cmp_ = Comparator(grun, orun)
    report = []
    try:
        bad = cmp_.check(-1, None)
        report.append(bad)
        T = wl.steps if steps is None else steps
        for t in range(T):
            grun.step(t)
            if t in materialize_at:
                grun.opt.materialize()
            out = orun.step(t)
            bad = cmp_.check(t, out)
            if log:
                log(f"{wl.name} step {t}: {'ok' if not bad else bad}")
            report.append(bad)
            if bad:
                break
        inexact = grun.opt.inexact_chunks()
    finally:
        grun.close()
    return report, inexact
