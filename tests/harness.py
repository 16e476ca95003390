"""Drive the HIP library and the CPU oracle through the same synthetic
workload, step by step, and compare them.

The GPU side generates every input on the device (synth device fills); the
oracle side generates the same values on the host (synth host fills, bit
identical) for either the whole shard or a sample of chunks.  Every
computation of the method is local to a chunk, so the oracle run on a sample
of chunks reproduces exactly what a full run computes on those chunks.
"""
import os

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

def sample_chunks(lay, seg_off, stride=50, min_frac=0.02):
    """Chunks to check at scale: every partial (ragged) chunk, the first and
    the last chunk of every segment, and every `stride`-th of the remaining
    chunks; the stride is lowered until the sample holds at least `min_frac`
    of the shard's elements."""
    seg_off = np.asarray(seg_off, dtype=np.int64)
    nch = lay.nchunks
    if nch == 0:
        return np.zeros(0, np.int64)
    seg = np.searchsorted(seg_off, lay.cstart, side="right") - 1
    first = np.ones(nch, bool)
    first[1:] = seg[1:] != seg[:-1]
    last = np.ones(nch, bool)
    last[:-1] = seg[:-1] != seg[1:]
    ragged = lay.clen != lay.clen.max()
    must = first | last | ragged
    rest = np.flatnonzero(~must)
    n = int(lay.clen.sum())
    s = max(1, int(stride))
    while True:
        pick = rest[s // 2::s]
        chosen = np.union1d(np.flatnonzero(must), pick)
        if s == 1 or int(lay.clen[chosen].sum()) >= min_frac * n:
            return chosen.astype(np.int64)
        s = max(1, (s * 4) // 5)


def oracle_threads():
    """Threads for the oracle side (ZO_ORACLE_THREADS, else at most 16 of the
    cores this process may use)."""
    env = os.environ.get("ZO_ORACLE_THREADS")
    if env:
        return max(1, int(env))
    return max(1, min(16, len(os.sched_getaffinity(0))))


# ---------------------------------------------------------------------------
# oracle run (full shard or a sample of chunks)
# ---------------------------------------------------------------------------

def _runs(ids):
    """Split sorted chunk ids into maximal runs of consecutive ids:
    (first id, count) pairs."""
    if len(ids) == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    brk = np.flatnonzero(np.diff(ids) != 1) + 1
    starts = np.concatenate([[0], brk])
    ends = np.concatenate([brk, [len(ids)]])
    return ids[starts].astype(np.int64), (ends - starts).astype(np.int64)


class OracleRun:
    """The oracle on the chunks `chunk_ids` (sorted; default: every chunk) of a
    workload, laid out back to back; inputs are generated at their global
    indices."""

    def __init__(self, wl, chunk_ids=None, literal=False, grad_dtype="f32"):
        self.wl = wl
        self.grad_dtype = grad_dtype
        self.full = orc.Layout.from_segments(wl.seg_off, wl.chunk)
        if chunk_ids is None:
            chunk_ids = np.arange(self.full.nchunks, dtype=np.int64)
        self.ids = np.asarray(chunk_ids, dtype=np.int64)
        assert np.all(np.diff(self.ids) > 0), "chunk ids must be sorted and distinct"
        self.lay = orc.Layout.from_lengths(self.full.clen[self.ids])
        self.n = self.lay.n
        f = self.full
        self.ranges = [(int(f.cstart[c]), int(f.clen[c])) for c in self.ids]
        self.wranges = [(int(f.cword[c]), int((f.clen[c] + 63) // 64)) for c in self.ids]
        # maximal runs of consecutive chunks: element, word and chunk ranges
        c0, cnt = _runs(self.ids)
        cl = c0 + cnt - 1
        self.run_c0, self.run_nc = c0, cnt
        self.run_e0 = f.cstart[c0] if len(c0) else np.zeros(0, np.int64)
        self.run_ne = (f.cstart[cl] + f.clen[cl] - self.run_e0) if len(c0) else self.run_e0
        self.run_w0 = f.cword[c0] if len(c0) else np.zeros(0, np.int64)
        self.run_nw = (f.cword[cl] + (f.clen[cl] + 63) // 64 - self.run_w0) if len(c0) \
            else self.run_w0
        x0 = self.gather_normal(C.STREAM_X, 0, wl.sigma_x)
        if wl.algorithm == "frozen-variance":
            self.worker = orc.FVWorker(self.lay, x0, wl.beta1, wl.beta2, wl.eps)
        else:
            self.worker = orc.Worker(self.lay, x0, wl.beta1, wl.beta2, wl.eps,
                                     literal_momentum=literal)

    def gather_normal(self, stream, step, sigma, per_mille=0, factor=1.0):
        k = synth.key(0, stream, step)
        return synth.normal_host_ranges(self.run_e0, self.run_ne, k, C.ksigma(sigma),
                                        per_mille, factor)

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
        words = np.empty((W - 1, self.lay.nwords), np.uint64)
        scales = np.empty((W - 1, self.lay.nchunks), np.float32)
        for w in range(1, W):
            words[w - 1] = synth.bits_host_ranges(self.run_w0, self.run_nw,
                                                  synth.key(w, C.STREAM_BITS, t))
            scales[w - 1] = synth.scales_host_ranges(self.run_c0, self.run_nc,
                                                     synth.key(w, C.STREAM_SCALES, t), base)
        return words, scales

    def state(self, k):
        return getattr(self.worker, k)

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


class ParallelOracle:
    """The oracle on a set of chunks, split into `parts` contiguous pieces of
    about equal element counts, each an OracleRun stepped on its own thread
    (the oracle and the input fills are C called through ctypes, which drops
    the GIL).  Every computation of the method is local to a chunk, so the
    pieces together compute exactly what one run over all the chunks would;
    states and outputs are the pieces' in chunk order."""

    OUT_KEYS = ("own_words", "own_scales", "srv_words", "srv_scales")

    def __init__(self, wl, chunk_ids=None, parts=None, grad_dtype="f32"):
        from concurrent.futures import ThreadPoolExecutor
        self.wl = wl
        self.full = orc.Layout.from_segments(wl.seg_off, wl.chunk)
        if chunk_ids is None:
            chunk_ids = np.arange(self.full.nchunks, dtype=np.int64)
        ids = np.unique(np.asarray(chunk_ids, dtype=np.int64))
        parts = max(1, min(parts or oracle_threads(), len(ids)))
        cum = np.cumsum(self.full.clen[ids]) if len(ids) else np.zeros(0, np.int64)
        tot = int(cum[-1]) if len(ids) else 0
        cuts = [0] + [int(np.searchsorted(cum, tot * k / parts)) for k in range(1, parts)] + \
            [len(ids)]
        pieces = [ids[a:b] for a, b in zip(cuts[:-1], cuts[1:]) if b > a] or [ids]
        self.runs = [OracleRun(wl, p, grad_dtype=grad_dtype) for p in pieces]
        self.ids = ids
        self.n = sum(r.n for r in self.runs)
        self.ranges = [rg for r in self.runs for rg in r.ranges]
        self.wranges = [rg for r in self.runs for rg in r.wranges]
        self.pool = ThreadPoolExecutor(max_workers=len(self.runs))

    def step(self, t):
        outs = list(self.pool.map(lambda r: r.step(t), self.runs))
        if not outs[0]:
            return outs[0]
        return {k: np.concatenate([o[k] for o in outs]) for k in self.OUT_KEYS}

    def state(self, k):
        return np.concatenate([r.state(k) for r in self.runs])

    def close(self):
        self.pool.shutdown()


# ---------------------------------------------------------------------------
# GPU run
# ---------------------------------------------------------------------------

class GpuRun:
    STATE = ("x", "m", "v", "u", "err", "srv_err", "anchor")
    FV_STATE = ("x", "m", "v", "err", "srv_err")

    def __init__(self, wl, device="cuda", fused=True, srv_range=(0, -1), defer=False,
                 grad_dtype="f32", static=False):
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
                             algorithm=wl.algorithm, grad_dtype=grad_dtype, static=static)

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


def _mismatches(gpu, ref):
    """Elements that differ (binary32: -0 == +0; integers: exact)."""
    return int(np.count_nonzero(~(gpu == ref)))


class Comparator:
    def __init__(self, grun, orun):
        import torch
        from concurrent.futures import ThreadPoolExecutor
        self.torch = torch
        self.grun, self.orun = grun, orun
        el, wd = gather_index(orun)
        self.full = orun.n == orun.full.n
        dev = grun.g.device
        self.el = torch.as_tensor(el, device=dev)
        self.wd = torch.as_tensor(wd, device=dev)
        self.ch = torch.as_tensor(orun.ids, device=dev)
        self.pool = ThreadPoolExecutor(max_workers=4)

    def fetch(self, t, kind="elem"):
        if self.full:
            n = self.orun.full.n if kind == "elem" else (
                self.orun.full.nwords if kind == "word" else self.orun.full.nchunks)
            return t[:n].cpu().numpy()
        idx = {"elem": self.el, "word": self.wd, "chunk": self.ch}[kind]
        return t.index_select(0, idx).cpu().numpy()

    def check(self, t, out):
        """Compare every state after step t; returns a dict of mismatch counts
        (floats: -0 == +0; packed words: exact).  The server range is the
        whole shard, so the server error has the elements' indices."""
        self.torch.cuda.synchronize()
        pairs = {}
        for k in self.grun.keys:
            pairs[k] = (self.fetch(self.grun.opt.current(k)), self.orun.state(k))
        if out:
            pairs["own_words"] = (self.fetch(self.grun.packed[0], "word").view(np.uint64),
                                  out["own_words"])
            pairs["own_scales"] = (self.fetch(self.grun.scales[0], "chunk"), out["own_scales"])
            pairs["srv_words"] = (self.fetch(self.grun.srv_packed, "word").view(np.uint64),
                                  out["srv_words"])
            pairs["srv_scales"] = (self.fetch(self.grun.srv_scales, "chunk"), out["srv_scales"])
        counts = dict(zip(pairs, self.pool.map(lambda kv: _mismatches(*kv), pairs.values())))
        return {k: v for k, v in counts.items() if v}

    def close(self):
        self.pool.shutdown()


def run_parity(wl, steps=None, chunk_ids=None, fused=True, log=None, defer=False,
               materialize_at=(), grad_dtype="f32"):
    """Run both sides for `steps` steps; return per-step mismatch dicts.
    defer: deferred sync writes (the logical state is compared);
    materialize_at: steps after which the deferred writes are forced out;
    grad_dtype: element type of the gradients handed to the library."""
    grun = GpuRun(wl, fused=fused, defer=defer, grad_dtype=grad_dtype)
    orun = ParallelOracle(wl, chunk_ids, grad_dtype=grad_dtype)
    cmp_ = Comparator(grun, orun)
    if log:
        log(f"{wl.name}: oracle on {len(orun.ids)} of {orun.full.nchunks} chunks "
            f"({orun.n} of {orun.full.n} elements, "
            f"{int((orun.full.clen[orun.ids] != wl.chunk).sum())} of "
            f"{int((orun.full.clen != wl.chunk).sum())} ragged chunks), "
            f"{len(orun.runs)} threads")
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
        cmp_.close()
        orun.close()
        grun.close()
    return report, inexact
