"""CPU oracle of 0/1 Adam -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
(``paper_2202_06009_amd``) and imports nothing from it.

The arithmetic lives in ``zo_oracle.c`` (plain single-threaded C, binary32
with every rounding pinned); this module only marshals numpy arrays and
orders the calls the way Algorithm 1 of the paper orders its lines
(``Worker``; ``FVWorker`` does the same for Algorithm 4):
momentum / model / buffer, then the sync block (Algorithm 2 worker half, the
server half, momentum approximation and model reconstruction), then the
variance block.  ``brute_adam`` holds an independent binary64 Adam (the
paper's Equation 2) used to pin the oracle.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_DEFAULT_LIB = os.path.join(HERE, "liboracle.so")
# ZO_ORACLE_LIB: another build of the oracle's source (the mutation tests
# load deliberately broken copies to show that the pins catch them)
_LIB_PATH = os.environ.get("ZO_ORACLE_LIB") or _DEFAULT_LIB

ZR_OK = 0
ZR_EINVAL = -1
ZR_EINEXACT = -6

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_u64p = np.ctypeslib.ndpointer(dtype=np.uint64, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")


class _Params(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("c1", ctypes.c_float),
                ("c2", ctypes.c_float), ("literal_momentum", ctypes.c_int32)]


class _State(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("m", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("u", ctypes.c_void_p), ("anchor", ctypes.c_void_p),
                ("gamma_sum", ctypes.c_float)]


def _load():
    if _LIB_PATH == _DEFAULT_LIB and not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, f32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
    lib.zr_count_chunks.argtypes = [i32, _i64p, i32]
    lib.zr_count_chunks.restype = i64
    lib.zr_build_chunks.argtypes = [i32, _i64p, i32, _i64p, _i64p, _i64p]
    lib.zr_build_chunks.restype = i64
    lib.zr_tree_abs_sum.argtypes = [_f32p, i64]
    lib.zr_tree_abs_sum.restype = f32
    lib.zr_compress_chunk.argtypes = [_f32p, i64, _u8p]
    lib.zr_compress_chunk.restype = f32
    lib.zr_pack_chunk.argtypes = [_u8p, i64, _u64p]
    lib.zr_pack_chunk.restype = None
    lib.zr_unpack_chunk.argtypes = [_u64p, i64, _u8p]
    lib.zr_unpack_chunk.restype = None
    lib.zr_ef_compress.argtypes = [i64, _i64p, _i64p, _i64p, _f32p, _f32p, _u64p, _f32p]
    lib.zr_ef_compress.restype = ctypes.c_int
    lib.zr_server.argtypes = [i32, i64, i64, _i64p, _i64p, _i64p, _u64p, i64, _f32p, i64,
                              _f32p, _u64p, _f32p, vp]
    lib.zr_server.restype = ctypes.c_int
    lib.zr_decompress.argtypes = [i64, _i64p, _i64p, _i64p, _u64p, _f32p, _f32p]
    lib.zr_decompress.restype = None
    lib.zr_dense_average.argtypes = [i32, i64, _f32p, _f32p]
    lib.zr_dense_average.restype = ctypes.c_int
    lib.zr_params_init.argtypes = [ctypes.POINTER(_Params), f32, f32, f32, i32]
    lib.zr_params_init.restype = None
    lib.zr_half_step.argtypes = [ctypes.POINTER(_Params), ctypes.POINTER(_State), i64, f32, _f32p]
    lib.zr_half_step.restype = None
    lib.zr_sync_dense.argtypes = [ctypes.POINTER(_Params), ctypes.POINTER(_State), i64, _f32p]
    lib.zr_sync_dense.restype = None
    lib.zr_variance.argtypes = [ctypes.POINTER(_Params), ctypes.POINTER(_State), i64, _f32p]
    lib.zr_variance.restype = None
    lib.zr_fv_step.argtypes = [ctypes.POINTER(_Params), _f32p, _f32p, _f32p, i64, f32, _f32p,
                               i32]
    lib.zr_fv_step.restype = None
    return lib


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = _load()
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc):
    if rc == ZR_EINEXACT:
        raise OracleError("server sum over workers was not exact in binary64")
    if rc != ZR_OK:
        raise OracleError(f"oracle error {rc}")


# ---------------------------------------------------------------------------
# Layout
# ---------------------------------------------------------------------------

class Layout:
    """Chunk table of a flat shard: every segment is cut into chunks of at most
    ``chunk`` elements; chunk c starts at ``cstart[c]``, has ``clen[c]``
    elements and owns packed words ``cword[c] .. cword[c] + ceil(clen/64)``."""

    def __init__(self, cstart, clen, cword, nwords, n):
        self.cstart = np.ascontiguousarray(cstart, dtype=np.int64)
        self.clen = np.ascontiguousarray(clen, dtype=np.int64)
        self.cword = np.ascontiguousarray(cword, dtype=np.int64)
        self.nchunks = int(len(self.clen))
        self.nwords = int(nwords)
        self.n = int(n)

    @classmethod
    def from_segments(cls, seg_off, chunk):
        seg = np.ascontiguousarray(seg_off, dtype=np.int64)
        nseg = len(seg) - 1
        nch = lib().zr_count_chunks(nseg, seg, int(chunk))
        cs = np.zeros(nch, np.int64)
        cl = np.zeros(nch, np.int64)
        cw = np.zeros(nch, np.int64)
        nw = lib().zr_build_chunks(nseg, seg, int(chunk), cs, cl, cw)
        return cls(cs, cl, cw, nw, int(seg[-1]))

    @classmethod
    def from_lengths(cls, lengths):
        """A compact shard made of the given chunk lengths back to back (used to
        run the oracle on a sample of another layout's chunks)."""
        cl = np.ascontiguousarray(lengths, dtype=np.int64)
        cs = np.concatenate([[0], np.cumsum(cl)[:-1]]).astype(np.int64)
        words = (cl + 63) // 64
        cw = np.concatenate([[0], np.cumsum(words)[:-1]]).astype(np.int64)
        return cls(cs, cl, cw, int(words.sum()), int(cl.sum()))


# ---------------------------------------------------------------------------
# Equation 3 and packing on single chunks
# ---------------------------------------------------------------------------

def tree_abs_sum(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return np.float32(lib().zr_tree_abs_sum(a, len(a)))


def compress_chunk(a):
    """C[a] of Equation 3 on one chunk -> (scale, bits with 1 meaning +1)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = np.zeros(len(a), np.uint8)
    s = lib().zr_compress_chunk(a, len(a), bits)
    return np.float32(s), bits


def pack_chunk(bits):
    bits = np.ascontiguousarray(bits, dtype=np.uint8)
    words = np.zeros((len(bits) + 63) // 64, np.uint64)
    lib().zr_pack_chunk(bits, len(bits), words)
    return words


def unpack_chunk(words, n):
    words = np.ascontiguousarray(words, dtype=np.uint64)
    bits = np.zeros(n, np.uint8)
    lib().zr_unpack_chunk(words, n, bits)
    return bits


# ---------------------------------------------------------------------------
# Algorithm 2
# ---------------------------------------------------------------------------

def ef_compress(layout, z, delta):
    """Worker half of Algorithm 2 on every chunk. Updates ``delta`` in place and
    returns (packed words, scales)."""
    words = np.zeros(layout.nwords, np.uint64)
    scales = np.zeros(layout.nchunks, np.float32)
    _check(lib().zr_ef_compress(layout.nchunks, layout.cstart, layout.clen, layout.cword,
                                np.ascontiguousarray(z, np.float32), delta, words, scales))
    return words, scales


def server(layout, words_w, scales_w, srv_delta, c0=0, c1=None, want_avg=False):
    """Server half of Algorithm 2 over chunks [c0, c1).

    ``words_w`` is [W, nwords_in_range] and ``scales_w`` is [W, nchunks_in_range];
    slot w is worker w.  ``srv_delta`` (updated in place) covers the range's
    elements.  Returns (server words over the whole layout, server scales over
    the whole layout, averages or None); only the range is written."""
    c1 = layout.nchunks if c1 is None else c1
    words_w = np.ascontiguousarray(words_w, dtype=np.uint64)
    scales_w = np.ascontiguousarray(scales_w, dtype=np.float32)
    W = words_w.shape[0]
    srv_words = np.zeros(layout.nwords, np.uint64)
    srv_scales = np.zeros(layout.nchunks, np.float32)
    avg = np.zeros(len(srv_delta), np.float32) if want_avg else None
    _check(lib().zr_server(W, c0, c1, layout.cstart, layout.clen, layout.cword,
                           words_w, words_w.shape[1], scales_w, scales_w.shape[1],
                           srv_delta, srv_words, srv_scales,
                           avg.ctypes.data if avg is not None else None))
    return srv_words, srv_scales, avg


def decompress(layout, words, scales):
    out = np.zeros(layout.n, np.float32)
    lib().zr_decompress(layout.nchunks, layout.cstart, layout.clen, layout.cword,
                        np.ascontiguousarray(words, np.uint64),
                        np.ascontiguousarray(scales, np.float32), out)
    return out


def dense_average(z_w):
    z_w = np.ascontiguousarray(z_w, dtype=np.float32)
    out = np.zeros(z_w.shape[1], np.float32)
    _check(lib().zr_dense_average(z_w.shape[0], z_w.shape[1], z_w, out))
    return out


# ---------------------------------------------------------------------------
# Algorithm 1 (one worker) and the single-GPU formulation of a step
# ---------------------------------------------------------------------------

class Worker:
    """One worker's optimizer state under Algorithm 1: model x, momentum m,
    variance v, buffer u, worker error delta (Algorithm 2), server error
    (when this worker also plays the server), anchor x_{t'} and Gamma."""

    def __init__(self, layout, x0, beta1=0.9, beta2=0.999, eps=1e-8, literal_momentum=False,
                 srv_range=None):
        self.layout = layout
        n = layout.n
        self.params = _Params()
        lib().zr_params_init(ctypes.byref(self.params), beta1, beta2, eps,
                             1 if literal_momentum else 0)
        self.x = np.array(x0, dtype=np.float32, copy=True)
        self.m = np.zeros(n, np.float32)
        self.v = np.zeros(n, np.float32)
        self.u = np.zeros(n, np.float32)
        self.err = np.zeros(n, np.float32)
        self.anchor = self.x.copy()
        c0, c1 = srv_range if srv_range is not None else (0, layout.nchunks)
        self.srv_range = (c0, c1)
        ne = (int(layout.cstart[c1 - 1] + layout.clen[c1 - 1]) - int(layout.cstart[c0])
              if c1 > c0 else 0)
        self.srv_err = np.zeros(ne, np.float32)
        self.gamma_sum = np.float32(0.0)

    def _state(self):
        st = _State()
        st.x = self.x.ctypes.data
        st.m = self.m.ctypes.data
        st.v = self.v.ctypes.data
        st.u = self.u.ctypes.data
        st.anchor = self.anchor.ctypes.data
        st.gamma_sum = float(self.gamma_sum)
        return st

    def half_step(self, gamma, g):
        """Momentum, model and buffer lines (every step)."""
        st = self._state()
        lib().zr_half_step(ctypes.byref(self.params), ctypes.byref(st), self.layout.n,
                           float(gamma), np.ascontiguousarray(g, np.float32))
        self.gamma_sum = np.float32(st.gamma_sum)

    def compress(self):
        """Worker half of Algorithm 2 on u_{t+1/2}."""
        return ef_compress(self.layout, self.u, self.err)

    def sync_dense(self, ubar):
        """Sync lines given the averaged buffer."""
        st = self._state()
        lib().zr_sync_dense(ctypes.byref(self.params), ctypes.byref(st), self.layout.n,
                            np.ascontiguousarray(ubar, np.float32))
        self.gamma_sum = np.float32(st.gamma_sum)

    def sync(self, srv_words, srv_scales):
        self.sync_dense(decompress(self.layout, srv_words, srv_scales))

    def variance(self, gbar):
        """Variance line at t in T_v."""
        st = self._state()
        lib().zr_variance(ctypes.byref(self.params), ctypes.byref(st), self.layout.n,
                          np.ascontiguousarray(gbar, np.float32))

    def snapshot(self):
        return {k: getattr(self, k).copy() for k in
                ("x", "m", "v", "u", "err", "srv_err", "anchor")} | {
                    "gamma_sum": np.float32(self.gamma_sum)}

    def step(self, gamma, g, sync, var, gbar=None, peer_words=None, peer_scales=None,
             compress=True, peer_dense=None):
        """One step of Algorithm 1 for worker 0 in the single-GPU formulation:
        the other W-1 workers exist only as their packed sign buffers
        ``peer_words`` [W-1, nwords] and scales ``peer_scales`` [W-1, nchunks]
        (or, with compression off, their dense buffers ``peer_dense``).

        Returns a dict with the own and server packed outputs at sync steps."""
        out = {}
        self.half_step(gamma, g)
        if sync:
            if compress:
                own_w, own_s = self.compress()
                if peer_words is not None and len(peer_words):
                    words_w = np.concatenate([own_w[None, :], peer_words], axis=0)
                    scales_w = np.concatenate([own_s[None, :], peer_scales], axis=0)
                else:
                    words_w, scales_w = own_w[None, :], own_s[None, :]
                sw, ss, _ = server(self.layout, words_w, scales_w, self.srv_err)
                self.sync(sw, ss)
                out.update(own_words=own_w, own_scales=own_s, srv_words=sw, srv_scales=ss)
            else:
                z = self.u[None, :] if peer_dense is None else np.concatenate(
                    [self.u[None, :], peer_dense], axis=0)
                self.sync_dense(dense_average(z))
        if var:
            self.variance(g if gbar is None else gbar)
        return out


class FVWorker:
    """One worker's state under Algorithm 4 (the frozen-variance framework;
    1-bit Adam when T_v is a prefix of the steps): model x, momentum m,
    variance v, worker error delta and server error of Algorithm 2, which
    compresses the gradients at every step outside T_v."""

    def __init__(self, layout, x0, beta1=0.9, beta2=0.999, eps=1e-8):
        self.layout = layout
        n = layout.n
        self.params = _Params()
        lib().zr_params_init(ctypes.byref(self.params), beta1, beta2, eps, 0)
        self.x = np.array(x0, dtype=np.float32, copy=True)
        self.m = np.zeros(n, np.float32)
        self.v = np.zeros(n, np.float32)
        self.err = np.zeros(n, np.float32)
        self.srv_err = np.zeros(n, np.float32)

    def apply(self, gamma, gbar, update_v):
        lib().zr_fv_step(ctypes.byref(self.params), self.x, self.m, self.v, self.layout.n,
                         float(gamma), np.ascontiguousarray(gbar, np.float32),
                         1 if update_v else 0)

    def step(self, gamma, g, full, gbar=None, peer_words=None, peer_scales=None):
        """One step for worker 0.  full (t in T_v): gbar is the full-precision
        average.  Otherwise g is compressed with the worker error, averaged
        with the peers' packed buffers by the server (with the server error)
        and the server's compressed average is the step's gradient.
        Returns the own and server packed outputs of a compressed step."""
        if full:
            self.apply(gamma, g if gbar is None else gbar, True)
            return {}
        own_w, own_s = ef_compress(self.layout, g, self.err)
        if peer_words is not None and len(peer_words):
            words_w = np.concatenate([own_w[None, :], peer_words], axis=0)
            scales_w = np.concatenate([own_s[None, :], peer_scales], axis=0)
        else:
            words_w, scales_w = own_w[None, :], own_s[None, :]
        sw, ss, _ = server(self.layout, words_w, scales_w, self.srv_err)
        self.apply(gamma, decompress(self.layout, sw, ss), False)
        return dict(own_words=own_w, own_scales=own_s, srv_words=sw, srv_scales=ss)

