"""Python binding of the 0/1 Adam hot-path library (``libzoadam.so``).

Argument marshalling only: every step of the optimizer runs in the HIP
kernels behind the C ABI declared in ``include/zo_adam.h``.  Functions keep
the C names (``zo_adam_init``, ``zo_local_step``, ...); ``ZoAdam`` wraps a
handle for convenience.  Device buffers are torch tensors (PyTorch provides
device memory and streams only).  There is no fallback: if the library is not
built, every call raises.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libzoadam.so")

ZO_OK, ZO_EINVAL, ZO_EALIGN, ZO_ESTATE, ZO_EHIP, ZO_ENOMEM, ZO_ESCRATCH = 0, -1, -2, -3, -4, -5, -6
ZO_ALG_ZERO_ONE_ADAM, ZO_ALG_FROZEN_VARIANCE = 0, 1
ZO_DTYPE_F32, ZO_DTYPE_F16, ZO_DTYPE_BF16 = 0, 1, 2
GRAD_DTYPES = {"f32": ZO_DTYPE_F32, "f16": ZO_DTYPE_F16, "bf16": ZO_DTYPE_BF16}
ALGORITHMS = {"zero-one": ZO_ALG_ZERO_ONE_ADAM, "frozen-variance": ZO_ALG_FROZEN_VARIANCE}

# Every function the header declares (checked by the CPU export test).
EXPORTS = (
    "zo_adam_init", "zo_adam_init_static", "zo_adam_destroy", "zo_set_stream", "zo_local_step",
    "zo_compress_pack_ef", "zo_unpack_average", "zo_sync_update", "zo_variance_update",
    "zo_fullprec_step", "zo_materialize", "zo_state_location", "zo_read_state", "zo_num_chunks",
    "zo_packed_words",
    "zo_server_range", "zo_chunk_table", "zo_gamma_sum", "zo_next_step", "zo_inexact_chunks",
    "zo_strerror", "zo_last_hip_error", "zo_diag_divsqrt", "zo_diag_copy", "zo_diag_stream",
    "zo_diag_server_pattern",
    "zo_config_check", "zo_plan_num_chunks", "zo_plan_chunks",
)


class ZoError(RuntimeError):
    def __init__(self, status, where, detail=""):
        self.status = status
        msg = f"{where}: {strerror(status)} ({status})"
        if detail:
            msg += f": {detail}"
        super().__init__(msg)


class _Config(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("world", ctypes.c_int32), ("chunk", ctypes.c_int32), ("n", ctypes.c_int64),
                ("nseg", ctypes.c_int32), ("seg_off", ctypes.POINTER(ctypes.c_int64)),
                ("ntv", ctypes.c_int32), ("tv", ctypes.POINTER(ctypes.c_int64)),
                ("ntu", ctypes.c_int32), ("tu", ctypes.POINTER(ctypes.c_int64)),
                ("srv_chunk_begin", ctypes.c_int64), ("srv_chunk_end", ctypes.c_int64),
                ("defer_sync_writes", ctypes.c_int32), ("algorithm", ctypes.c_int32),
                ("grad_dtype", ctypes.c_int32)]


class _State(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in ("x", "m", "v", "u", "err", "srv_err", "anchor")]


_lib = None


def lib():
    """Load the library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, f32, ci = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                 ctypes.c_float, ctypes.c_int)
        pi64 = ctypes.POINTER(ctypes.c_int64)
        sig = {
            "zo_adam_init": ([ctypes.POINTER(vp), ctypes.POINTER(_Config),
                              ctypes.POINTER(_State), vp], ci),
            "zo_adam_init_static": ([ctypes.POINTER(vp), ctypes.POINTER(_Config),
                                     ctypes.POINTER(_State), vp], ci),
            "zo_adam_destroy": ([vp], ci),
            "zo_set_stream": ([vp, vp], ci),
            "zo_local_step": ([vp, i64, f32, vp, vp], ci),
            "zo_compress_pack_ef": ([vp, i64, f32, vp, vp, vp], ci),
            "zo_unpack_average": ([vp, i64, vp, vp, vp, vp, vp], ci),
            "zo_sync_update": ([vp, i64, vp, vp, vp], ci),
            "zo_variance_update": ([vp, i64, vp], ci),
            "zo_materialize": ([vp], ci),
            "zo_fullprec_step": ([vp, i64, f32, vp], ci),
            "zo_read_state": ([vp, i32, vp], ci),
            "zo_state_location": ([vp, ctypes.POINTER(vp), ctypes.POINTER(i32),
                                   ctypes.POINTER(f32)], ci),
            "zo_num_chunks": ([vp], i64),
            "zo_packed_words": ([vp], i64),
            "zo_server_range": ([vp, pi64, pi64, pi64, pi64, pi64, pi64], ci),
            "zo_chunk_table": ([vp, vp, vp, vp], ci),
            "zo_gamma_sum": ([vp], f32),
            "zo_next_step": ([vp], i64),
            "zo_inexact_chunks": ([vp, pi64], ci),
            "zo_strerror": ([ci], ctypes.c_char_p),
            "zo_last_hip_error": ([vp], ctypes.c_char_p),
            "zo_diag_divsqrt": ([vp, vp, vp, vp, i64, vp], ci),
            "zo_diag_copy": ([vp, vp, i64, ci, vp], ci),
            "zo_diag_stream": ([vp, i32, vp, i32, i64, vp], ci),
            "zo_diag_server_pattern": ([vp, vp], ci),
            "zo_config_check": ([ctypes.POINTER(_Config)], ci),
            "zo_plan_num_chunks": ([i32, vp, i32], i64),
            "zo_plan_chunks": ([i32, vp, i32, vp, vp, vp], i64),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def strerror(status):
    return lib().zo_strerror(int(status)).decode()


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------

def _ptr(t):
    """Device pointer of a tensor (or None)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _i64_array(values):
    vals = [int(v) for v in values]
    arr = (ctypes.c_int64 * max(1, len(vals)))(*vals)
    return arr, len(vals)


def make_config(*, beta1, beta2, eps, world, chunk, seg_off, tv=(), tu=(), srv_chunk_begin=0,
                srv_chunk_end=-1, defer_sync_writes=False, algorithm="zero-one",
                grad_dtype="f32"):
    """Build a C config; returns (struct, keepalive) -- keep both alive."""
    seg, nseg1 = _i64_array(seg_off)
    tva, ntv = _i64_array(tv)
    tua, ntu = _i64_array(tu)
    cfg = _Config(beta1=float(beta1), beta2=float(beta2), eps=float(eps), world=int(world),
                  chunk=int(chunk), n=int(list(seg_off)[-1]), nseg=nseg1 - 1,
                  seg_off=ctypes.cast(seg, ctypes.POINTER(ctypes.c_int64)), ntv=ntv,
                  tv=ctypes.cast(tva, ctypes.POINTER(ctypes.c_int64)), ntu=ntu,
                  tu=ctypes.cast(tua, ctypes.POINTER(ctypes.c_int64)),
                  srv_chunk_begin=int(srv_chunk_begin), srv_chunk_end=int(srv_chunk_end),
                  defer_sync_writes=1 if defer_sync_writes else 0,
                  algorithm=ALGORITHMS[algorithm], grad_dtype=GRAD_DTYPES[grad_dtype])
    return cfg, (seg, tva, tua)


# ---------------------------------------------------------------------------
# the C names
# ---------------------------------------------------------------------------

def zo_config_check(**kw):
    cfg, keep = make_config(**kw)
    return lib().zo_config_check(ctypes.byref(cfg))


def zo_plan_chunks(seg_off, chunk):
    """Chunk table (start, len, word lists) and total packed words, host only."""
    seg, n1 = _i64_array(seg_off)
    nch = lib().zo_plan_num_chunks(n1 - 1, seg, int(chunk))
    if nch < 0:
        raise ZoError(nch, "zo_plan_num_chunks")
    st = (ctypes.c_int64 * max(1, nch))()
    ln = (ctypes.c_int64 * max(1, nch))()
    wd = (ctypes.c_int64 * max(1, nch))()
    nw = lib().zo_plan_chunks(n1 - 1, seg, int(chunk), st, ln, wd)
    if nw < 0:
        raise ZoError(nw, "zo_plan_chunks")
    return list(st)[:nch], list(ln)[:nch], list(wd)[:nch], nw


def zo_adam_init(cfg_kwargs, state, stream=None, static=False):
    """zo_adam_init, or zo_adam_init_static (no allocation) with static=True."""
    cfg, keep = make_config(**cfg_kwargs)
    keys = ("x", "m", "v", "u", "err", "srv_err", "anchor")
    st = _State(**{k: (state[k].data_ptr() if state.get(k) is not None else None) for k in keys})
    for k in keys:
        _ptr(state.get(k))
    h = ctypes.c_void_p()
    name = "zo_adam_init_static" if static else "zo_adam_init"
    rc = getattr(lib(), name)(ctypes.byref(h), ctypes.byref(cfg), ctypes.byref(st),
                              _stream(stream))
    if rc != ZO_OK:
        raise ZoError(rc, name)
    return h


def _call(h, name, *args):
    rc = getattr(lib(), name)(h, *args)
    if rc != ZO_OK:
        detail = lib().zo_last_hip_error(h).decode() if rc == ZO_EHIP else ""
        raise ZoError(rc, name, detail)


def zo_local_step(h, t, gamma, g, gbar=None):
    _call(h, "zo_local_step", int(t), float(gamma), _ptr(g), _ptr(gbar))


def zo_compress_pack_ef(h, t, gamma, g, packed0, scales0):
    _call(h, "zo_compress_pack_ef", int(t), float(gamma), _ptr(g), _ptr(packed0), _ptr(scales0))


def zo_unpack_average(h, t, packed, scales, srv_packed, srv_scales, avg_debug=None):
    _call(h, "zo_unpack_average", int(t), _ptr(packed), _ptr(scales), _ptr(srv_packed),
          _ptr(srv_scales), _ptr(avg_debug))


def zo_diag_server_pattern(h, packed):
    _call(h, "zo_diag_server_pattern", _ptr(packed))


def zo_sync_update(h, t, srv_packed, srv_scales, gbar=None):
    _call(h, "zo_sync_update", int(t), _ptr(srv_packed), _ptr(srv_scales), _ptr(gbar))


def zo_variance_update(h, t, gbar):
    _call(h, "zo_variance_update", int(t), _ptr(gbar))


def zo_fullprec_step(h, t, gamma, gbar):
    _call(h, "zo_fullprec_step", int(t), float(gamma), _ptr(gbar))


def zo_materialize(h):
    _call(h, "zo_materialize")


U_IN_BUFFER, U_ZERO, U_GAMMA_M = 0, 1, 2
ZO_STATE_X, ZO_STATE_M, ZO_STATE_U = 0, 1, 2


def zo_read_state(h, which, out, stream=None):
    """The current x / m / u (which = ZO_STATE_*) into the device tensor out."""
    _call(h, "zo_read_state", int(which), _ptr(out))


def zo_state_location(h):
    """(device address of the buffer holding x, u mode, u gamma): u is in its
    buffer (U_IN_BUFFER), +0 (U_ZERO) or +0 + gamma * m (U_GAMMA_M)."""
    x = ctypes.c_void_p()
    mode = ctypes.c_int32()
    gam = ctypes.c_float()
    rc = lib().zo_state_location(h, ctypes.byref(x), ctypes.byref(mode), ctypes.byref(gam))
    if rc != ZO_OK:
        raise ZoError(rc, "zo_state_location")
    return x.value, mode.value, gam.value


def zo_adam_destroy(h):
    rc = lib().zo_adam_destroy(h)
    if rc != ZO_OK:
        raise ZoError(rc, "zo_adam_destroy")


def zo_diag_divsqrt(a, b, q, r, stream=None):
    rc = lib().zo_diag_divsqrt(_ptr(a), _ptr(b), _ptr(q), _ptr(r), a.numel(), _stream(stream))
    if rc != ZO_OK:
        raise ZoError(rc, "zo_diag_divsqrt")


def zo_diag_copy(src, dst, nontemporal=True, stream=None):
    rc = lib().zo_diag_copy(_ptr(src), _ptr(dst), src.numel(), 1 if nontemporal else 0,
                            _stream(stream))
    if rc != ZO_OK:
        raise ZoError(rc, "zo_diag_copy")


def zo_diag_stream(srcs, dsts, stream=None):
    """dst[w] = sum(srcs) + w over float32 device tensors of one length."""
    n = srcs[0].numel()
    for t in list(srcs) + list(dsts):
        if t.numel() != n:
            raise ValueError("every stream must have the same length")
    sa = (ctypes.c_void_p * len(srcs))(*[_ptr(t).value for t in srcs])
    da = (ctypes.c_void_p * len(dsts))(*[_ptr(t).value for t in dsts])
    rc = lib().zo_diag_stream(sa, len(srcs), da, len(dsts), n, _stream(stream))
    if rc != ZO_OK:
        raise ZoError(rc, "zo_diag_stream")


_TORCH_GRAD = {"f32": "float32", "f16": "float16", "bf16": "bfloat16"}


def _need(t, what, dtype, n):
    """A tensor of torch dtype `dtype` with at least n elements (the C ABI
    takes bare pointers, so a short buffer would be read or written past
    its end on the device)."""
    if t is None:
        raise ValueError(f"{what}: a tensor is required")
    if str(t.dtype).replace("torch.", "") != dtype:
        raise ValueError(f"{what}: expected {dtype}, got {t.dtype}")
    if t.numel() < n:
        raise ValueError(f"{what}: needs at least {n} elements, has {t.numel()}")


class ZoAdam:
    """One worker's 0/1 Adam optimizer state on one GPU (a handle of the C ABI).

    ``state`` maps x, m, v, u, err, srv_err, anchor to float32 device tensors;
    x holds x_0.  The handle enqueues on ``stream`` (torch's current stream by
    default).  Every method checks its tensors' element types and sizes
    against the configuration before anything reaches the device."""

    def __init__(self, *, beta1, beta2, eps, world, chunk, seg_off, tv=(), tu=(), state,
                 srv_chunk_begin=0, srv_chunk_end=-1, defer_sync_writes=False,
                 algorithm="zero-one", grad_dtype="f32", stream=None, static=False):
        self.cfg = dict(beta1=beta1, beta2=beta2, eps=eps, world=world, chunk=chunk,
                        seg_off=list(seg_off), tv=list(tv), tu=list(tu),
                        srv_chunk_begin=srv_chunk_begin, srv_chunk_end=srv_chunk_end,
                        defer_sync_writes=defer_sync_writes, algorithm=algorithm,
                        grad_dtype=grad_dtype)
        self.h = None
        self._sizes()
        n = self.n
        fv = algorithm == "frozen-variance"
        for k in ("x", "m", "v", "err", "u", "anchor"):
            if fv and k in ("u", "anchor") and state.get(k) is None:
                continue
            if n:
                _need(state.get(k), f"state[{k!r}]", "float32", n)
        if self.r_elems:
            _need(state.get("srv_err"), "state['srv_err']", "float32", self.r_elems)
        self.state = state
        self.h = zo_adam_init(self.cfg, state, stream, static=static)

    def _sizes(self):
        """Shard length, chunks, packed words and the server range, from the
        host planning helpers (an invalid configuration is left to
        zo_adam_init to reject)."""
        c = self.cfg
        start, ln, word, nwords = zo_plan_chunks(c["seg_off"], c["chunk"])
        nch = len(ln)
        self.n, self.nchunks, self.nwords = int(c["seg_off"][-1]), nch, int(nwords)
        c0 = int(c["srv_chunk_begin"])
        c1 = nch if c["srv_chunk_end"] < 0 else int(c["srv_chunk_end"])
        self.r_chunks = self.r_words = self.r_elems = 0
        if 0 <= c0 < c1 <= nch:
            self.r_chunks = c1 - c0
            self.r_words = word[c1 - 1] + (ln[c1 - 1] + 63) // 64 - word[c0]
            self.r_elems = start[c1 - 1] + ln[c1 - 1] - start[c0]

    def _grad(self, t, what):
        if self.n:
            _need(t, what, _TORCH_GRAD[self.cfg["grad_dtype"]], self.n)

    def _server_out(self, srv_packed, srv_scales):
        if self.nchunks:
            _need(srv_packed, "srv_packed", "int64", self.nwords)
            _need(srv_scales, "srv_scales", "float32", self.nchunks)

    def close(self):
        if self.h is not None:
            zo_adam_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_stream(self, stream):
        rc = lib().zo_set_stream(self.h, _stream(stream))
        if rc != ZO_OK:
            raise ZoError(rc, "zo_set_stream")

    # the six hot-path calls
    def local_step(self, t, gamma, g, gbar=None):
        self._grad(g, "g")
        if gbar is not None:
            self._grad(gbar, "gbar")
        zo_local_step(self.h, t, gamma, g, gbar)

    def compress_pack_ef(self, t, gamma, g, packed0, scales0):
        if g is not None:
            self._grad(g, "g")
        if self.nchunks:
            _need(packed0, "packed0", "int64", self.nwords)
            _need(scales0, "scales0", "float32", self.nchunks)
        zo_compress_pack_ef(self.h, t, gamma, g, packed0, scales0)

    def diag_server_pattern(self, packed):
        """The server's memory accesses without its arithmetic (the server
        error is rewritten unchanged); see zo_diag_server_pattern."""
        if self.r_chunks:
            _need(packed, "packed", "int64", int(self.cfg["world"]) * self.r_words)
        zo_diag_server_pattern(self.h, packed)

    def unpack_average(self, t, packed, scales, srv_packed, srv_scales, avg_debug=None):
        W = int(self.cfg["world"])
        if self.r_chunks:
            _need(packed, "packed", "int64", W * self.r_words)
            _need(scales, "scales", "float32", W * self.r_chunks)
        self._server_out(srv_packed, srv_scales)
        if avg_debug is not None:
            _need(avg_debug, "avg_debug", "float32", self.r_elems)
        zo_unpack_average(self.h, t, packed, scales, srv_packed, srv_scales, avg_debug)

    def sync_update(self, t, srv_packed, srv_scales, gbar=None):
        self._server_out(srv_packed, srv_scales)
        if gbar is not None:
            self._grad(gbar, "gbar")
        zo_sync_update(self.h, t, srv_packed, srv_scales, gbar)

    def variance_update(self, t, gbar):
        self._grad(gbar, "gbar")
        zo_variance_update(self.h, t, gbar)

    def fullprec_step(self, t, gamma, gbar):
        self._grad(gbar, "gbar")
        zo_fullprec_step(self.h, t, gamma, gbar)

    def materialize(self):
        zo_materialize(self.h)

    def current(self, name):
        """State `name` as it is now: x, m and u through zo_read_state (deferred
        sync writes may keep them elsewhere), the others from their buffers."""
        which = {"x": ZO_STATE_X, "m": ZO_STATE_M, "u": ZO_STATE_U}.get(name)
        if which is None or (name == "u" and self.cfg["algorithm"] != "zero-one"):
            return self.state[name]
        out = self.state[name].new_empty(self.state[name].shape)
        zo_read_state(self.h, which, out)
        return out

    # queries
    @property
    def num_chunks(self):
        return int(lib().zo_num_chunks(self.h))

    @property
    def packed_words(self):
        return int(lib().zo_packed_words(self.h))

    @property
    def gamma_sum(self):
        return float(lib().zo_gamma_sum(self.h))

    @property
    def next_step(self):
        return int(lib().zo_next_step(self.h))

    def server_range(self):
        vals = [ctypes.c_int64() for _ in range(6)]
        rc = lib().zo_server_range(self.h, *[ctypes.byref(v) for v in vals])
        if rc != ZO_OK:
            raise ZoError(rc, "zo_server_range")
        keys = ("chunk0", "nchunks", "word0", "nwords", "elem0", "nelems")
        return {k: v.value for k, v in zip(keys, vals)}

    def chunk_table(self):
        n = self.num_chunks
        arrs = [(ctypes.c_int64 * max(1, n))() for _ in range(3)]
        rc = lib().zo_chunk_table(self.h, *arrs)
        if rc != ZO_OK:
            raise ZoError(rc, "zo_chunk_table")
        return [list(a)[:n] for a in arrs]

    def inexact_chunks(self):
        c = ctypes.c_int64()
        rc = lib().zo_inexact_chunks(self.h, ctypes.byref(c))
        if rc != ZO_OK:
            raise ZoError(rc, "zo_inexact_chunks")
        return c.value
