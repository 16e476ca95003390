"""Seeded synthetic inputs shared by the tests and the benchmark.

Host fills (numpy) and device fills (torch tensors on the current stream)
produce the same bits from the same (seed, stream, step, index); see
``synth.hip`` for the definitions.  This package holds no optimizer
arithmetic.
"""
import ctypes
import os

import numpy as np

from . import configs  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "libzosynth.so")
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_LIB_PATH)
        i64, u64, u32, f32, vp = (ctypes.c_int64, ctypes.c_uint64, ctypes.c_uint32,
                                  ctypes.c_float, ctypes.c_void_p)
        L.zs_key.argtypes = [u64, u32, i64]
        L.zs_key.restype = u64
        L.zs_fill_normal_host.argtypes = [vp, i64, i64, u64, f32, u32, f32]
        L.zs_fill_normal_host.restype = None
        L.zs_fill_bits_host.argtypes = [vp, i64, i64, u64]
        L.zs_fill_bits_host.restype = None
        L.zs_fill_scales_host.argtypes = [vp, i64, i64, u64, f32]
        L.zs_fill_scales_host.restype = None
        L.zs_fill_normal_host_ranges.argtypes = [vp, i64, vp, vp, u64, f32, u32, f32]
        L.zs_fill_normal_host_ranges.restype = None
        L.zs_fill_bits_host_ranges.argtypes = [vp, i64, vp, vp, u64]
        L.zs_fill_bits_host_ranges.restype = None
        L.zs_fill_scales_host_ranges.argtypes = [vp, i64, vp, vp, u64, f32]
        L.zs_fill_scales_host_ranges.restype = None
        L.zs_fill_normal_dev.argtypes = [vp, i64, i64, u64, f32, u32, f32, vp]
        L.zs_fill_normal_dev.restype = ctypes.c_int
        L.zs_fill_bits_dev.argtypes = [vp, i64, i64, u64, vp]
        L.zs_fill_bits_dev.restype = ctypes.c_int
        L.zs_fill_scales_dev.argtypes = [vp, i64, i64, u64, f32, vp]
        L.zs_fill_scales_dev.restype = ctypes.c_int
        _lib = L
    return _lib


def key(seed, stream, step):
    return int(lib().zs_key(int(seed), int(stream), int(step)))


# ------------------------------------------------------------------- host side
def normal_host(n, idx0, k, ksig, per_mille=0, factor=1.0):
    out = np.empty(int(n), np.float32)
    lib().zs_fill_normal_host(out.ctypes.data, int(n), int(idx0), k, float(ksig),
                              int(per_mille), float(factor))
    return out


def bits_host(nwords, word0, k):
    out = np.empty(int(nwords), np.uint64)
    lib().zs_fill_bits_host(out.ctypes.data, int(nwords), int(word0), k)
    return out


def scales_host(n, idx0, k, base):
    out = np.empty(int(n), np.float32)
    lib().zs_fill_scales_host(out.ctypes.data, int(n), int(idx0), k, float(base))
    return out


def _ranges(starts, lens):
    s = np.ascontiguousarray(starts, dtype=np.int64)
    n = np.ascontiguousarray(lens, dtype=np.int64)
    assert s.shape == n.shape
    return s, n, int(n.sum())


def normal_host_ranges(starts, lens, k, ksig, per_mille=0, factor=1.0):
    """normal_host over several index ranges, concatenated."""
    s, n, tot = _ranges(starts, lens)
    out = np.empty(tot, np.float32)
    lib().zs_fill_normal_host_ranges(out.ctypes.data, len(s), s.ctypes.data, n.ctypes.data, k,
                                     float(ksig), int(per_mille), float(factor))
    return out


def bits_host_ranges(word0s, nwords, k):
    """bits_host over several word ranges, concatenated."""
    s, n, tot = _ranges(word0s, nwords)
    out = np.empty(tot, np.uint64)
    lib().zs_fill_bits_host_ranges(out.ctypes.data, len(s), s.ctypes.data, n.ctypes.data, k)
    return out


def scales_host_ranges(starts, lens, k, base):
    """scales_host over several index ranges, concatenated."""
    s, n, tot = _ranges(starts, lens)
    out = np.empty(tot, np.float32)
    lib().zs_fill_scales_host_ranges(out.ctypes.data, len(s), s.ctypes.data, n.ctypes.data, k,
                                     float(base))
    return out


# ----------------------------------------------------------------- device side
def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _chk(rc):
    if rc != 0:
        raise RuntimeError(f"synth device fill failed: hipError {rc}")


def normal_dev(t, idx0, k, ksig, per_mille=0, factor=1.0, stream=None):
    assert t.is_cuda and t.is_contiguous()
    _chk(lib().zs_fill_normal_dev(t.data_ptr(), t.numel(), int(idx0), k, float(ksig),
                                  int(per_mille), float(factor), _stream_ptr(stream)))


def bits_dev(t, word0, k, stream=None):
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8
    _chk(lib().zs_fill_bits_dev(t.data_ptr(), t.numel(), int(word0), k, _stream_ptr(stream)))


def scales_dev(t, idx0, k, base, stream=None):
    assert t.is_cuda and t.is_contiguous()
    _chk(lib().zs_fill_scales_dev(t.data_ptr(), t.numel(), int(idx0), k, float(base),
                                  _stream_ptr(stream)))
