"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

Holds the counter-based generator (Philox4x32-10 with an Irwin-Hall(4)
transform, synth/csrc/philox.h) in a host build (gcc, libsynth_cpu.so) and
a device build (hipcc, libsynth_hip.so), plus the workload descriptions in
synth.workloads.  Nothing here computes any step of the delta-extraction
method.
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from . import workloads  # noqa: F401
from .workloads import ABSVAL, SIGMA

_HERE = os.path.dirname(os.path.abspath(__file__))
CPU_LIB = os.path.join(_HERE, "libsynth_cpu.so")
HIP_LIB = os.path.join(_HERE, "libsynth_hip.so")

_cpu = None
_hip = None


def _load_cpu():
    global _cpu
    if _cpu is None:
        if not os.path.exists(CPU_LIB):
            from .build import build_cpu
            build_cpu()
        lib = ctypes.CDLL(CPU_LIB)
        lib.synth_scale.restype = ctypes.c_double
        lib.synth_scale.argtypes = [ctypes.c_double]
        lib.synth_word.restype = ctypes.c_uint32
        lib.synth_word.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32,
                                   ctypes.c_uint64]
        lib.synth_fill_cpu.restype = None
        lib.synth_fill_cpu.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                       ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64,
                                       ctypes.c_double, ctypes.c_int]
        lib.synth_fill_2d_cpu.restype = None
        lib.synth_fill_2d_cpu.argtypes = [ctypes.c_void_p] + [ctypes.c_int64] * 3 + [
            ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32] + [ctypes.c_int64] * 3 + [
            ctypes.c_double, ctypes.c_int]
        lib.synth_philox_block.restype = None
        lib.synth_philox_block.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        _cpu = lib
    return _cpu


def _load_hip():
    global _hip
    if _hip is None:
        if not os.path.exists(HIP_LIB):
            raise RuntimeError("synth: %s is not built (run __graft_entry__.build())" % HIP_LIB)
        lib = ctypes.CDLL(HIP_LIB)
        lib.synth_fill_2d_hip.restype = ctypes.c_int
        lib.synth_fill_2d_hip.argtypes = [ctypes.c_void_p] + [ctypes.c_int64] * 3 + [
            ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32] + [ctypes.c_int64] * 3 + [
            ctypes.c_double, ctypes.c_int, ctypes.c_void_p]
        lib.synth_fill_hip.restype = ctypes.c_int
        lib.synth_fill_hip.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64,
                                       ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64,
                                       ctypes.c_double, ctypes.c_int, ctypes.c_void_p]
        _hip = lib
    return _hip


def scale(sigma: float) -> float:
    """sigma*sqrt(3)*2^-32 in binary64 (computed by the C build)."""
    return _load_cpu().synth_scale(sigma)


def word(seed: int, tensor: int, kind: int, index: int) -> int:
    """First Philox word at (seed, tensor, kind, index)."""
    return _load_cpu().synth_word(seed, tensor, kind, index)


def philox_block(ctr, key):
    """Raw Philox4x32-10 block (for known-answer tests)."""
    c = (ctypes.c_uint32 * 4)(*ctr)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    _load_cpu().synth_philox_block(c, k, o)
    return tuple(int(x) for x in o)


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def fill_cpu(out: np.ndarray, seed: int, tensor: int, kind: int, index_base: int = 0,
             threads: int = 1, chunk: int = 1 << 22) -> np.ndarray:
    """Fill a float32 host array with the draws of (seed, tensor, kind)."""
    assert out.dtype == np.float32 and out.flags.c_contiguous
    lib = _load_cpu()
    sc = lib.synth_scale(SIGMA[kind])
    ab = ABSVAL[kind]
    n = out.size
    base = out.ctypes.data

    def run(lo):
        hi = min(n, lo + chunk)
        lib.synth_fill_cpu(base + 4 * lo, hi - lo, seed, tensor, kind, index_base + lo, sc, ab)

    starts = range(0, n, chunk)
    if threads <= 1 or n <= chunk:
        for lo in starts:
            run(lo)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, starts))
    return out


def draw_cpu(n: int, seed: int, tensor: int, kind: int, index_base: int = 0,
             threads: int = 1) -> np.ndarray:
    return fill_cpu(np.empty(n, np.float32), seed, tensor, kind, index_base, threads)


def fill_gpu(ptr: int, n: int, seed: int, tensor: int, kind: int, index_base: int = 0,
             stream: int = 0) -> None:
    """Fill n float32 elements at device address ptr on a HIP stream."""
    lib = _load_hip()
    rc = lib.synth_fill_hip(ptr, n, seed, tensor, kind, index_base,
                            _load_cpu().synth_scale(SIGMA[kind]), ABSVAL[kind], stream)
    if rc != 0:
        raise RuntimeError("synth_fill_hip failed with hipError %d" % rc)


def fill_cpu_2d(out: np.ndarray, seed: int, tensor: int, kind: int, row0: int, col0: int,
                canon_ncols: int) -> np.ndarray:
    """Fill a 2-D float32 host array (rows may be strided) with the draws of
    the canonical block starting at (row0, col0) of a tensor with
    canon_ncols columns."""
    assert out.dtype == np.float32 and out.ndim == 2 and out.strides[1] == 4
    lib = _load_cpu()
    lib.synth_fill_2d_cpu(out.ctypes.data, out.shape[0], out.shape[1], out.strides[0] // 4, seed,
                          tensor, kind, row0, col0, canon_ncols, lib.synth_scale(SIGMA[kind]),
                          ABSVAL[kind])
    return out


def fill_gpu_2d(ptr: int, nrows: int, ncols: int, row_stride: int, seed: int, tensor: int,
                kind: int, row0: int, col0: int, canon_ncols: int, stream: int = 0) -> None:
    """Device version of fill_cpu_2d (row_stride in elements)."""
    lib = _load_hip()
    rc = lib.synth_fill_2d_hip(ptr, nrows, ncols, row_stride, seed, tensor, kind, row0, col0,
                               canon_ncols, _load_cpu().synth_scale(SIGMA[kind]), ABSVAL[kind],
                               stream)
    if rc != 0:
        raise RuntimeError("synth_fill_2d_hip failed with hipError %d" % rc)
