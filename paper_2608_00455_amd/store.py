"""ctypes binding of the storage-mediated publication path (include/dte_store.h).

Argument marshalling only: chunking, compression, checksums, manifests and
the device kernels run inside libdte.so.  Functions raise DteError on a
non-OK status, except `commit` (returns whether a version was published)
and `read_*` (return the entry total, which may exceed the capacity).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import List, Sequence, Tuple

import numpy as np

from . import binding as B

CODEC_NONE, CODEC_ZSTD = 0, 1


class dte_store_segment(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("flat_begin", ctypes.c_int64),
                ("numel", ctypes.c_int64)]


class dte_store_options(ctypes.Structure):
    _fields_ = [("codec", ctypes.c_int32), ("level", ctypes.c_int32),
                ("threads", ctypes.c_int32), ("index_transform", ctypes.c_int32),
                ("chunk_entries", ctypes.c_int64)]


class dte_store_piece(ctypes.Structure):
    _fields_ = [("sender_begin", ctypes.c_int64), ("sender_end", ctypes.c_int64),
                ("segment", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("local_cols", ctypes.c_int64), ("canon_cols", ctypes.c_int64),
                ("canon_row0", ctypes.c_int64), ("canon_col0", ctypes.c_int64)]


class dte_store_stats(ctypes.Structure):
    _fields_ = [("entries", ctypes.c_int64), ("chunks", ctypes.c_int64),
                ("raw_bytes", ctypes.c_int64), ("stored_bytes", ctypes.c_int64)]


EXPORTED = ("dte_store_write_part_host", "dte_store_write_part_device",
            "dte_store_write_part_host_mapped", "dte_store_write_part_device_mapped",
            "dte_store_commit",
            "dte_store_latest", "dte_store_chain", "dte_store_read_host",
            "dte_store_read_device", "dte_store_xxh64")

_bound = False


def _lib():
    global _bound
    L = B._lib()
    if not _bound:
        P, I64, I32, S = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32
        seg_p = ctypes.POINTER(dte_store_segment)
        opt_p = ctypes.POINTER(dte_store_options)
        st_p = ctypes.POINTER(dte_store_stats)
        L.dte_store_write_part_host.restype = S
        L.dte_store_write_part_host.argtypes = [ctypes.c_char_p, I64, I32, seg_p, I32, P, P, I64,
                                                opt_p, st_p]
        L.dte_store_write_part_device.restype = S
        L.dte_store_write_part_device.argtypes = [ctypes.c_char_p, I64, I32, seg_p, I32, P, P, P,
                                                  I64, opt_p, st_p, P]
        pc_p = ctypes.POINTER(dte_store_piece)
        L.dte_store_write_part_host_mapped.restype = S
        L.dte_store_write_part_host_mapped.argtypes = [ctypes.c_char_p, I64, I32, seg_p, I32, pc_p,
                                                       I32, P, P, I64, opt_p, st_p]
        L.dte_store_write_part_device_mapped.restype = S
        L.dte_store_write_part_device_mapped.argtypes = [ctypes.c_char_p, I64, I32, seg_p, I32,
                                                         pc_p, I32, P, P, P, I64, opt_p, st_p, P]
        L.dte_store_commit.restype = S
        L.dte_store_commit.argtypes = [ctypes.c_char_p, I64, I64, I32, ctypes.POINTER(I32)]
        L.dte_store_latest.restype = S
        L.dte_store_latest.argtypes = [ctypes.c_char_p, ctypes.POINTER(I64)]
        L.dte_store_chain.restype = S
        L.dte_store_chain.argtypes = [ctypes.c_char_p, I64, I64, ctypes.POINTER(I64), I32,
                                      ctypes.POINTER(I32)]
        L.dte_store_read_host.restype = S
        L.dte_store_read_host.argtypes = [ctypes.c_char_p, I64, I64, P, P, I64,
                                          ctypes.POINTER(I64), I32, st_p]
        L.dte_store_read_device.restype = S
        L.dte_store_read_device.argtypes = [ctypes.c_char_p, I64, I64, P, P, I64,
                                            ctypes.POINTER(I64), I32, st_p, P]
        L.dte_store_xxh64.restype = ctypes.c_uint64
        L.dte_store_xxh64.argtypes = [P, I64, ctypes.c_uint64]
        _bound = True
    return L


@dataclass
class Options:
    codec: int = CODEC_ZSTD
    level: int = 3
    threads: int = 8
    index_transform: int = 1
    chunk_entries: int = 1 << 20

    def c(self) -> dte_store_options:
        return dte_store_options(self.codec, self.level, self.threads, self.index_transform,
                                 self.chunk_entries)


@dataclass
class Stats:
    entries: int
    chunks: int
    raw_bytes: int
    stored_bytes: int


def _stats(s: dte_store_stats) -> Stats:
    return Stats(s.entries, s.chunks, s.raw_bytes, s.stored_bytes)


def segments_of(names: Sequence[str], begins: Sequence[int], numels: Sequence[int]):
    """Host array of dte_store_segment (keeps the name buffers alive)."""
    arr = (dte_store_segment * max(1, len(names)))()
    keep = []
    for i, (nm, b, n) in enumerate(zip(names, begins, numels)):
        raw = nm.encode()
        keep.append(raw)
        arr[i] = dte_store_segment(raw, int(b), int(n))
    return arr, len(names), keep


def _dir(d) -> bytes:
    return str(d).encode()


def pieces_of(rows):
    """Host array of dte_store_piece from tuples (sender_begin, sender_end,
    segment, local_cols, canon_cols, canon_row0, canon_col0)."""
    arr = (dte_store_piece * max(1, len(rows)))()
    for i, (b, e, sg, lc, cc, r0, c0) in enumerate(rows):
        arr[i] = dte_store_piece(b, e, sg, 0, lc, cc, r0, c0)
    return arr, len(rows)


def write_part_host(d, version, writer, segs, idx: np.ndarray, val: np.ndarray,
                    opt: Options = Options(), pieces=None) -> Stats:
    arr, nseg, _keep = segs
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    val = np.ascontiguousarray(val, dtype=np.uint16)
    st = dte_store_stats()
    ip = idx.ctypes.data if idx.size else None
    vp = val.ctypes.data if val.size else None
    if pieces is None:
        rc = _lib().dte_store_write_part_host(_dir(d), version, writer, arr, nseg, ip, vp,
                                              idx.size, ctypes.byref(opt.c()), ctypes.byref(st))
    else:
        parr, npc = pieces
        rc = _lib().dte_store_write_part_host_mapped(_dir(d), version, writer, arr, nseg, parr,
                                                     npc, ip, vp, idx.size,
                                                     ctypes.byref(opt.c()), ctypes.byref(st))
    B._check("dte_store_write_part_host", rc)
    return _stats(st)


def write_part_device(d, version, writer, segs, idx_ptr: int, val_ptr: int, count_ptr: int,
                      capacity: int, opt: Options = Options(), stream: int = 0,
                      pieces=None) -> Stats:
    arr, nseg, _keep = segs
    st = dte_store_stats()
    if pieces is None:
        rc = _lib().dte_store_write_part_device(_dir(d), version, writer, arr, nseg,
                                                idx_ptr or None, val_ptr or None, count_ptr,
                                                capacity, ctypes.byref(opt.c()),
                                                ctypes.byref(st), stream or None)
    else:
        parr, npc = pieces
        rc = _lib().dte_store_write_part_device_mapped(_dir(d), version, writer, arr, nseg, parr,
                                                       npc, idx_ptr or None, val_ptr or None,
                                                       count_ptr, capacity,
                                                       ctypes.byref(opt.c()), ctypes.byref(st),
                                                       stream or None)
    B._check("dte_store_write_part_device", rc)
    return _stats(st)


def commit(d, version, parent, nwriters) -> bool:
    out = ctypes.c_int32(0)
    B._check("dte_store_commit", _lib().dte_store_commit(_dir(d), version, parent, nwriters,
                                                         ctypes.byref(out)))
    return bool(out.value)


def latest(d) -> int:
    out = ctypes.c_int64(0)
    B._check("dte_store_latest", _lib().dte_store_latest(_dir(d), ctypes.byref(out)))
    return out.value


def chain(d, base, newest, max_versions=1024) -> List[int]:
    out = (ctypes.c_int64 * max(1, max_versions))()
    n = ctypes.c_int32(0)
    B._check("dte_store_chain", _lib().dte_store_chain(_dir(d), base, newest, out, max_versions,
                                                       ctypes.byref(n)))
    return [int(out[i]) for i in range(n.value)]


def read_host(d, version, base, capacity=None, threads=8) -> Tuple[np.ndarray, np.ndarray, Stats]:
    """Entries of `version` (parent must be `base`) as host arrays."""
    if capacity is None:
        cnt = ctypes.c_int64(0)
        st = _lib().dte_store_read_host(_dir(d), version, base, None, None, 0,
                                        ctypes.byref(cnt), threads, None)
        B._check("dte_store_read_host", st)
        capacity = cnt.value
    idx = np.empty(max(1, capacity), np.int64)
    val = np.empty(max(1, capacity), np.uint16)
    cnt = ctypes.c_int64(0)
    s = dte_store_stats()
    B._check("dte_store_read_host",
             _lib().dte_store_read_host(_dir(d), version, base, idx.ctypes.data, val.ctypes.data,
                                        capacity, ctypes.byref(cnt), threads, ctypes.byref(s)))
    k = min(cnt.value, capacity)
    return idx[:k], val[:k], _stats(s)


def read_device(d, version, base, idx_ptr: int, val_ptr: int, capacity: int, threads=8,
                stream: int = 0) -> Tuple[int, Stats]:
    cnt = ctypes.c_int64(0)
    s = dte_store_stats()
    B._check("dte_store_read_device",
             _lib().dte_store_read_device(_dir(d), version, base, idx_ptr or None, val_ptr or None,
                                          capacity, ctypes.byref(cnt), threads, ctypes.byref(s),
                                          stream or None))
    return cnt.value, _stats(s)


def raw_status(fn: str, *args) -> int:
    return getattr(_lib(), fn)(*args)


def xxh64(data: bytes, seed: int = 0) -> int:
    buf = ctypes.create_string_buffer(data, len(data))
    return int(_lib().dte_store_xxh64(buf if data else None, len(data), seed))
