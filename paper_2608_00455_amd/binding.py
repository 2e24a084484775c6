"""ctypes binding of libdte.so (include/dte.h): same names, argument
marshalling only.  Device buffers are passed as integer addresses (for
example torch.Tensor.data_ptr()), streams as integer hipStream_t handles
(torch.cuda.current_stream().cuda_stream); every step runs in the library.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdte.so")

DTE_OK, DTE_ERR_ARG, DTE_ERR_PLAN, DTE_ERR_CAPACITY, DTE_ERR_HIP = 0, 1, 2, 3, 4
DTE_ERR_IO, DTE_ERR_CORRUPT, DTE_ERR_CHAIN, DTE_ERR_UNSUPPORTED, DTE_ERR_HOST = 5, 6, 7, 8, 9
DTE_MAX_DIMS = 4
DTE_MAX_RANKS = 64

EXPORTED = ("dte_derive_scalars", "dte_extract_delta", "dte_ordered_workspace_bytes",
            "dte_extract_delta_ordered", "dte_extract_delta_ordered_noalloc",
            "dte_ordered_noalloc_max_capacity", "dte_plan_create", "dte_plan_destroy",
            "dte_plan_info", "dte_remap", "dte_extract_remap", "dte_apply", "dte_adamw_forward",
            "dte_status_string")


class DteError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__("%s: %s" % (fn, _lib().dte_status_string(status).decode()))
        self.status = status


DTE_ORDER_FOLDED, DTE_ORDER_LITERAL = 0, 1


class dte_adamw_step(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double),
                ("beta2", ctypes.c_double), ("eps", ctypes.c_double),
                ("weight_decay", ctypes.c_double), ("step", ctypes.c_int64),
                ("order", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class dte_scalars(ctypes.Structure):
    _fields_ = [("lrb1", ctypes.c_float), ("rbc2", ctypes.c_float), ("eps", ctypes.c_float),
                ("decay", ctypes.c_float), ("lr", ctypes.c_float), ("bc1", ctypes.c_float),
                ("bc2", ctypes.c_float), ("order", ctypes.c_int32)]


class dte_segment(ctypes.Structure):
    _fields_ = [("flat_begin", ctypes.c_int64), ("ndim", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("shape", ctypes.c_int64 * DTE_MAX_DIMS)]


class dte_op(ctypes.Structure):
    _fields_ = [("segment", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("dst_base", ctypes.c_int64),
                ("src_origin", ctypes.c_int64 * DTE_MAX_DIMS),
                ("extent", ctypes.c_int64 * DTE_MAX_DIMS),
                ("dst_origin", ctypes.c_int64 * DTE_MAX_DIMS),
                ("dst_shape", ctypes.c_int64 * DTE_MAX_DIMS)]


_L = None


def _lib():
    global _L
    if _L is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libdte.so is not built at %s: run __graft_entry__.build() "
                               "(the HIP path has no fallback)" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, I64, I32, S = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32
        L.dte_status_string.restype = ctypes.c_char_p
        L.dte_status_string.argtypes = [S]
        L.dte_derive_scalars.restype = S
        L.dte_derive_scalars.argtypes = [ctypes.POINTER(dte_adamw_step),
                                         ctypes.POINTER(dte_scalars)]
        L.dte_extract_delta.restype = S
        L.dte_extract_delta.argtypes = [P, P, P, I64, I64, ctypes.POINTER(dte_adamw_step), P, P,
                                        I64, P, P, P]
        L.dte_ordered_workspace_bytes.restype = I64
        L.dte_ordered_workspace_bytes.argtypes = [I64]
        L.dte_extract_delta_ordered.restype = S
        L.dte_extract_delta_ordered.argtypes = [P, P, P, I64, I64,
                                                ctypes.POINTER(dte_adamw_step), P, P, I64, P, P,
                                                I64, P, P]
        L.dte_extract_delta_ordered_noalloc.restype = S
        L.dte_extract_delta_ordered_noalloc.argtypes = [P, P, P, I64, I64,
                                                        ctypes.POINTER(dte_adamw_step), P, P,
                                                        I64, P, P, P]
        L.dte_ordered_noalloc_max_capacity.restype = I64
        L.dte_ordered_noalloc_max_capacity.argtypes = []
        L.dte_plan_create.restype = S
        L.dte_plan_create.argtypes = [ctypes.POINTER(dte_segment), I32, ctypes.POINTER(dte_op),
                                      I32, I32, ctypes.POINTER(I64), ctypes.POINTER(P)]
        L.dte_plan_destroy.restype = None
        L.dte_plan_destroy.argtypes = [P]
        L.dte_plan_info.restype = S
        L.dte_plan_info.argtypes = [P, ctypes.POINTER(I64), ctypes.POINTER(I32),
                                    ctypes.POINTER(I32)]
        L.dte_remap.restype = S
        L.dte_remap.argtypes = [P, P, P, P, I64, ctypes.POINTER(P), ctypes.POINTER(P),
                                ctypes.POINTER(I64), P, P]
        L.dte_extract_remap.restype = S
        L.dte_extract_remap.argtypes = [P, P, P, I64, I64, ctypes.POINTER(dte_adamw_step), P,
                                        ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(I64),
                                        P, P, P]
        L.dte_apply.restype = S
        L.dte_apply.argtypes = [P, ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(P), P,
                                ctypes.POINTER(I64), P]
        L.dte_adamw_forward.restype = S
        L.dte_adamw_forward.argtypes = [P, P, P, P, I64, ctypes.POINTER(dte_adamw_step), P]
        _L = L
    return _L


def _check(fn, st):
    if st != DTE_OK:
        raise DteError(fn, st)


def _hp(hp) -> dte_adamw_step:
    if isinstance(hp, dte_adamw_step):
        return hp
    return dte_adamw_step(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, hp.step,
                          getattr(hp, "order", DTE_ORDER_FOLDED), 0)


def _ptrs(xs):
    return (ctypes.c_void_p * len(xs))(*[int(x) for x in xs])


def _i64s(xs):
    return (ctypes.c_int64 * len(xs))(*[int(x) for x in xs])


def dte_status_string(status: int) -> str:
    return _lib().dte_status_string(status).decode()


def dte_derive_scalars(hp) -> dte_scalars:
    out = dte_scalars()
    _check("dte_derive_scalars", _lib().dte_derive_scalars(ctypes.byref(_hp(hp)),
                                                           ctypes.byref(out)))
    return out


def dte_extract_delta(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor,
                      out_prev=0, stream=0):
    _check("dte_extract_delta",
           _lib().dte_extract_delta(p, m, v, n, index_base, ctypes.byref(_hp(hp)), out_idx,
                                    out_val, capacity, cursor, out_prev or None, stream or None))


def dte_ordered_workspace_bytes(capacity) -> int:
    return int(_lib().dte_ordered_workspace_bytes(capacity))


def dte_extract_delta_ordered(p, m, v, n, index_base, hp, out_idx, out_val, capacity, cursor,
                              workspace, workspace_bytes, out_prev=0, stream=0):
    _check("dte_extract_delta_ordered",
           _lib().dte_extract_delta_ordered(p, m, v, n, index_base, ctypes.byref(_hp(hp)),
                                            out_idx, out_val, capacity, cursor,
                                            workspace or None, workspace_bytes,
                                            out_prev or None, stream or None))


def dte_extract_delta_ordered_noalloc(p, m, v, n, index_base, hp, out_idx, out_val, capacity,
                                      cursor, out_prev=0, stream=0):
    _check("dte_extract_delta_ordered_noalloc",
           _lib().dte_extract_delta_ordered_noalloc(p, m, v, n, index_base,
                                                    ctypes.byref(_hp(hp)), out_idx, out_val,
                                                    capacity, cursor, out_prev or None,
                                                    stream or None))


def dte_ordered_noalloc_max_capacity() -> int:
    return int(_lib().dte_ordered_noalloc_max_capacity())


def dte_extract_remap(p, m, v, n, index_base, hp, plan, out_off, out_val, rank_capacity,
                      rank_count, count, stream=0):
    _check("dte_extract_remap",
           _lib().dte_extract_remap(p, m, v, n, index_base, ctypes.byref(_hp(hp)), plan,
                                    _ptrs(out_off), _ptrs(out_val), _i64s(rank_capacity),
                                    rank_count, count, stream or None))


def dte_adamw_forward(p, m, v, g, n, hp, stream=0):
    _check("dte_adamw_forward",
           _lib().dte_adamw_forward(p, m, v, g, n, ctypes.byref(_hp(hp)), stream or None))


def dte_plan_create(segments, ops, nranks, rank_numel) -> int:
    """segments / ops: sequences of dte_segment / dte_op; returns the handle."""
    segs = (dte_segment * len(segments))(*segments)
    opa = (dte_op * max(1, len(ops)))(*ops)
    handle = ctypes.c_void_p()
    _check("dte_plan_create",
           _lib().dte_plan_create(segs, len(segments), opa, len(ops), nranks,
                                  _i64s(rank_numel), ctypes.byref(handle)))
    return handle.value


def dte_plan_destroy(plan: int) -> None:
    _lib().dte_plan_destroy(plan)


def dte_plan_info(plan: int):
    total, nranks, rep = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
    _check("dte_plan_info", _lib().dte_plan_info(plan, ctypes.byref(total), ctypes.byref(nranks),
                                                 ctypes.byref(rep)))
    return total.value, nranks.value, rep.value


def dte_remap(plan, idx, val, count, in_capacity, out_off, out_val, rank_capacity, rank_count,
              stream=0):
    _check("dte_remap",
           _lib().dte_remap(plan, idx, val, count, in_capacity, _ptrs(out_off), _ptrs(out_val),
                            _i64s(rank_capacity), rank_count, stream or None))


def dte_apply(plan, shards, off, val, rank_count, rank_capacity, stream=0):
    _check("dte_apply",
           _lib().dte_apply(plan, _ptrs(shards), _ptrs(off), _ptrs(val), rank_count,
                            _i64s(rank_capacity), stream or None))


def raw_status(fn: str, *args) -> int:
    """Call an entry point and return its raw status (for error-path tests)."""
    return getattr(_lib(), fn)(*args)
