"""Per-element steps of the oracle (test infrastructure only).

Thin numpy wrappers over liboracle.so (dte_oracle.c) for the binary32
arithmetic, plus numpy's flatnonzero as the paper's nonzero step.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


class Scalars(ctypes.Structure):
    _fields_ = [("lrb1", ctypes.c_float), ("rbc2", ctypes.c_float), ("eps", ctypes.c_float),
                ("decay", ctypes.c_float), ("b1", ctypes.c_float), ("b2", ctypes.c_float),
                ("omb1", ctypes.c_float), ("omb2", ctypes.c_float), ("lr", ctypes.c_float),
                ("bc1", ctypes.c_float), ("bc2", ctypes.c_float), ("order", ctypes.c_int32)]

    def bits(self):
        """The four scalars of the inverse as binary32 bit patterns."""
        return tuple(int(np.float32(getattr(self, f)).view(np.uint32))
                     for f in ("lrb1", "rbc2", "eps", "decay"))


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from .build import build
            build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        L.oracle_derive_scalars.restype = ctypes.c_int
        L.oracle_derive_scalars.argtypes = [ctypes.c_double] * 5 + [
            ctypes.c_int64, ctypes.c_int32, ctypes.POINTER(Scalars)]
        L.oracle_adamw_forward.restype = None
        L.oracle_adamw_forward.argtypes = [P, P, P, P, ctypes.c_int64, ctypes.POINTER(Scalars),
                                           P, P, P]
        L.oracle_invert.restype = None
        L.oracle_invert.argtypes = [P, P, P, ctypes.c_int64, ctypes.POINTER(Scalars), P]
        L.oracle_bf16.restype = ctypes.c_uint16
        L.oracle_bf16.argtypes = [ctypes.c_float]
        L.oracle_bf16_array.restype = None
        L.oracle_bf16_array.argtypes = [P, ctypes.c_int64, P]
        L.oracle_bf16_patterns.restype = None
        L.oracle_bf16_patterns.argtypes = [ctypes.c_uint32, ctypes.c_int64, P]
        _lib = L
    return _lib


def derive_scalars(hp) -> Scalars:
    """Step scalars of the inverse and the forward step (sec. 4.1; appendix A),
    for the operation order hp.order (0 folded, 1 literal eq. adamw_inverse)."""
    s = Scalars()
    rc = lib().oracle_derive_scalars(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay,
                                     hp.step, getattr(hp, "order", 0), ctypes.byref(s))
    if rc != 0:
        raise ValueError("invalid AdamW hyperparameters: %r" % (hp,))
    return s


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a


def adamw_forward(p_prev, m_prev, v_prev, g, sc: Scalars):
    """One AdamW step (sec. 4.1, eq. adamw_moments; appendix A forward)."""
    p_prev, m_prev, v_prev, g = map(_f32, (p_prev, m_prev, v_prev, g))
    n = p_prev.size
    assert m_prev.size == n and v_prev.size == n and g.size == n
    p, m, v = (np.empty(n, np.float32) for _ in range(3))
    lib().oracle_adamw_forward(p_prev.ctypes.data, m_prev.ctypes.data, v_prev.ctypes.data,
                               g.ctypes.data, n, ctypes.byref(sc), p.ctypes.data,
                               m.ctypes.data, v.ctypes.data)
    return p, m, v


def invert(p, m, v, sc: Scalars):
    """theta_hat_{t-1} (sec. 4.1, eq. adamw_inverse)."""
    p, m, v = map(_f32, (p, m, v))
    n = p.size
    ph = np.empty(n, np.float32)
    lib().oracle_invert(p.ctypes.data, m.ctypes.data, v.ctypes.data, n, ctypes.byref(sc),
                        ph.ctypes.data)
    return ph


def bf16(x):
    """Q_BF16 then B_16 (sec. 4.2.1): BF16 bit patterns as uint16."""
    x = _f32(x)
    out = np.empty(x.size, np.uint16)
    lib().oracle_bf16_array(x.ctypes.data, x.size, out.ctypes.data)
    return out.reshape(x.shape)


def bf16_patterns(first: int, n: int):
    out = np.empty(n, np.uint16)
    lib().oracle_bf16_patterns(first, n, out.ctypes.data)
    return out


def detect(p, m, v, sc: Scalars, flat_begin: int = 0):
    """Converter-aligned detection of one tensor (sec. 4.2.1,
    eq. canonical_delta_detection), after the inversion of sec. 4.1.

    Returns (I, V, ph): I = flat trainer offsets (flat_begin + canonical
    index) of the changed elements in ascending order, V = their target BF16
    patterns, ph = the reconstructed previous weights.
    """
    ph = invert(p, m, v, sc)                 # sec. 4.1
    b_old = bf16(ph)                         # Q_BF16 of the previous version
    b_new = bf16(p)                          # Q_BF16 of the current version
    mask = b_new != b_old                    # M = B16(new) != B16(old)
    idx = np.flatnonzero(mask)               # I = nonzero(M)
    val = b_new[idx]                         # V = vec(new)[I]
    return idx.astype(np.int64) + np.int64(flat_begin), val, ph
