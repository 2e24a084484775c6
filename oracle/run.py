"""Oracle driver: a whole workload on the CPU (test infrastructure only).

State generation (seeded draws, then one forward AdamW step), then the
method in the paper's order: inversion (sec. 4.1), BF16 detection
(sec. 4.2.1), receiver remap (sec. 4.2.2), direct apply (sec. 4.3).
Tensors are processed one at a time (the paper's streaming per converter
unit, sec. 4.1) and, for large tensors, in element windows; a thread pool
runs independent windows side by side.
"""
from __future__ import annotations

import os
import time
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import synth
from synth.workloads import KIND_GRAD, KIND_M_PREV, KIND_P_PREV, KIND_V_PREV

from . import core


@dataclass
class Window:
    tensor: int
    lo: int            # element range [lo, hi) inside the tensor
    hi: int


@dataclass
class Diagnostics:
    n: int = 0
    changed: int = 0              # |I|
    fp32_recon_mismatch: int = 0  # #{ph != p_prev} as binary32 bits
    bf16_recon_mismatch: int = 0  # #{b(ph) != b(p_prev)}
    true_changed: int = 0         # #{b(p_prev) != b(p)}
    apply_vs_prev_diff: int = 0   # #{b(p_prev) != b(ph) and b(ph) == b(p)}

    def add(self, o: "Diagnostics"):
        for f in self.__dataclass_fields__:
            setattr(self, f, getattr(self, f) + getattr(o, f))


@dataclass
class WindowResult:
    window: Window
    idx: np.ndarray
    val: np.ndarray
    diag: Diagnostics
    ph: Optional[np.ndarray] = None
    p: Optional[np.ndarray] = None
    m: Optional[np.ndarray] = None
    v: Optional[np.ndarray] = None
    p_prev: Optional[np.ndarray] = None


def draws(wl, k: int, lo: int, hi: int, threads: int = 1):
    """Pre-step weights, moments and gradient of tensor k, elements [lo, hi)
    (zero moments and gradient for an untouched tensor)."""
    t = wl.tensors[k]
    n = hi - lo
    p_prev = synth.draw_cpu(n, wl.seed, k, KIND_P_PREV, lo, threads)
    if t.touched:
        m_prev = synth.draw_cpu(n, wl.seed, k, KIND_M_PREV, lo, threads)
        v_prev = synth.draw_cpu(n, wl.seed, k, KIND_V_PREV, lo, threads)
        g = synth.draw_cpu(n, wl.seed, k, KIND_GRAD, lo, threads)
    else:
        m_prev = np.zeros(n, np.float32)
        v_prev = np.zeros(n, np.float32)
        g = np.zeros(n, np.float32)
    return p_prev, m_prev, v_prev, g


def state(wl, k: int, lo: int, hi: int, sc: core.Scalars, threads: int = 1):
    """Pre-step draws and the post-step state of tensor k, elements [lo, hi)."""
    p_prev, m_prev, v_prev, g = draws(wl, k, lo, hi, threads)
    p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)
    return p_prev, p, m, v


def count_diagnostics(p_prev, ph, p, changed: int) -> Diagnostics:
    """Reconstruction diagnostics of one window.  The inverse gives a
    numerical reconstruction of the previous weights, not a bitwise
    recovery (sec. 4.1), so beside the delta size the oracle counts, per
    element of the window: binary32 patterns of theta_hat that differ from
    the true pre-step weights p_prev; BF16 patterns that differ, b(theta_hat)
    != b(p_prev); the true BF16 changes b(p_prev) != b(p); and the elements
    that a receiver holding b(p_prev) would keep stale after apply,
    b(p_prev) != b(theta_hat) == b(p)."""
    b_prev = core.bf16(p_prev)
    b_ph = core.bf16(ph)
    b_p = core.bf16(p)
    d = Diagnostics(n=int(p.size), changed=changed)
    d.fp32_recon_mismatch = int(np.count_nonzero(ph.view(np.uint32) != p_prev.view(np.uint32)))
    d.bf16_recon_mismatch = int(np.count_nonzero(b_ph != b_prev))
    d.true_changed = int(np.count_nonzero(b_prev != b_p))
    d.apply_vs_prev_diff = int(np.count_nonzero((b_prev != b_ph) & (b_ph == b_p)))
    return d


def run_window(wl, w: Window, sc: core.Scalars, keep=(), threads: int = 1) -> WindowResult:
    begin = wl.flat_begins()[w.tensor]
    p_prev, p, m, v = state(wl, w.tensor, w.lo, w.hi, sc, threads)
    idx, val, ph = core.detect(p, m, v, sc, begin + w.lo)
    d = count_diagnostics(p_prev, ph, p, int(idx.size))
    r = WindowResult(w, idx, val, d)
    for name in keep:
        setattr(r, name, locals()[name])
    return r


def windows(wl, max_window: int = 1 << 24, tensors=None) -> List[Window]:
    out = []
    for k, t in enumerate(wl.tensors):
        if tensors is not None and k not in tensors:
            continue
        for lo in range(0, t.numel, max_window):
            out.append(Window(k, lo, min(t.numel, lo + max_window)))
    return out


def scalars(wl, hp=None) -> List[core.Scalars]:
    """Step scalars of every tensor, from its parameter group's
    hyperparameters (the weight-decay coefficient is per group, sec. 4.1)."""
    return [core.derive_scalars(wl.group_hp(k, hp)) for k in range(len(wl.tensors))]


@dataclass
class Result:
    idx: np.ndarray
    val: np.ndarray
    diag: Diagnostics
    parts: List[WindowResult] = field(default_factory=list)
    seconds: float = 0.0


def extract(wl, hp=None, wins: Optional[List[Window]] = None, keep=(), threads: int = 0,
            max_window: int = 1 << 24) -> Result:
    """Detection over the given windows (default: the whole trainer shard)."""
    sc = scalars(wl, hp)
    wins = wins if wins is not None else windows(wl, max_window)
    threads = threads or synth.default_threads()
    t0 = time.perf_counter()
    if threads <= 1 or len(wins) <= 1:
        parts = [run_window(wl, w, sc[w.tensor], keep, threads=max(1, threads)) for w in wins]
    else:
        with ThreadPoolExecutor(threads) as ex:
            parts = list(ex.map(lambda w: run_window(wl, w, sc[w.tensor], keep), wins))
    diag = Diagnostics()
    for r in parts:
        diag.add(r.diag)
    idx = np.concatenate([r.idx for r in parts]) if parts else np.zeros(0, np.int64)
    val = np.concatenate([r.val for r in parts]) if parts else np.zeros(0, np.uint16)
    srt = np.argsort(idx, kind="stable")
    return Result(idx[srt], val[srt], diag, parts if keep else [], time.perf_counter() - t0)


def flat(parts: List[WindowResult], name: str) -> np.ndarray:
    """Concatenate a kept per-window array in window order."""
    return np.concatenate([getattr(r, name) for r in parts])


def cpu_threads() -> int:
    return synth.default_threads()


def host_description() -> str:
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return "%s, %d usable cores" % (model or "unknown CPU", len(os.sched_getaffinity(0)))
