"""Device buffers and call sequencing for the three hot calls.

torch is used for device memory and streams only; every step of the path
runs inside libdte.so.  `DeltaPipeline` owns the delta buffers (I, V and
the cursor), the per-receiver buckets and counts, and the receiver shards,
and chains dte_extract_delta -> dte_remap -> dte_apply on one stream.
`generate_state` produces a synthetic post-step trainer state on the device
(seeded draws from `synth`, then the library's AdamW step).
"""
from __future__ import annotations

from typing import List, Optional

import torch

from . import binding as B
from .layouts import PlanSpec, build_spec


def check_buffer(t, n, dtype, device, name):
    """The library takes raw addresses and element counts, so a buffer of
    the wrong type, layout, device or length would be read or written out
    of bounds: refuse it here."""
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s: expected a torch.Tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s: dtype %s, expected %s" % (name, t.dtype, dtype))
    if t.device != device:
        raise ValueError("%s: on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s: not contiguous" % name)
    if t.numel() < n:
        raise ValueError("%s: %d elements, %d needed" % (name, t.numel(), n))


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Plan:
    """Owned dte_plan handle."""

    def __init__(self, spec: PlanSpec):
        self.spec = spec
        self.handle = B.dte_plan_create(spec.c_segments(), spec.c_ops(), spec.nranks,
                                        spec.rank_numel)
        self.total, self.nranks, self.max_replication = B.dte_plan_info(self.handle)

    def close(self):
        if self.handle:
            B.dte_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover - interpreter shutdown order
        try:
            self.close()
        except Exception:
            pass


class DeltaPipeline:
    def __init__(self, spec: PlanSpec, capacity: int, rank_capacity: Optional[List[int]] = None,
                 device="cuda", shards: Optional[List[torch.Tensor]] = None,
                 ordered: bool = False):
        self.plan = Plan(spec)
        self.ordered = ordered
        self.device = torch.device(device)
        self.capacity = int(capacity)
        R = self.plan.nranks
        rc = rank_capacity or [self.capacity] * R
        self.rank_capacity = [int(x) for x in rc]
        self.idx = torch.empty(max(1, self.capacity), dtype=torch.int64, device=self.device)
        self.val = torch.empty(max(1, self.capacity), dtype=torch.int16, device=self.device)
        self.cursor = torch.zeros(1, dtype=torch.int64, device=self.device)
        self.off = [torch.empty(max(1, c), dtype=torch.int64, device=self.device)
                    for c in self.rank_capacity]
        self.rval = [torch.empty(max(1, c), dtype=torch.int16, device=self.device)
                     for c in self.rank_capacity]
        self.rank_count = torch.zeros(R, dtype=torch.int64, device=self.device)
        if shards is None:
            shards = [torch.zeros(max(1, n), dtype=torch.int16, device=self.device)
                      for n in spec.rank_numel]
        if len(shards) != R:
            raise ValueError("shards: %d buffers for %d receiver ranks" % (len(shards), R))
        for r, (t, n) in enumerate(zip(shards, spec.rank_numel)):
            check_buffer(t, n, torch.int16, self.idx.device, "shards[%d]" % r)
        self.shards = shards
        self.workspace = None
        if ordered:
            nbytes = B.dte_ordered_workspace_bytes(self.capacity)
            self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)

    # -- the three hot calls ------------------------------------------------
    def reset(self, stream=None):
        """Start a fresh delta (cursor = 0); a fill kernel, graph-safe."""
        with torch.cuda.stream(stream) if stream is not None else _null():
            self.cursor.zero_()

    def _check_state(self, p, m, v, n, out_prev=None) -> int:
        """Element count of the call (all of p when n is None), after
        checking p, m, v (and out_prev) for it."""
        if not isinstance(p, torch.Tensor):
            raise TypeError("p: expected a torch.Tensor")
        n = p.numel() if n is None else int(n)
        for t, name in ((p, "p"), (m, "m"), (v, "v")):
            check_buffer(t, n, torch.float32, self.idx.device, name)
        if out_prev is not None:
            check_buffer(out_prev, n, torch.float32, self.idx.device, "out_prev")
        return n

    def extract(self, p, m, v, hp, n=None, index_base=0, out_prev=None, stream=None):
        n = self._check_state(p, m, v, n, out_prev)
        prev = out_prev.data_ptr() if out_prev is not None else 0
        if self.ordered:
            B.dte_extract_delta_ordered(p.data_ptr(), m.data_ptr(), v.data_ptr(), n, index_base,
                                        hp, self.idx.data_ptr(), self.val.data_ptr(),
                                        self.capacity, self.cursor.data_ptr(),
                                        self.workspace.data_ptr(), self.workspace.numel(), prev,
                                        _stream(stream))
        else:
            B.dte_extract_delta(p.data_ptr(), m.data_ptr(), v.data_ptr(), n, index_base, hp,
                                self.idx.data_ptr(), self.val.data_ptr(), self.capacity,
                                self.cursor.data_ptr(), prev, _stream(stream))

    def remap(self, stream=None):
        B.dte_remap(self.plan.handle, self.idx.data_ptr(), self.val.data_ptr(),
                    self.cursor.data_ptr(), self.capacity, [t.data_ptr() for t in self.off],
                    [t.data_ptr() for t in self.rval], self.rank_capacity,
                    self.rank_count.data_ptr(), _stream(stream))

    def apply(self, stream=None):
        B.dte_apply(self.plan.handle, [t.data_ptr() for t in self.shards],
                    [t.data_ptr() for t in self.off], [t.data_ptr() for t in self.rval],
                    self.rank_count.data_ptr(), self.rank_capacity, _stream(stream))

    def extract_runs(self, p, m, v, runs, out_prev=None, stream=None):
        """One dte_extract_delta per run (begin, end, hp) of the flat shard,
        appending to the same delta (parameter groups, sec. 4.1)."""
        for b, e, hp in runs:
            self.extract(p[b:e], m[b:e], v[b:e], hp, n=e - b, index_base=b,
                         out_prev=out_prev[b:e] if out_prev is not None else None,
                         stream=stream)

    def extract_remap(self, p, m, v, hp, n=None, index_base=0, stream=None):
        """Changed entries routed straight into the buckets (adds to
        rank_count and to the cursor; clear both first, see step_fused)."""
        n = self._check_state(p, m, v, n)
        B.dte_extract_remap(p.data_ptr(), m.data_ptr(), v.data_ptr(), n, index_base, hp,
                            self.plan.handle, [t.data_ptr() for t in self.off],
                            [t.data_ptr() for t in self.rval], self.rank_capacity,
                            self.rank_count.data_ptr(), self.cursor.data_ptr(), _stream(stream))

    def step_fused(self, p, m, v, hp, stream=None, runs=None):
        """The step with detection and remap in one kernel, then apply."""
        with torch.cuda.stream(stream) if stream is not None else _null():
            self.cursor.zero_()
            self.rank_count.zero_()
        if runs is None:
            self.extract_remap(p, m, v, hp, stream=stream)
        else:
            for b, e, h in runs:
                self.extract_remap(p[b:e], m[b:e], v[b:e], h, n=e - b, index_base=b,
                                   stream=stream)
        self.apply(stream)

    def step(self, p, m, v, hp, stream=None, runs=None):
        """reset, extract (over `runs` when the shard has several parameter
        groups), remap, apply."""
        self.reset(stream)
        if runs is None:
            self.extract(p, m, v, hp, stream=stream)
        else:
            self.extract_runs(p, m, v, runs, stream=stream)
        self.remap(stream)
        self.apply(stream)

    # -- host read-back (tests) --------------------------------------------
    def delta(self, raw=False):
        """(idx, val) on the host, sorted by idx (as written with raw=True);
        and the cursor value."""
        total = int(self.cursor.item())
        k = min(total, self.capacity)
        idx = self.idx[:k].cpu().numpy()
        val = self.val[:k].cpu().numpy().view("uint16")
        if raw:
            return idx, val, total
        order = idx.argsort(kind="stable")
        return idx[order], val[order], total

    def buckets(self):
        counts = self.rank_count.cpu().numpy()
        out = []
        for r in range(self.plan.nranks):
            k = min(int(counts[r]), self.rank_capacity[r])
            off = self.off[r][:k].cpu().numpy()
            val = self.rval[r][:k].cpu().numpy().view("uint16")
            order = off.argsort(kind="stable")
            out.append((off[order], val[order]))
        return out, counts

    def close(self):
        self.plan.close()


class _null:
    def __enter__(self):
        return None

    def __exit__(self, *a):
        return False


def generate_state(wl, hp=None, device="cuda"):
    """Post-step state (p, m, v) of workload `wl` on the device, laid out as
    the trainer shard (the sender segments of `layouts.sender_segments`).

    Every element is drawn (synth) at its canonical coordinates, so the
    canonical and Megatron-Core layouts hold the same model state; then one
    dte_adamw_forward over the whole flat shard.  Untouched tensors get zero
    moments and gradient.  Returns three flat float32 tensors.
    """
    import synth
    from synth.workloads import KIND_GRAD, KIND_M_PREV, KIND_P_PREV, KIND_V_PREV

    from .layouts import sender_segments

    hp = hp or wl.hp
    segs = sender_segments(wl)
    n = 0
    for sg in segs:
        k = 1
        for x in sg.shape:
            k *= x
        n += k
    dev = torch.device(device)
    p = torch.empty(n, dtype=torch.float32, device=dev)
    m = torch.empty(n, dtype=torch.float32, device=dev)
    v = torch.empty(n, dtype=torch.float32, device=dev)
    g = torch.empty(n, dtype=torch.float32, device=dev)
    s = torch.cuda.current_stream().cuda_stream
    kinds = ((p, KIND_P_PREV), (m, KIND_M_PREV), (v, KIND_V_PREV), (g, KIND_GRAD))
    begin = 0
    for sg in segs:
        numel = 1
        for x in sg.shape:
            numel *= x
        for sp in sg.pieces:
            t = wl.tensors[sp.tensor]
            whole = tuple(sp.extent) == tuple(t.shape)
            assert not whole or not any(sp.local_lo)
            for buf, kind in kinds:
                if kind != KIND_P_PREV and not t.touched:
                    buf[begin:begin + numel].zero_()
                    continue
                if whole:
                    synth.fill_gpu(buf[begin:].data_ptr(), t.numel, wl.seed, sp.tensor, kind, 0, s)
                else:
                    # 2-D piece: extent rows x cols at local_lo of the segment
                    cols = sg.shape[1]
                    first = begin + sp.local_lo[0] * cols + sp.local_lo[1]
                    synth.fill_gpu_2d(buf[first:].data_ptr(), sp.extent[0], sp.extent[1], cols,
                                      wl.seed, sp.tensor, kind, sp.canon_lo[0], sp.canon_lo[1],
                                      t.shape[1], s)
        begin += numel
    for b, e, h in group_runs(wl, hp):
        B.dte_adamw_forward(p[b:].data_ptr(), m[b:].data_ptr(), v[b:].data_ptr(),
                            g[b:].data_ptr(), e - b, h, s)
    torch.cuda.current_stream().synchronize()
    del g
    return p, m, v


def group_runs(wl, hp=None):
    """Maximal runs [begin, end) of consecutive sender segments whose
    parameter groups derive bit-identical step scalars, with the group's
    hyperparameters: one extract call per run.  Without parameter groups,
    or where the groups' scalars coincide (at small learning rates the
    decay factor rounds to 1 whatever the weight decay), this is one run
    over the whole shard."""
    from .layouts import sender_segments

    hp = hp or wl.hp
    runs = []
    begin = 0
    for sg in sender_segments(wl):
        numel = 1
        for x in sg.shape:
            numel *= x
        h = wl.group_hp(sg.pieces[0].tensor, hp)
        key = bytes(B.dte_derive_scalars(h))
        if runs and runs[-1][3] == key:
            runs[-1][1] = begin + numel
        else:
            runs.append([begin, begin + numel, h, key])
        begin += numel
    return [(b, e, h) for b, e, h, _ in runs]


def spec_for(wl) -> PlanSpec:
    return build_spec(wl)
