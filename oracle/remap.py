"""Oracle's receiver-space remap and direct sparse apply (test
infrastructure only).

remap: sec. 4.2.2 -- for each changed flat index, u = unravel(i, n_s)
(eq. canonical_unravel); the change belongs to op o when
a_s <= u < a_s + e component-wise; its receiver index is
j_r = ravel(u - a_s + a_r, n_r) (eq. receiver_local_remapping), here offset
by the flat base of the receiver view inside rank r's buffer.  Every op of
the plan is applied, so a change is partitioned or replicated as the layout
says.  The value is carried unchanged.

apply: sec. 4.3, eq. direct_sparse_apply -- vec(W_r)[I] <- V.
"""
from __future__ import annotations

import numpy as np


def remap(plan, idx, val):
    """(I, V) in flat trainer offsets -> per-rank (off, val), each sorted by off.

    Entries outside every segment are an error (assertion)."""
    idx = np.asarray(idx, dtype=np.int64)
    val = np.asarray(val)            # BF16 patterns (uint16), or any tag dtype
    begins = np.asarray(plan.seg_begin, dtype=np.int64)
    assert idx.size == 0 or (idx.min() >= 0 and idx.max() < plan.total)
    seg = np.searchsorted(begins, idx, side="right") - 1
    ops_of = {}
    for o in plan.ops:
        ops_of.setdefault(o.segment, []).append(o)
    out_off = [[] for _ in range(plan.nranks)]
    out_val = [[] for _ in range(plan.nranks)]
    order = np.argsort(seg, kind="stable")
    seg_sorted = seg[order]
    bounds = np.flatnonzero(np.diff(seg_sorted)) + 1
    starts = np.concatenate([[0], bounds])
    ends = np.concatenate([bounds, [seg_sorted.size]])
    for lo, hi in zip(starts, ends):
        if lo == hi:
            continue
        s = int(seg_sorted[lo])
        sel = order[lo:hi]
        li = idx[sel] - begins[s]
        shape = plan.seg_shape[s]
        assert np.all((li >= 0) & (li < int(np.prod(shape))))
        u = np.unravel_index(li, shape)                       # eq. canonical_unravel
        for o in ops_of.get(s, []):
            inside = np.ones(li.size, dtype=bool)
            for d in range(len(shape)):                       # containment
                inside &= (u[d] >= o.src_origin[d]) & (u[d] < o.src_origin[d] + o.extent[d])
            if not inside.any():
                continue
            coord = tuple(u[d][inside] - o.src_origin[d] + o.dst_origin[d]
                          for d in range(len(shape)))
            j = np.ravel_multi_index(coord, o.dst_shape)     # eq. receiver_local_remapping
            out_off[o.rank].append(np.int64(o.dst_base) + j.astype(np.int64))
            out_val[o.rank].append(val[sel][inside])
    res = []
    for r in range(plan.nranks):
        off = np.concatenate(out_off[r]) if out_off[r] else np.zeros(0, np.int64)
        v = np.concatenate(out_val[r]) if out_val[r] else np.zeros(0, val.dtype)
        srt = np.argsort(off, kind="stable")
        res.append((off[srt], v[srt]))
    return res


def apply(shards, buckets):
    """vec(W_r)[I] <- V for every rank (in place); returns shards."""
    for r, (off, v) in enumerate(buckets):
        shards[r][off] = v
    return shards


def layout(plan, values_flat):
    """Receiver shards holding every canonical element: the dense image of
    the remap of all N indices, as a list of per-rank uint16 arrays."""
    n = plan.total
    values_flat = np.asarray(values_flat, dtype=np.uint16)
    assert values_flat.size == n
    shards = [np.zeros(plan.rank_numel[r], np.uint16) for r in range(plan.nranks)]
    buckets = remap(plan, np.arange(n, dtype=np.int64), values_flat)
    return apply(shards, buckets)
