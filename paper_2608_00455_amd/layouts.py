"""Transfer-plan construction for the receiver layouts (paper sec. 4.2.2:
the plan T is precomputed from sender and receiver shard metadata;
Observation 3: the layouts fix it before synchronisation).

Host-side metadata only: the result is handed to dte_plan_create, which
validates it (coverage, bounds, single writer per receiver element).

Sender side: the flat trainer shard is a sequence of segments (one
dte_segment each).  With the canonical layout they are the Hugging Face
tensors in parameter order.  With the Megatron-Core layout they are one
trainer tensor-parallel rank's optimizer-native tensors, and the converter
of sec. 4.2.1 (appendix B) is folded into the plan: each segment is a set of
pieces, each piece a box of the segment that is a box of one canonical
tensor (fused linear_qkv: per key/value group j the g query heads, then K_j,
then V_j, eq. mcore_fused_qkv, rank r holding rows R_r, eq. mcore_tp_shard;
linear_fc1: [gate_r; up_r]; linear_proj / linear_fc2: input columns of the
rank; layernorms whole), and every plan operation is the intersection of a
sender piece with a receiver piece of the same canonical tensor.
Receiver side, per rank, a flat BF16 buffer of consecutive tensors:
  dense, tensor parallel degree P (rank r):
    embed_tokens / lm_head  rows [r V/P, (r+1) V/P)
    per layer: input_layernorm (whole), qkv_proj = [q_r; k_r; v_r] (row
    slices), q_norm, k_norm (whole), o_proj columns [r qd/P, ...),
    post_attention_layernorm (whole), gate_up_proj = [gate_r; up_r] (row
    slices), down_proj columns [r I/P, ...); then norm (whole), lm_head.
  MoE, R ranks, attention TP degree A, E experts per rank (rank r):
    per layer: input_layernorm, attention block as above on shard r % A,
    post_attention_layernorm, router (whole), w13 [E, 2I, h] with expert
    e = r E + s in slot s as [gate_e; up_e], w2 [E, h, I] with down_e.
An expert slot of w13 / w2 is addressed as its own 2-D view at the slot's
flat offset, so every plan operation has the rank of its canonical tensor.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Tuple

from .binding import DTE_MAX_DIMS, dte_op, dte_segment


@dataclass
class Piece:
    """Receiver piece: box [src_lo, src_lo + extent) of canonical tensor
    `tensor` placed at dst_lo of a receiver view."""
    tensor: int
    src_lo: Tuple[int, ...]
    extent: Tuple[int, ...]
    dst_lo: Tuple[int, ...]


@dataclass
class SPiece:
    """Sender piece: box [local_lo, local_lo + extent) of a sender segment
    holding box [canon_lo, canon_lo + extent) of canonical tensor `tensor`."""
    local_lo: Tuple[int, ...]
    extent: Tuple[int, ...]
    tensor: int
    canon_lo: Tuple[int, ...]


@dataclass
class SenderSeg:
    name: str
    shape: Tuple[int, ...]
    pieces: List[SPiece]


@dataclass
class View:
    name: str
    shape: Tuple[int, ...]
    pieces: List[Piece] = field(default_factory=list)


@dataclass
class PlanSpec:
    segments: List[Tuple[int, Tuple[int, ...]]]      # (flat_begin, shape) of sender segments
    views: List[List[Tuple[int, View]]]               # per rank: (flat base, view)
    rank_numel: List[int]
    senders: List[SenderSeg] = field(default_factory=list)

    @property
    def nranks(self) -> int:
        return len(self.rank_numel)

    def c_segments(self) -> List[dte_segment]:
        out = []
        for begin, shape in self.segments:
            sg = dte_segment()
            sg.flat_begin = begin
            sg.ndim = len(shape)
            for d in range(DTE_MAX_DIMS):
                sg.shape[d] = shape[d] if d < len(shape) else 1
            out.append(sg)
        return out

    def c_ops(self) -> List[dte_op]:
        by_tensor: Dict[int, List[Tuple[int, SPiece]]] = {}
        for si, seg in enumerate(self.senders):
            for sp in seg.pieces:
                by_tensor.setdefault(sp.tensor, []).append((si, sp))
        ops = []
        for rank, views in enumerate(self.views):
            for base, vw in views:
                nd = len(vw.shape)
                for pc in vw.pieces:
                    for si, sp in by_tensor.get(pc.tensor, []):
                        lo = [max(pc.src_lo[d], sp.canon_lo[d]) for d in range(nd)]
                        hi = [min(pc.src_lo[d] + pc.extent[d], sp.canon_lo[d] + sp.extent[d])
                              for d in range(nd)]
                        if any(lo[d] >= hi[d] for d in range(nd)):
                            continue
                        o = dte_op()
                        o.segment = si
                        o.rank = rank
                        o.dst_base = base
                        for d in range(DTE_MAX_DIMS):
                            used = d < nd
                            o.src_origin[d] = sp.local_lo[d] + lo[d] - sp.canon_lo[d] if used else 0
                            o.extent[d] = hi[d] - lo[d] if used else 1
                            o.dst_origin[d] = pc.dst_lo[d] + lo[d] - pc.src_lo[d] if used else 0
                            o.dst_shape[d] = vw.shape[d] if used else 1
                        ops.append(o)
        return ops

    @property
    def total(self) -> int:
        if not self.segments:
            return 0
        b, shp = self.segments[-1]
        n = 1
        for x in shp:
            n *= x
        return b + n


def _part(total: int, parts: int, i: int) -> Tuple[int, int]:
    if total % parts:
        raise ValueError("%d does not split evenly into %d parts" % (total, parts))
    w = total // parts
    return i * w, w


class _Index:
    """Segment lookup by (layer, role, expert)."""

    def __init__(self, wl):
        self.wl = wl
        self.key: Dict[Tuple, int] = {}
        for k, t in enumerate(wl.tensors):
            self.key[(t.layer, t.role, t.expert)] = k
        self.layers = sorted({t.layer for t in wl.tensors if t.layer is not None})

    def seg(self, layer, role, expert=None):
        return self.key.get((layer, role, expert))

    def shape(self, k):
        return tuple(self.wl.tensors[k].shape)


def _whole(ix, k, name):
    s = ix.shape(k)
    return View(name, s, [Piece(k, (0,) * len(s), s, (0,) * len(s))])


def _stack_rows(ix, name, parts):
    """View made of row slices [lo, lo+cnt) of 2-D segments, stacked in order."""
    cols = ix.shape(parts[0][0])[1]
    rows, pieces = 0, []
    for k, lo, cnt in parts:
        assert ix.shape(k)[1] == cols
        pieces.append(Piece(k, (lo, 0), (cnt, cols), (rows, 0)))
        rows += cnt
    return View(name, (rows, cols), pieces)


def _col_slice(ix, name, k, lo, cnt):
    rows = ix.shape(k)[0]
    return View(name, (rows, cnt), [Piece(k, (0, lo), (rows, cnt), (0, 0))])


def _attention_views(ix, L, P, a, pre):
    q, k, v, o = (ix.seg(L, r) for r in ("q", "k", "v", "o"))
    qlo, qn = _part(ix.shape(q)[0], P, a)
    klo, kn = _part(ix.shape(k)[0], P, a)
    views = [_stack_rows(ix, pre + "qkv_proj", [(q, qlo, qn), (k, klo, kn), (v, klo, kn)])]
    for role, nm in (("q_norm", "q_norm"), ("k_norm", "k_norm")):
        s = ix.seg(L, role)
        if s is not None:
            views.append(_whole(ix, s, pre + nm))
    olo, on = _part(ix.shape(o)[1], P, a)
    views.append(_col_slice(ix, pre + "o_proj", o, olo, on))
    return views


def _dense_rank(ix, r, P):
    views = []
    emb = ix.seg(None, "embed")
    if emb is not None:
        lo, n = _part(ix.shape(emb)[0], P, r)
        views.append(_stack_rows(ix, "embed_tokens", [(emb, lo, n)]))
    for L in ix.layers:
        pre = "layers.%d." % L
        views.append(_whole(ix, ix.seg(L, "in_norm"), pre + "input_layernorm"))
        views += _attention_views(ix, L, P, r, pre)
        views.append(_whole(ix, ix.seg(L, "post_norm"), pre + "post_attention_layernorm"))
        g, u, d = ix.seg(L, "gate"), ix.seg(L, "up"), ix.seg(L, "down")
        lo, n = _part(ix.shape(g)[0], P, r)
        views.append(_stack_rows(ix, pre + "gate_up_proj", [(g, lo, n), (u, lo, n)]))
        dlo, dn = _part(ix.shape(d)[1], P, r)
        views.append(_col_slice(ix, pre + "down_proj", d, dlo, dn))
    fn = ix.seg(None, "final_norm")
    if fn is not None:
        views.append(_whole(ix, fn, "norm"))
    head = ix.seg(None, "lm_head")
    if head is not None:
        lo, n = _part(ix.shape(head)[0], P, r)
        views.append(_stack_rows(ix, "lm_head", [(head, lo, n)]))
    return views


def _moe_rank(ix, r, R, A, E):
    views = []
    for L in ix.layers:
        pre = "layers.%d." % L
        views.append(_whole(ix, ix.seg(L, "in_norm"), pre + "input_layernorm"))
        views += _attention_views(ix, L, A, r % A, pre)
        views.append(_whole(ix, ix.seg(L, "post_norm"), pre + "post_attention_layernorm"))
        views.append(_whole(ix, ix.seg(L, "router"), pre + "router"))
        for slot in range(E):                       # w13 slots, then w2 slots
            e = r * E + slot
            g, u = ix.seg(L, "expert_gate", e), ix.seg(L, "expert_up", e)
            ie = ix.shape(g)[0]
            views.append(_stack_rows(ix, pre + "w13[%d]" % slot, [(g, 0, ie), (u, 0, ie)]))
        for slot in range(E):
            e = r * E + slot
            views.append(_whole(ix, ix.seg(L, "expert_down", e), pre + "w2[%d]" % slot))
    return views


def _whole_piece(shape, k):
    return SPiece((0,) * len(shape), tuple(shape), k, (0,) * len(shape))


def sender_segments(wl) -> List[SenderSeg]:
    """The trainer shard's segments and their canonical pieces."""
    ix = _Index(wl)
    sd = wl.sender
    if sd.kind == "canonical":
        return [SenderSeg(t.name, tuple(t.shape), [_whole_piece(t.shape, k)])
                for k, t in enumerate(wl.tensors)]
    if sd.kind != "mcore":
        raise ValueError("unknown sender layout %r" % sd.kind)
    if wl.receiver.kind != "tp":
        raise ValueError("the Megatron-Core sender layout is built for dense models")
    P, r = sd.tp, sd.rank
    d = wl.dims
    g, dh = d.heads_q // d.heads_kv, d.head_dim
    segs: List[SenderSeg] = []

    def whole(k, name):
        segs.append(SenderSeg(name, ix.shape(k), [_whole_piece(ix.shape(k), k)]))

    def row_slice(k, name):
        rows, cols = ix.shape(k)
        lo, n = _part(rows, P, r)
        segs.append(SenderSeg(name, (n, cols), [SPiece((0, 0), (n, cols), k, (lo, 0))]))

    def col_slice(k, name):
        rows, cols = ix.shape(k)
        lo, n = _part(cols, P, r)
        segs.append(SenderSeg(name, (rows, n), [SPiece((0, 0), (rows, n), k, (0, lo))]))

    emb = ix.seg(None, "embed")
    if emb is not None:
        row_slice(emb, "embedding.word_embeddings.weight")
    for L in ix.layers:
        pre = "decoder.layers.%d." % L
        whole(ix.seg(L, "in_norm"), pre + "self_attention.linear_qkv.layer_norm_weight")
        q, k, v = ix.seg(L, "q"), ix.seg(L, "k"), ix.seg(L, "v")
        h = ix.shape(q)[1]
        j0, nj = _part(d.heads_kv, P, r)          # key/value groups of this rank
        per_group = (g + 2) * dh
        pieces = []
        for jj in range(nj):
            j = j0 + jj
            base = jj * per_group
            pieces.append(SPiece((base, 0), (g * dh, h), q, (j * g * dh, 0)))
            pieces.append(SPiece((base + g * dh, 0), (dh, h), k, (j * dh, 0)))
            pieces.append(SPiece((base + (g + 1) * dh, 0), (dh, h), v, (j * dh, 0)))
        segs.append(SenderSeg(pre + "self_attention.linear_qkv.weight", (nj * per_group, h),
                              pieces))
        for role, nm in (("q_norm", "q_layernorm"), ("k_norm", "k_layernorm")):
            kk = ix.seg(L, role)
            if kk is not None:
                whole(kk, pre + "self_attention." + nm + ".weight")
        col_slice(ix.seg(L, "o"), pre + "self_attention.linear_proj.weight")
        whole(ix.seg(L, "post_norm"), pre + "mlp.linear_fc1.layer_norm_weight")
        gt, up = ix.seg(L, "gate"), ix.seg(L, "up")
        rows, cols = ix.shape(gt)
        lo, n = _part(rows, P, r)
        segs.append(SenderSeg(pre + "mlp.linear_fc1.weight", (2 * n, cols),
                              [SPiece((0, 0), (n, cols), gt, (lo, 0)),
                               SPiece((n, 0), (n, cols), up, (lo, 0))]))
        col_slice(ix.seg(L, "down"), pre + "mlp.linear_fc2.weight")
    fn = ix.seg(None, "final_norm")
    if fn is not None:
        whole(fn, "decoder.final_layernorm.weight")
    head = ix.seg(None, "lm_head")
    if head is not None:
        row_slice(head, "output_layer.weight")
    return segs


def build_spec(wl) -> PlanSpec:
    ix = _Index(wl)
    senders = sender_segments(wl)
    segments, pos = [], 0
    for sg in senders:
        segments.append((pos, tuple(sg.shape)))
        n = 1
        for x in sg.shape:
            n *= x
        pos += n
    rc = wl.receiver
    per_rank = []
    for r in range(rc.nranks):
        if rc.kind == "tp":
            vs = _dense_rank(ix, r, rc.tp)
        elif rc.kind == "moe_ep":
            if rc.ranks % rc.attn_tp:
                raise ValueError("ranks must be a multiple of the attention TP degree")
            vs = _moe_rank(ix, r, rc.ranks, rc.attn_tp, rc.experts_per_rank)
        else:
            raise ValueError("unknown receiver layout %r" % rc.kind)
        per_rank.append(vs)
    placed, numel = [], []
    for vs in per_rank:
        base, lst = 0, []
        for vw in vs:
            lst.append((base, vw))
            n = 1
            for x in vw.shape:
                n *= x
            base += n
        placed.append(lst)
        numel.append(base)
    return PlanSpec(segments, placed, numel, senders)


def store_pieces(wl):
    """The trainer shard as pieces of canonical tensors for the storage
    path (dte_store_piece rows: sender_begin, sender_end, segment,
    local_cols, canon_cols, canon_row0, canon_col0).  Every sender piece
    covers whole rows of its segment.  Tensors that every tensor-parallel
    rank holds whole (the norms) are published by rank 0 only."""
    rows, pos = [], 0
    replicated = wl.sender.kind == "mcore" and wl.sender.tp > 1
    for sg in sender_segments(wl):
        numel = 1
        for x in sg.shape:
            numel *= x
        cols = sg.shape[-1] if len(sg.shape) == 2 else numel
        for sp in sorted(sg.pieces, key=lambda x: x.local_lo):
            t = wl.tensors[sp.tensor]
            if len(sg.shape) == 2:
                if sp.extent[1] != cols or sp.local_lo[1] != 0:
                    raise ValueError("store pieces must cover whole rows of %s" % sg.name)
                b = pos + sp.local_lo[0] * cols
                e = b + sp.extent[0] * cols
                owner = sp.tensor
                rows.append((b, e, owner, cols, t.shape[1], sp.canon_lo[0], sp.canon_lo[1]))
            else:
                owner = sp.tensor if not (replicated and wl.sender.rank != 0) else -1
                rows.append((pos, pos + numel, owner, numel, numel, 0, 0))
        pos += numel
    return rows
