"""Oracle's transfer plan (test infrastructure only).

Builds the paper's transfer plan T (sec. 4.2.2): for each canonical
parameter p and receiver r, the hyperrectangular overlap between the
sender's canonical tensor view (shape n_s) and the receiver-local shard
(shape n_r), given by the origins a_s, a_r and the extent e.

The receiver layouts are a reading of the inference engine's sharding (the
paper gives only the fused-QKV example of appendix B):
  dense TP=P: qkv_proj = [q_r; k_r; v_r], gate_up_proj = [gate_r; up_r]
  (row slices), o_proj and down_proj split along their input columns,
  embed_tokens and lm_head split by vocabulary rows, norms replicated;
  per-rank flat order embed, per layer [input_layernorm, qkv_proj, q_norm,
  k_norm, o_proj, post_attention_layernorm, gate_up_proj, down_proj], norm,
  lm_head.
  MoE: expert e on rank e // E in slot e % E of w13 [E, 2I, h] (gate rows
  then up rows) and w2 [E, h, I]; attention TP=A on shard r % A, replicated
  over ranks // A groups; router and norms replicated on every rank.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Tuple


@dataclass
class Op:
    segment: int
    rank: int
    dst_base: int                 # flat offset of the receiver view in rank's buffer
    src_origin: Tuple[int, ...]   # a_s
    extent: Tuple[int, ...]       # e
    dst_origin: Tuple[int, ...]   # a_r
    dst_shape: Tuple[int, ...]    # n_r


@dataclass
class Plan:
    seg_begin: List[int]
    seg_shape: List[Tuple[int, ...]]
    ops: List[Op]
    rank_numel: List[int]
    views: List[List[Tuple[str, int, Tuple[int, ...]]]]   # per rank: (name, base, shape)

    @property
    def nranks(self):
        return len(self.rank_numel)

    @property
    def total(self):
        return self.seg_begin[-1] + _prod(self.seg_shape[-1]) if self.seg_begin else 0


def _prod(shape):
    n = 1
    for s in shape:
        n *= s
    return n


class _RankBuffer:
    def __init__(self):
        self.size = 0
        self.views = []

    def view(self, name, shape):
        base = self.size
        self.views.append((name, base, tuple(shape)))
        self.size += _prod(shape)
        return base


def build_plan(wl) -> Plan:
    seg_begin, seg_shape, seg_of = [], [], {}
    pos = 0
    for k, t in enumerate(wl.tensors):
        seg_begin.append(pos)
        seg_shape.append(tuple(t.shape))
        seg_of[t.name] = k
        pos += t.numel
    rc = wl.receiver
    R = rc.nranks
    bufs = [_RankBuffer() for _ in range(R)]
    ops: List[Op] = []

    def whole(seg, rank, base, shape):
        nd = len(shape)
        ops.append(Op(seg, rank, base, (0,) * nd, tuple(shape), (0,) * nd, tuple(shape)))

    def rows(seg, rank, base, dst_shape, src_row, nrows, dst_row):
        cols = seg_shape[seg][1]
        ops.append(Op(seg, rank, base, (src_row, 0), (nrows, cols), (dst_row, 0),
                      tuple(dst_shape)))

    def cols(seg, rank, base, dst_shape, src_col, ncols):
        nrows = seg_shape[seg][0]
        ops.append(Op(seg, rank, base, (0, src_col), (nrows, ncols), (0, 0), tuple(dst_shape)))

    by_layer = {}
    for k, t in enumerate(wl.tensors):
        by_layer.setdefault(t.layer, {}).setdefault(t.role, []).append(k)

    def one(layer, role):
        ks = by_layer.get(layer, {}).get(role, [])
        assert len(ks) <= 1
        return ks[0] if ks else None

    def replicated(seg, name, ranks):
        for r in ranks:
            whole(seg, r, bufs[r].view(name, seg_shape[seg]), seg_shape[seg])

    def vocab_rows(seg, name, P, ranks_of_shard):
        V, h = seg_shape[seg]
        assert V % P == 0
        for sh in range(P):
            for r in ranks_of_shard(sh):
                base = bufs[r].view(name, (V // P, h))
                rows(seg, r, base, (V // P, h), sh * (V // P), V // P, 0)

    def attention(layer, P, ranks_of_shard, pre):
        q, k, v, o = (one(layer, x) for x in ("q", "k", "v", "o"))
        qn, kn = one(layer, "q_norm"), one(layer, "k_norm")
        qd, h = seg_shape[q]
        kd = seg_shape[k][0]
        assert qd % P == 0 and kd % P == 0
        qs, ks = qd // P, kd // P
        for sh in range(P):
            for r in ranks_of_shard(sh):
                shape = (qs + 2 * ks, h)
                base = bufs[r].view(pre + "qkv_proj", shape)
                rows(q, r, base, shape, sh * qs, qs, 0)
                rows(k, r, base, shape, sh * ks, ks, qs)
                rows(v, r, base, shape, sh * ks, ks, qs + ks)
                if qn is not None:
                    whole(qn, r, bufs[r].view(pre + "q_norm", seg_shape[qn]), seg_shape[qn])
                if kn is not None:
                    whole(kn, r, bufs[r].view(pre + "k_norm", seg_shape[kn]), seg_shape[kn])
                oshape = (seg_shape[o][0], qs)
                cols(o, r, bufs[r].view(pre + "o_proj", oshape), oshape, sh * qs, qs)

    if rc.kind == "tp":
        P = R
        solo = lambda sh: [sh]  # noqa: E731
        emb = [k for k, t in enumerate(wl.tensors) if t.role == "embed"]
        for k in emb:
            vocab_rows(k, "embed_tokens", P, solo)
        layers = sorted(x for x in by_layer if x is not None)
        for layer in layers:
            pre = "layers.%d." % layer
            attn_ranks = range(R)
            # input_layernorm precedes the attention block in the rank buffer
            replicated(one(layer, "in_norm"), pre + "input_layernorm", attn_ranks)
            # attention emits qkv, q_norm, k_norm, o per rank in rank order;
            # the rank buffers are independent, so per-rank order is preserved
            attention(layer, P, solo, pre)
            replicated(one(layer, "post_norm"), pre + "post_attention_layernorm", range(R))
            g, u, d = one(layer, "gate"), one(layer, "up"), one(layer, "down")
            I, h = seg_shape[g]
            assert I % P == 0
            Is = I // P
            for r in range(R):
                shape = (2 * Is, h)
                base = bufs[r].view(pre + "gate_up_proj", shape)
                rows(g, r, base, shape, r * Is, Is, 0)
                rows(u, r, base, shape, r * Is, Is, Is)
                dshape = (seg_shape[d][0], Is)
                cols(d, r, bufs[r].view(pre + "down_proj", dshape), dshape, r * Is, Is)
        for k, t in enumerate(wl.tensors):
            if t.role == "final_norm":
                replicated(k, "norm", range(R))
        for k, t in enumerate(wl.tensors):
            if t.role == "lm_head":
                vocab_rows(k, "lm_head", P, solo)
    elif rc.kind == "moe_ep":
        A, E = rc.attn_tp, rc.experts_per_rank
        assert R % A == 0
        group = lambda sh: [r for r in range(R) if r % A == sh]  # noqa: E731
        layers = sorted(x for x in by_layer if x is not None)
        for layer in layers:
            pre = "layers.%d." % layer
            replicated(one(layer, "in_norm"), pre + "input_layernorm", range(R))
            attention(layer, A, group, pre)
            replicated(one(layer, "post_norm"), pre + "post_attention_layernorm", range(R))
            replicated(one(layer, "router"), pre + "router", range(R))
            gates = sorted(by_layer[layer]["expert_gate"], key=lambda k: wl.tensors[k].expert)
            ups = sorted(by_layer[layer]["expert_up"], key=lambda k: wl.tensors[k].expert)
            downs = sorted(by_layer[layer]["expert_down"], key=lambda k: wl.tensors[k].expert)
            n_exp = len(gates)
            assert n_exp == E * R
            Ie, h = seg_shape[gates[0]]
            w13 = [bufs[r].view(pre + "w13", (E, 2 * Ie, h)) for r in range(R)]
            w2 = [bufs[r].view(pre + "w2", (E, h, Ie)) for r in range(R)]
            for e in range(n_exp):
                r, slot = e // E, e % E
                slab13 = w13[r] + slot * 2 * Ie * h
                rows(gates[e], r, slab13, (2 * Ie, h), 0, Ie, 0)
                rows(ups[e], r, slab13, (2 * Ie, h), 0, Ie, Ie)
                slab2 = w2[r] + slot * h * Ie
                whole(downs[e], r, slab2, (h, Ie))
    else:
        raise ValueError("unknown receiver kind %r" % rc.kind)

    return Plan(seg_begin, seg_shape, ops, [b.size for b in bufs], [b.views for b in bufs])
