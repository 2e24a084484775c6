"""Oracle's Megatron-Core sender layout and converter (test infrastructure only).

The trainer holds optimizer-native MCore tensors (appendix B): the fused
GQA projection W_QKV^MCore built per eq. mcore_fused_qkv, stored per
tensor-parallel rank as the row range R_r of eq. mcore_tp_shard.  The
paper's converter C (sec. 4.2.1, eq. aligned_conversion) gathers the TP
pieces of one converter unit and unpacks them into the canonical tensors
(eq. canonical_qkv_unpacking, eq. qkv_converter); detection then compares
BF16 patterns in that canonical space (eq. canonical_delta_detection).

Readings (the paper gives only the fused-QKV example and says the same
principle covers the other fused or sharded parameters):
  linear_fc1 on rank r is [gate_r; up_r] (rows of each projection split
  evenly), so the gathered fc1 is concat_r [gate_r; up_r];
  linear_proj and linear_fc2 are split along their input columns;
  embedding and output layer along vocabulary rows; layernorms are whole
  on every rank.
  Flat order of rank r's shard: embedding, per layer [input layernorm,
  linear_qkv, q_layernorm, k_layernorm, linear_proj, pre-MLP layernorm,
  linear_fc1, linear_fc2], final layernorm, output layer.
  Each trainer rank detects and sends the canonical elements it holds.

The arithmetic is that of core (inversion in MCore space, sec. 4.1; BF16
detection after conversion, sec. 4.2.1); this module only moves elements.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Tuple

import numpy as np

from . import core, run


# -- eq. mcore_fused_qkv / eq. canonical_qkv_unpacking -----------------------
def fuse_qkv(Wq: np.ndarray, Wk: np.ndarray, Wv: np.ndarray, hq: int, hkv: int,
             dh: int) -> np.ndarray:
    """W_QKV^MCore: for j = 0..hkv-1 the row blocks Q_jg..Q_(j+1)g-1, K_j, V_j."""
    g = hq // hkv
    blocks = []
    for j in range(hkv):
        for i in range(j * g, (j + 1) * g):
            blocks.append(Wq[i * dh:(i + 1) * dh])
        blocks.append(Wk[j * dh:(j + 1) * dh])
        blocks.append(Wv[j * dh:(j + 1) * dh])
    return np.concatenate(blocks, axis=0)


def unfuse_qkv(W: np.ndarray, hq: int, hkv: int, dh: int):
    """The converter of eq. qkv_converter: (W_Q, W_K, W_V) from W_QKV^MCore."""
    g = hq // hkv
    cols = W.shape[1]
    groups = W.reshape(hkv, (g + 2) * dh, cols)
    Wq = groups[:, :g * dh, :].reshape(hq * dh, cols)
    Wk = groups[:, g * dh:(g + 1) * dh, :].reshape(hkv * dh, cols)
    Wv = groups[:, (g + 1) * dh:, :].reshape(hkv * dh, cols)
    return Wq, Wk, Wv


# -- eq. mcore_tp_shard and its gather ---------------------------------------
def tp_shard(W: np.ndarray, P: int, r: int, axis: int) -> np.ndarray:
    n = W.shape[axis]
    assert n % P == 0, "dimension %d does not split into %d ranks" % (n, P)
    w = n // P
    return np.take(W, np.arange(r * w, (r + 1) * w), axis=axis)


def tp_gather(shards: List[np.ndarray], axis: int) -> np.ndarray:
    return np.concatenate(shards, axis=axis)


@dataclass
class Unit:
    """One converter unit: an MCore parameter and the canonical tensors that
    its conversion produces together."""
    name: str
    tensors: Tuple[int, ...]                  # canonical ordinals
    axis: int                                 # TP split axis; -1: whole on every rank
    pack: Callable                            # canonical arrays -> full MCore tensor
    unpack: Callable                          # full MCore tensor -> canonical arrays


def units(wl) -> List[Unit]:
    """The converter units of the dense model in rank-shard order."""
    d = wl.dims
    P = wl.sender.tp
    roles: Dict[Tuple, int] = {(t.layer, t.role): k for k, t in enumerate(wl.tensors)}
    ident = (lambda a: a[0], lambda W: (W,))
    out: List[Unit] = []

    def single(name, k, axis):
        if k is not None:
            out.append(Unit(name, (k,), axis, *ident))

    single("embedding.word_embeddings.weight", roles.get((None, "embed")), 0)
    layers = sorted({t.layer for t in wl.tensors if t.layer is not None})
    for L in layers:
        pre = "decoder.layers.%d." % L
        single(pre + "self_attention.linear_qkv.layer_norm_weight", roles[(L, "in_norm")], -1)
        out.append(Unit(pre + "self_attention.linear_qkv.weight",
                        (roles[(L, "q")], roles[(L, "k")], roles[(L, "v")]), 0,
                        lambda a: fuse_qkv(a[0], a[1], a[2], d.heads_q, d.heads_kv, d.head_dim),
                        lambda W: unfuse_qkv(W, d.heads_q, d.heads_kv, d.head_dim)))
        single(pre + "self_attention.q_layernorm.weight", roles.get((L, "q_norm")), -1)
        single(pre + "self_attention.k_layernorm.weight", roles.get((L, "k_norm")), -1)
        single(pre + "self_attention.linear_proj.weight", roles[(L, "o")], 1)
        single(pre + "mlp.linear_fc1.layer_norm_weight", roles[(L, "post_norm")], -1)

        def pack_fc1(a):
            gate, up = a
            return tp_gather([np.concatenate([tp_shard(gate, P, r, 0), tp_shard(up, P, r, 0)])
                              for r in range(P)], 0)

        def unpack_fc1(W):
            per_rank = [tp_shard(W, P, r, 0) for r in range(P)]
            half = W.shape[0] // (2 * P)
            return (tp_gather([x[:half] for x in per_rank], 0),
                    tp_gather([x[half:] for x in per_rank], 0))

        out.append(Unit(pre + "mlp.linear_fc1.weight", (roles[(L, "gate")], roles[(L, "up")]),
                        0, pack_fc1, unpack_fc1))
        single(pre + "mlp.linear_fc2.weight", roles[(L, "down")], 1)
    single("decoder.final_layernorm.weight", roles.get((None, "final_norm")), -1)
    single("output_layer.weight", roles.get((None, "lm_head")), 0)
    return out


def local(unit: Unit, full: np.ndarray, P: int, r: int) -> np.ndarray:
    """Rank r's piece of the full MCore tensor of a unit."""
    return full if unit.axis < 0 else tp_shard(full, P, r, unit.axis)


def canonical_index(wl) -> np.ndarray:
    """For every element of the sender rank's flat shard, the flat offset of
    the same element in the canonical trainer shard (the canonical tensors
    back to back in parameter order).  Built by running the packing and
    sharding on arrays of canonical offsets."""
    begins = wl.flat_begins()
    P, r = wl.sender.tp, wl.sender.rank
    parts = []
    for u in units(wl):
        arrs = [np.arange(begins[k], begins[k] + wl.tensors[k].numel, dtype=np.int64)
                .reshape(wl.tensors[k].shape) for k in u.tensors]
        parts.append(local(u, u.pack(arrs), P, r).reshape(-1))
    return np.concatenate(parts) if parts else np.zeros(0, np.int64)


@dataclass
class Result:
    idx: np.ndarray        # canonical flat offsets, ascending
    val: np.ndarray        # target BF16 patterns


def extract(wl, hp=None, threads: int = 0) -> Result:
    """Detection for the sender rank, in the paper's order, one converter
    unit at a time: the unit's MCore tensors on every TP rank (the seeded
    canonical state packed per eq. mcore_fused_qkv and sharded per
    eq. mcore_tp_shard), the inversion on each rank's optimizer-native
    shard (sec. 4.1), gather and conversion of both versions
    (eq. aligned_conversion), BF16 comparison per canonical tensor
    (eq. canonical_delta_detection); kept are the changes to elements that
    the sender rank holds."""
    scs = run.scalars(wl, hp)
    threads = threads or run.cpu_threads()
    begins = wl.flat_begins()
    P, r = wl.sender.tp, wl.sender.rank
    idx_parts, val_parts = [], []
    for u in units(wl):
        sc = scs[u.tensors[0]]                # the tensors of a unit share a group
        p_c, m_c, v_c = [], [], []
        for k in u.tensors:
            t = wl.tensors[k]
            _, p, m, v = run.state(wl, k, 0, t.numel, sc, threads)
            p_c.append(p.reshape(t.shape))
            m_c.append(m.reshape(t.shape))
            v_c.append(v.reshape(t.shape))
        p_full, m_full, v_full = u.pack(p_c), u.pack(m_c), u.pack(v_c)
        ranks = range(P) if u.axis >= 0 else [0]
        ph_local = []
        for q in ranks:
            pl = local(u, p_full, P, q)
            ph = core.invert(pl.reshape(-1), local(u, m_full, P, q).reshape(-1),
                             local(u, v_full, P, q).reshape(-1), sc)
            ph_local.append(ph.reshape(pl.shape))
        ph_full = tp_gather(ph_local, u.axis) if u.axis >= 0 else ph_local[0]
        held = local(u, u.pack([np.arange(begins[k], begins[k] + wl.tensors[k].numel,
                                          dtype=np.int64).reshape(wl.tensors[k].shape)
                                for k in u.tensors]), P, r).reshape(-1)
        for j, (old, new) in enumerate(zip(u.unpack(ph_full), u.unpack(p_full))):
            b = begins[u.tensors[j]]
            mine = np.zeros(old.size, bool)
            mine[held[(held >= b) & (held < b + old.size)] - b] = True
            b_old = core.bf16(np.ascontiguousarray(old).reshape(-1))
            b_new = core.bf16(np.ascontiguousarray(new).reshape(-1))
            changed = np.flatnonzero((b_new != b_old) & mine)
            idx_parts.append(changed.astype(np.int64) + np.int64(b))
            val_parts.append(b_new[changed])
    idx = np.concatenate(idx_parts) if idx_parts else np.zeros(0, np.int64)
    val = np.concatenate(val_parts) if val_parts else np.zeros(0, np.uint16)
    order = np.argsort(idx, kind="stable")
    return Result(idx[order], val[order])
