"""Dense receiver route for pinning the transfer plan and remap.

Builds every receiver rank's flat buffer from canonical tensors with torch
cat / chunk / stack, written independently of any plan code: if a plan maps
canonical flat offsets to receiver coordinates correctly, remapping *all*
offsets (tags = arange(N)) reproduces these buffers exactly.  The layouts
are the receiver conventions of the workloads (see synth.workloads.Receiver):
dense TP: qkv_proj = [q_r; k_r; v_r], gate_up_proj = [gate_r; up_r],
o_proj / down_proj column splits, embed / lm_head vocab-row splits, norms
replicated; MoE: experts e // E on rank, w13 = stack([gate_e; up_e]),
w2 = stack(down_e), attention TP on shard r % A, router and norms replicated.
"""
import torch


def _views(wl, tags):
    by, pos = {}, 0
    for t in wl.tensors:
        by[(t.layer, t.role, t.expert)] = tags[pos:pos + t.numel].view(*t.shape)
        pos += t.numel
    layers = sorted({t.layer for t in wl.tensors if t.layer is not None})
    return by, layers


def _attention(by, L, P, a):
    g = lambda role: by.get((L, role, None))  # noqa: E731
    parts = [torch.cat([g("q").chunk(P, 0)[a], g("k").chunk(P, 0)[a], g("v").chunk(P, 0)[a]], 0)]
    if g("q_norm") is not None:
        parts += [g("q_norm"), g("k_norm")]
    parts.append(g("o").chunk(P, 1)[a])
    return parts


def dense_receivers(wl, tags):
    by, layers = _views(wl, tags)
    rc = wl.receiver
    out = []
    if rc.kind == "tp":
        P = rc.tp
        for r in range(P):
            parts = []
            if (None, "embed", None) in by:
                parts.append(by[(None, "embed", None)].chunk(P, 0)[r])
            for L in layers:
                g = lambda role: by[(L, role, None)]  # noqa: E731
                parts.append(g("in_norm"))
                parts += _attention(by, L, P, r)
                parts.append(g("post_norm"))
                parts.append(torch.cat([g("gate").chunk(P, 0)[r], g("up").chunk(P, 0)[r]], 0))
                parts.append(g("down").chunk(P, 1)[r])
            if (None, "final_norm", None) in by:
                parts.append(by[(None, "final_norm", None)])
            if (None, "lm_head", None) in by:
                parts.append(by[(None, "lm_head", None)].chunk(P, 0)[r])
            out.append(torch.cat([p.reshape(-1) for p in parts]))
    else:
        R, A, E = rc.ranks, rc.attn_tp, rc.experts_per_rank
        for r in range(R):
            parts = []
            for L in layers:
                g = lambda role, e=None: by[(L, role, e)]  # noqa: E731
                parts.append(g("in_norm"))
                parts += _attention(by, L, A, r % A)
                parts.append(g("post_norm"))
                parts.append(g("router"))
                mine = range(r * E, (r + 1) * E)
                parts.append(torch.stack([torch.cat([g("expert_gate", e), g("expert_up", e)], 0)
                                          for e in mine]))
                parts.append(torch.stack([g("expert_down", e) for e in mine]))
            out.append(torch.cat([p.reshape(-1) for p in parts]))
    return out
