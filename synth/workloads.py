"""Synthetic workloads: tensor lists, seeds, step hyperparameters and
receiver-layout descriptors.

Shared by the CPU oracle and the GPU path.  This module describes *what*
the inputs are (shapes, order, seeds, value scales) and holds none of the
method's arithmetic: neither the AdamW step, nor the BF16 rounding, nor the
transfer-plan construction lives here.

Shapes follow the Qwen3 family in Hugging Face parameter order (the
canonical space of the paper's converter-aligned detection, sec. 4.2.1;
canonical Q/K/V shapes are eq. canonical_qkv_shapes of appendix B).
Value scales: p_prev sigma 0.02, m_prev sigma 1e-4, v_prev = |sigma 1e-6|,
gradient sigma 1e-3, drawn per element by the seeded generator of
synth/csrc/philox.h.  The paper's evaluation (sec. 5.1) uses
training-generated RL states of Qwen3-8B and Qwen3-30B-A3B; these seeded
states of the same shapes stand in for them.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

# Draw kinds (third Philox counter word).
KIND_P_PREV, KIND_M_PREV, KIND_V_PREV, KIND_GRAD = 0, 1, 2, 3
SIGMA = {KIND_P_PREV: 0.02, KIND_M_PREV: 1e-4, KIND_V_PREV: 1e-6, KIND_GRAD: 1e-3}
ABSVAL = {KIND_P_PREV: 0, KIND_M_PREV: 0, KIND_V_PREV: 1, KIND_GRAD: 0}

# Tensor ordinal used for the per-layer expert-selection draws (config of
# the MoE workload): far above any real tensor ordinal.
EXPERT_PICK_TENSOR = 0x7FFF0000
EXPERT_PICK_KIND = 0xE


@dataclass(frozen=True)
class Tensor:
    """One canonical (Hugging Face) parameter of the trainer shard."""
    name: str
    shape: Tuple[int, ...]
    role: str                 # embed, q, k, v, o, q_norm, k_norm, gate, up, down,
                              # in_norm, post_norm, final_norm, lm_head, router,
                              # expert_gate, expert_up, expert_down
    layer: Optional[int] = None
    expert: Optional[int] = None
    touched: bool = True      # False: zero moments and gradient (untouched expert)

    @property
    def numel(self) -> int:
        n = 1
        for s in self.shape:
            n *= s
        return n


ORDER_FOLDED, ORDER_LITERAL = 0, 1


@dataclass(frozen=True)
class StepHP:
    """Hyperparameters of the one AdamW step (one parameter group), and the
    binary32 operation order of the step and its inverse (ORDER_FOLDED:
    bias corrections folded into two scalars; ORDER_LITERAL: the inverse's
    printed expression with its four divisions)."""
    lr: float
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    step: int = 100
    order: int = ORDER_FOLDED


@dataclass(frozen=True)
class Receiver:
    """Inference-side layout descriptor.

    kind 'tp': dense model, tensor parallel degree `tp` (fused qkv and
    gate_up column splits, o/down row splits, vocab-row splits of embed and
    lm_head, norms replicated).
    kind 'moe_ep': MoE layers, `ranks` receivers; attention TP degree
    `attn_tp` replicated over ranks // attn_tp groups; experts split
    `experts_per_rank` per rank; router and norms replicated on all ranks.
    """
    kind: str
    tp: int = 1
    ranks: int = 1
    attn_tp: int = 1
    experts_per_rank: int = 0

    @property
    def nranks(self) -> int:
        return self.tp if self.kind == 'tp' else self.ranks


@dataclass(frozen=True)
class Sender:
    """Trainer-side layout of the flat shard.

    kind 'canonical': the canonical tensors back to back in parameter order.
    kind 'mcore': the optimizer-native Megatron-Core tensors of tensor
    parallel rank `rank` of `tp` (per layer: input layernorm, fused
    linear_qkv rows of the rank, q/k layernorms, linear_proj input columns
    of the rank, pre-MLP layernorm, fused linear_fc1 [gate; up] rows of the
    rank, linear_fc2 input columns of the rank; before the layers the
    embedding's vocabulary rows of the rank, after them the final layernorm
    and the output layer's vocabulary rows of the rank).  Values are drawn per
    canonical element, so the same model state is seen in either layout.
    """
    kind: str = "canonical"
    tp: int = 1
    rank: int = 0


@dataclass(frozen=True)
class ModelDims:
    hidden: int
    heads_q: int
    heads_kv: int
    head_dim: int
    intermediate: int = 0
    vocab: int = 0
    experts: int = 0
    expert_intermediate: int = 0
    qk_norm: bool = True


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    seed: int
    dims: ModelDims
    tensors: Tuple[Tensor, ...]
    hp: StepHP
    receiver: Receiver
    sweep_lr: Tuple[float, ...] = field(default_factory=tuple)
    sender: Sender = field(default_factory=Sender)
    # Two parameter groups: the 1-D tensors (norms) without weight decay,
    # the rest with hp.weight_decay.
    no_decay_norms: bool = False

    def group_hp(self, k: int, hp: Optional[StepHP] = None) -> StepHP:
        """Step hyperparameters of the parameter group holding tensor k."""
        hp = hp or self.hp
        if self.no_decay_norms and len(self.tensors[k].shape) == 1:
            return replace(hp, weight_decay=0.0)
        return hp

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)

    def flat_begins(self):
        out, pos = [], 0
        for t in self.tensors:
            out.append(pos)
            pos += t.numel
        return out


def _dense_layer(d: ModelDims, layer: int, with_qk_norm: bool):
    h, qd, kd = d.hidden, d.heads_q * d.head_dim, d.heads_kv * d.head_dim
    pre = f"model.layers.{layer}."
    ts = [
        Tensor(pre + "self_attn.q_proj.weight", (qd, h), "q", layer),
        Tensor(pre + "self_attn.k_proj.weight", (kd, h), "k", layer),
        Tensor(pre + "self_attn.v_proj.weight", (kd, h), "v", layer),
        Tensor(pre + "self_attn.o_proj.weight", (h, qd), "o", layer),
    ]
    if with_qk_norm:
        ts += [Tensor(pre + "self_attn.q_norm.weight", (d.head_dim,), "q_norm", layer),
               Tensor(pre + "self_attn.k_norm.weight", (d.head_dim,), "k_norm", layer)]
    ts += [
        Tensor(pre + "mlp.gate_proj.weight", (d.intermediate, h), "gate", layer),
        Tensor(pre + "mlp.up_proj.weight", (d.intermediate, h), "up", layer),
        Tensor(pre + "mlp.down_proj.weight", (h, d.intermediate), "down", layer),
        Tensor(pre + "input_layernorm.weight", (h,), "in_norm", layer),
        Tensor(pre + "post_attention_layernorm.weight", (h,), "post_norm", layer),
    ]
    return ts


def untouched_experts(seed: int, layer: int, n_experts: int, n_untouched: int, word_fn):
    """Seeded choice of the experts whose moments and gradient are zero.

    Each expert e of the layer gets the first Philox word at
    (seed, EXPERT_PICK_TENSOR, EXPERT_PICK_KIND, layer * 2^16 + e); the
    n_untouched experts with the smallest (word, e) are untouched.
    `word_fn(seed, tensor, kind, index)` is the generator's word accessor.
    """
    keyed = sorted((word_fn(seed, EXPERT_PICK_TENSOR, EXPERT_PICK_KIND, layer * 65536 + e), e)
                   for e in range(n_experts))
    return frozenset(e for _, e in keyed[:n_untouched])


def _moe_layer(d: ModelDims, layer: int, untouched: frozenset):
    h, qd, kd = d.hidden, d.heads_q * d.head_dim, d.heads_kv * d.head_dim
    pre = f"model.layers.{layer}."
    ts = [
        Tensor(pre + "self_attn.q_proj.weight", (qd, h), "q", layer),
        Tensor(pre + "self_attn.k_proj.weight", (kd, h), "k", layer),
        Tensor(pre + "self_attn.v_proj.weight", (kd, h), "v", layer),
        Tensor(pre + "self_attn.o_proj.weight", (h, qd), "o", layer),
        Tensor(pre + "self_attn.q_norm.weight", (d.head_dim,), "q_norm", layer),
        Tensor(pre + "self_attn.k_norm.weight", (d.head_dim,), "k_norm", layer),
        Tensor(pre + "mlp.gate.weight", (d.experts, h), "router", layer),
    ]
    for e in range(d.experts):
        t = e not in untouched
        ep = pre + f"mlp.experts.{e}."
        ts += [
            Tensor(ep + "gate_proj.weight", (d.expert_intermediate, h), "expert_gate", layer, e, t),
            Tensor(ep + "up_proj.weight", (d.expert_intermediate, h), "expert_up", layer, e, t),
            Tensor(ep + "down_proj.weight", (h, d.expert_intermediate), "expert_down", layer, e, t),
        ]
    ts += [
        Tensor(pre + "input_layernorm.weight", (h,), "in_norm", layer),
        Tensor(pre + "post_attention_layernorm.weight", (h,), "post_norm", layer),
    ]
    return ts


SEED_BASE = 26080455 * 10

QWEN3_8B = ModelDims(hidden=4096, heads_q=32, heads_kv=8, head_dim=128,
                     intermediate=12288, vocab=151936)
QWEN3_30B_A3B = ModelDims(hidden=2048, heads_q=32, heads_kv=4, head_dim=128,
                          vocab=151936, experts=128, expert_intermediate=768)
TINY_BLOCK = ModelDims(hidden=1024, heads_q=8, heads_kv=2, head_dim=128,
                       intermediate=2816, qk_norm=False)


def tiny_block() -> Workload:
    """One dense block, 11,274,240 elements, receiver TP=2."""
    d = TINY_BLOCK
    return Workload("tiny_block_tp2",
                    "one dense block (hidden 1024, 8/2 heads x 128, MLP 2816), TP=2",
                    SEED_BASE + 1, d, tuple(_dense_layer(d, 0, False)), StepHP(lr=1e-6),
                    Receiver("tp", tp=2))


def _qwen3_8b_tensors(layers: int, with_embed: bool):
    d = QWEN3_8B
    ts = []
    if with_embed:
        ts.append(Tensor("model.embed_tokens.weight", (d.vocab, d.hidden), "embed"))
    for layer in range(layers):
        ts += _dense_layer(d, layer, True)
    if with_embed:
        ts.append(Tensor("model.norm.weight", (d.hidden,), "final_norm"))
        ts.append(Tensor("lm_head.weight", (d.vocab, d.hidden), "lm_head"))
    return tuple(ts)


def qwen3_8b(tp: int = 4) -> Workload:
    """Full Qwen3-8B state, 8,190,735,360 elements, receiver TP=tp."""
    name = "qwen3_8b_tp%d" % tp
    return Workload(name, "Qwen3-8B full state (36 layers, untied embed/lm_head), TP=%d" % tp,
                    SEED_BASE + 2, QWEN3_8B, _qwen3_8b_tensors(36, True), StepHP(lr=1e-6),
                    Receiver("tp", tp=tp))


def qwen3_30b_a3b_share(word_fn, layers: int = 12) -> Workload:
    """First `layers` of the 48 Qwen3-30B-A3B layers; 75% of experts untouched."""
    d = QWEN3_30B_A3B
    seed = SEED_BASE + 3
    ts = []
    for layer in range(layers):
        unt = untouched_experts(seed, layer, d.experts, d.experts * 3 // 4, word_fn)
        ts += _moe_layer(d, layer, unt)
    return Workload("qwen3_30b_a3b_%dl_ep8" % layers,
                    "Qwen3-30B-A3B first %d layers, 128 experts (96 untouched per layer), "
                    "8 receivers: EP 16 experts/rank, attention TP=2 x 4 replicas" % layers,
                    seed, d, tuple(ts), StepHP(lr=1e-6),
                    Receiver("moe_ep", ranks=8, attn_tp=2, experts_per_rank=16))


SWEEP_LR = (1e-7, 1e-6, 1e-5, 1e-4)


def qwen3_8b_layers_sweep(lr: float, layers: int = 4) -> Workload:
    """`layers` Qwen3-8B layers (192,946,432 elements each), receiver TP=4.

    All learning rates of the sweep share one seed, so they invert the same
    pre-step state under different step sizes.
    """
    return Workload("qwen3_8b_%dl_tp4_lr%g" % (layers, lr),
                    "%d Qwen3-8B layers, TP=4, lr=%g" % (layers, lr),
                    SEED_BASE + 4, QWEN3_8B, _qwen3_8b_tensors(layers, False), StepHP(lr=lr),
                    Receiver("tp", tp=4), sweep_lr=SWEEP_LR)


def scaled_dense(layers: int = 2, tp: int = 2, seed: int = SEED_BASE + 11,
                 hidden=256, heads_q=4, heads_kv=2, head_dim=64, intermediate=704,
                 vocab=1000, embed=True, lr=1e-6) -> Workload:
    """Small dense model with every tensor kind of the Qwen3 dense family."""
    d = ModelDims(hidden=hidden, heads_q=heads_q, heads_kv=heads_kv, head_dim=head_dim,
                  intermediate=intermediate, vocab=vocab)
    ts = []
    if embed:
        ts.append(Tensor("model.embed_tokens.weight", (vocab, hidden), "embed"))
    for layer in range(layers):
        ts += _dense_layer(d, layer, True)
    if embed:
        ts.append(Tensor("model.norm.weight", (hidden,), "final_norm"))
        ts.append(Tensor("lm_head.weight", (vocab, hidden), "lm_head"))
    return Workload("dense_small_%dl_tp%d" % (layers, tp), "small dense model, TP=%d" % tp,
                    seed, d, tuple(ts), StepHP(lr=lr), Receiver("tp", tp=tp))


def scaled_moe(word_fn, layers: int = 2, ranks: int = 4, attn_tp: int = 2, experts: int = 8,
               seed: int = SEED_BASE + 13, hidden=128, heads_q=4, heads_kv=2, head_dim=32,
               expert_intermediate=48, lr=1e-6) -> Workload:
    """Small MoE model with the structure of the Qwen3-30B-A3B share."""
    d = ModelDims(hidden=hidden, heads_q=heads_q, heads_kv=heads_kv, head_dim=head_dim,
                  experts=experts, expert_intermediate=expert_intermediate)
    ts = []
    for layer in range(layers):
        unt = untouched_experts(seed, layer, experts, experts * 3 // 4, word_fn)
        ts += _moe_layer(d, layer, unt)
    return Workload("moe_small_%dl_r%d" % (layers, ranks), "small MoE model", seed, d,
                    tuple(ts), StepHP(lr=lr),
                    Receiver("moe_ep", ranks=ranks, attn_tp=attn_tp,
                             experts_per_rank=experts // ranks))


def qwen3_8b_layers_mcore(layers: int = 4, trainer_tp: int = 2, trainer_rank: int = 0,
                          receiver_tp: int = 4, lr: float = 1e-6) -> Workload:
    """`layers` Qwen3-8B layers held as one trainer TP rank's Megatron-Core
    shard; receiver TP=receiver_tp (canonical tensors as qwen3_8b_layers_sweep)."""
    return Workload("qwen3_8b_%dl_mcore_tp%dr%d_to_tp%d" % (layers, trainer_tp, trainer_rank,
                                                           receiver_tp),
                    "%d Qwen3-8B layers, Megatron-Core shard of trainer TP rank %d/%d, "
                    "receiver TP=%d" % (layers, trainer_rank, trainer_tp, receiver_tp),
                    SEED_BASE + 6, QWEN3_8B, _qwen3_8b_tensors(layers, False), StepHP(lr=lr),
                    Receiver("tp", tp=receiver_tp), sender=Sender("mcore", trainer_tp,
                                                                  trainer_rank))


def scaled_mcore(layers: int = 2, trainer_tp: int = 2, trainer_rank: int = 0,
                 receiver_tp: int = 2, seed: int = SEED_BASE + 17, hidden=64, heads_q=8,
                 heads_kv=4, head_dim=16, intermediate=96, vocab=0, lr=1e-5) -> Workload:
    """Small dense model held as a Megatron-Core trainer shard (with
    embedding, final norm and output layer when vocab > 0)."""
    d = ModelDims(hidden=hidden, heads_q=heads_q, heads_kv=heads_kv, head_dim=head_dim,
                  intermediate=intermediate, vocab=vocab)
    ts = []
    if vocab:
        ts.append(Tensor("model.embed_tokens.weight", (vocab, hidden), "embed"))
    for layer in range(layers):
        ts += _dense_layer(d, layer, True)
    if vocab:
        ts.append(Tensor("model.norm.weight", (hidden,), "final_norm"))
        ts.append(Tensor("lm_head.weight", (vocab, hidden), "lm_head"))
    return Workload("dense_small_%dl_mcore_tp%dr%d_to_tp%d" % (layers, trainer_tp, trainer_rank,
                                                              receiver_tp),
                    "small dense model, Megatron-Core shard", seed, d, tuple(ts), StepHP(lr=lr),
                    Receiver("tp", tp=receiver_tp), sender=Sender("mcore", trainer_tp,
                                                                  trainer_rank))


def with_sender_rank(wl: Workload, rank: int) -> Workload:
    """The same workload seen from another trainer TP rank."""
    return replace(wl, sender=Sender(wl.sender.kind, wl.sender.tp, rank))


def canonical_twin(wl: Workload) -> Workload:
    """The same model state with the canonical sender layout."""
    return replace(wl, name=wl.name + "_canonical",
                   description=wl.description + " (canonical layout)", sender=Sender())


def with_norm_group(wl: Workload) -> Workload:
    """The same workload with the norms in a parameter group of their own
    (weight decay 0)."""
    return replace(wl, name=wl.name + "_nd", description=wl.description + ", norms without decay",
                   no_decay_norms=True)
