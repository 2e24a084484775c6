"""Reconstruction under another trainer's rounding -- TEST INFRASTRUCTURE
ONLY (prints a table; the product path never imports it).

The oracle's own forward step rounds in the order that its inverse undoes
(sec. 4.1: the inverse is a numerical reconstruction of the previous
weights).  A trainer built on torch.optim.AdamW (single-tensor path)
rounds differently: the decay multiplies the weights first, the first
moment is a linear interpolation, the bias corrections are applied to the
square root and the step size in binary64 scalars.  Here that optimizer
takes the step from the same seeded pre-step state on the CPU, and the
oracle then inverts its output (folded or literal order, sec. 4.1),
detects the BF16 changes (sec. 4.2.1) and counts, element by element, the
same reconstruction diagnostics as the oracle's driver:
  fp32_recon_mismatch  theta_hat != theta_{t-1} as binary32 patterns
  bf16_recon_mismatch  b(theta_hat) != b(theta_{t-1})
  true_changed         b(theta_{t-1}) != b(theta_t)
  apply_vs_prev_diff   b(theta_{t-1}) != b(theta_hat) == b(theta_t)
The detected delta itself is whatever the inverse gives for those inputs;
the GPU path is compared with the oracle on such states like on any other.

    python -m oracle.mode_b [--elements 20000000]
"""
from __future__ import annotations

import argparse
import sys

import numpy as np

from synth import workloads as W

from . import core, run


def torch_adamw_step(p_prev, m_prev, v_prev, g, hp):
    """One torch.optim.AdamW step (foreach and fused off) from step t-1;
    returns the post-step (theta, m, v) as binary32 arrays."""
    import torch
    param = torch.nn.Parameter(torch.from_numpy(np.array(p_prev, np.float32)))
    opt = torch.optim.AdamW([param], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False, fused=False)
    param.grad = torch.from_numpy(np.array(g, np.float32))
    opt.state[param] = {"step": torch.tensor(float(hp.step - 1)),
                        "exp_avg": torch.from_numpy(np.array(m_prev, np.float32)),
                        "exp_avg_sq": torch.from_numpy(np.array(v_prev, np.float32))}
    with torch.no_grad():
        opt.step()
    return (param.detach().numpy().copy(), opt.state[param]["exp_avg"].numpy().copy(),
            opt.state[param]["exp_avg_sq"].numpy().copy())


def windows_of(wl, total):
    """The first elements of every tensor of layer 0 (every tensor when the
    workload has no layer 0 tensors, or fewer elements than asked), in
    proportion to the tensors' sizes, `total` elements in all."""
    ks = [k for k, t in enumerate(wl.tensors) if t.layer == 0] or list(range(len(wl.tensors)))
    size = sum(wl.tensors[k].numel for k in ks)
    if size <= total:
        return [(k, wl.tensors[k].numel) for k in ks]
    return [(k, max(1, round(total * wl.tensors[k].numel / size))) for k in ks]


def diagnostics(wl, hp, total, trainer):
    """Diagnostics over the sample, the state stepped by `trainer` ("oracle"
    or "torch")."""
    sc = core.derive_scalars(hp)
    d = run.Diagnostics()
    for k, n in windows_of(wl, total):
        p_prev, m_prev, v_prev, g = run.draws(wl, k, 0, n)
        if trainer == "torch":
            p, m, v = torch_adamw_step(p_prev, m_prev, v_prev, g, hp)
        else:
            p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)
        idx, _, ph = core.detect(p, m, v, sc)
        d.add(run.count_diagnostics(p_prev, ph, p, int(idx.size)))
    return d


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--elements", type=int, default=20_000_000)
    a = ap.parse_args(argv)
    print("| workload | lr | trainer | inverse order | elements | changed | binary32 mismatches | "
          "BF16 mismatches | true changes | stale after apply |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    cases = [(W.tiny_block(), 1e-6)] + [(W.qwen3_8b_layers_sweep(lr), lr) for lr in W.SWEEP_LR]
    for wl, lr in cases:
        for trainer in ("oracle", "torch"):
            for order, name in ((W.ORDER_FOLDED, "folded"), (W.ORDER_LITERAL, "literal")):
                hp = W.StepHP(lr=lr, order=order, weight_decay=wl.hp.weight_decay,
                              step=wl.hp.step)
                d = diagnostics(wl, hp, a.elements, trainer)
                print("| %s | %g | %s | %s | %d | %d | %d | %d | %d | %d |" % (
                    wl.name, lr, "torch.optim.AdamW" if trainer == "torch" else "oracle step",
                    name, d.n, d.changed, d.fp32_recon_mismatch, d.bf16_recon_mismatch,
                    d.true_changed, d.apply_vs_prev_diff), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
