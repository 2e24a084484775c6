"""Effect of the input recipe on the change fraction and the
reconstruction counts -- TEST INFRASTRUCTURE ONLY (prints a table; the
product path never imports it).

The seeded generator shared by the oracle and the GPU path (synth) draws
each value as a centred Irwin-Hall(4) variate scaled to the standard
deviation sigma: bounded at 2 sqrt(3) sigma, with lighter tails than a
normal draw.  This script runs the oracle (forward AdamW step, inversion,
BF16 detection, reconstruction counts) on the same sample drawn both ways:
  irwin_hall : synth.draw_cpu, as every workload of the repository;
  normal     : numpy.random.Generator(Philox(key=[seed, 4 k + q]))
               .standard_normal, times sigma (absolute value for v), rounded
               to binary32.
Sample: the first elements of every tensor of layer 0 of the Qwen3-8B
workload, in proportion to the tensors' sizes, 2e7 elements in all; the
four learning rates of the sweep.

    python -m oracle.recipe_compare [--elements 20000000]
"""
from __future__ import annotations

import argparse
import sys

import numpy as np

import synth
from synth import workloads as W

from . import core, run

KINDS = (W.KIND_P_PREV, W.KIND_M_PREV, W.KIND_V_PREV, W.KIND_GRAD)


def sample(wl, total):
    ks = [k for k, t in enumerate(wl.tensors) if t.layer == 0]
    layer = sum(wl.tensors[k].numel for k in ks)
    out = [(k, max(1, round(total * wl.tensors[k].numel / layer))) for k in ks]
    return out


def draws(recipe, seed, k, n):
    vals = []
    for q in KINDS:
        if recipe == "irwin_hall":
            x = synth.draw_cpu(n, seed, k, q, 0, threads=synth.default_threads())
        else:
            z = np.random.Generator(np.random.Philox(key=[seed, 4 * k + q])).standard_normal(n)
            x = z * W.SIGMA[q]
            if W.ABSVAL[q]:
                x = np.abs(x)
            x = x.astype(np.float32)
        vals.append(x)
    return vals


def compare(total=20_000_000):
    wl = W.qwen3_8b(4)
    picks = sample(wl, total)
    rows = []
    for recipe in ("irwin_hall", "normal"):
        states = [(k, draws(recipe, wl.seed, k, n)) for k, n in picks]
        tail = sum(int(np.count_nonzero(np.abs(d[0]) > 2 * np.sqrt(3) * 0.02))
                   for _, d in states)
        for lr in W.SWEEP_LR:
            sc = core.derive_scalars(W.StepHP(lr=lr))
            d = run.Diagnostics()
            for k, (p_prev, m_prev, v_prev, g) in states:
                p, m, v = core.adamw_forward(p_prev, m_prev, v_prev, g, sc)
                idx, _, ph = core.detect(p, m, v, sc)
                d.add(run.count_diagnostics(p_prev, ph, p, int(idx.size)))
            rows.append({"recipe": recipe, "lr": lr, "n": d.n, "changed": d.changed,
                         "c": d.changed / d.n, "fp32_recon_mismatch": d.fp32_recon_mismatch,
                         "bf16_recon_mismatch": d.bf16_recon_mismatch,
                         "true_changed": d.true_changed,
                         "apply_vs_prev_diff": d.apply_vs_prev_diff,
                         "p_prev_beyond_2sqrt3_sigma": tail})
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--elements", type=int, default=20_000_000)
    a = ap.parse_args(argv)
    rows = compare(a.elements)
    print("| lr | recipe | elements | c | binary32 mismatches | BF16 mismatches | "
          "true changes | stale after apply | theta_{t-1} beyond 2 sqrt(3) sigma |")
    print("|---|---|---|---|---|---|---|---|---|")
    for r in sorted(rows, key=lambda r: (r["lr"], r["recipe"])):
        print("| %g | %s | %d | %.4f %% | %d | %d | %d | %d | %d |" % (
            r["lr"], r["recipe"], r["n"], 100 * r["c"], r["fp32_recon_mismatch"],
            r["bf16_recon_mismatch"], r["true_changed"], r["apply_vs_prev_diff"],
            r["p_prev_beyond_2sqrt3_sigma"]))
    return 0


if __name__ == "__main__":
    sys.exit(main())
