"""Oracle diagnostics of every workload (test infrastructure only).

Writes tests/golden/diagnostics.json: per workload the element count, the
changed count |I|, the number of elements whose reconstructed BF16 pattern
differs from the true previous one (b(theta_hat) != b(theta_{t-1})), the
binary32 reconstruction mismatches, the true change count and the
apply-vs-true-previous difference.  Calls only the oracle and the shared
input generator.

    python -m oracle.diagnostics [out.json]
"""
import json
import os
import sys
import time

import synth
from synth import workloads as W

from . import run


def workloads():
    yield W.tiny_block()
    yield W.qwen3_8b(4)
    yield W.qwen3_30b_a3b_share(synth.word)
    for lr in W.SWEEP_LR:
        yield W.qwen3_8b_layers_sweep(lr)


def main(path=None):
    path = path or os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                                "tests", "golden", "diagnostics.json")
    out = {"generator": "oracle/diagnostics.py", "host": run.host_description(), "workloads": {}}
    for wl in workloads():
        t = time.time()
        res = run.extract(wl)
        d = res.diag
        out["workloads"][wl.name] = {
            "elements": d.n, "lr": wl.hp.lr, "seed": wl.seed, "changed": d.changed,
            "bf16_recon_mismatch": d.bf16_recon_mismatch,
            "fp32_recon_mismatch": d.fp32_recon_mismatch,
            "true_changed": d.true_changed, "apply_vs_prev_diff": d.apply_vs_prev_diff,
        }
        print("%s: %s (%.1f s)" % (wl.name, out["workloads"][wl.name], time.time() - t),
              flush=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    return out


if __name__ == "__main__":
    main(sys.argv[1] if len(sys.argv) > 1 else None)
