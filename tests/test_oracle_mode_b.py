"""The reconstruction diagnostics with the step taken by torch.optim.AdamW
(oracle/mode_b.py): the driver's counts equal element-by-element counts of
the independent evaluator of tests/test_oracle_diagnostics.py on the same
torch-stepped states, and they differ from the oracle-stepped ones (the
two trainers round differently)."""
import numpy as np
import torch

import synth
from oracle import mode_b
from synth import workloads as W
from test_oracle_diagnostics import Evaluator, as_dict, expected_counts

N = 1200   # elements of each tensor of the sample


def small_windows(wl, total):
    return [(k, min(N, t.numel)) for k, t in enumerate(wl.tensors)]


def torch_step(p_prev, m_prev, v_prev, g, hp):
    param = torch.nn.Parameter(torch.from_numpy(p_prev.copy()))
    opt = torch.optim.AdamW([param], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay, foreach=False, fused=False)
    param.grad = torch.from_numpy(g.copy())
    opt.state[param] = {"step": torch.tensor(float(hp.step - 1)),
                        "exp_avg": torch.from_numpy(m_prev.copy()),
                        "exp_avg_sq": torch.from_numpy(v_prev.copy())}
    with torch.no_grad():
        opt.step()
    return (param.detach().numpy(), opt.state[param]["exp_avg"].numpy(),
            opt.state[param]["exp_avg_sq"].numpy())


def test_torch_stepped_counts_equal_elementwise_counts(monkeypatch):
    wl = W.scaled_dense(layers=1, tp=2, lr=1e-4)
    hp = wl.hp
    monkeypatch.setattr(mode_b, "windows_of", small_windows)
    got = as_dict(mode_b.diagnostics(wl, hp, 0, "torch"))
    ev = Evaluator(hp)
    want = dict(n=0, changed=0, fp32_recon_mismatch=0, bf16_recon_mismatch=0, true_changed=0,
                apply_vs_prev_diff=0)
    differ = 0
    for k, n in small_windows(wl, 0):
        t = wl.tensors[k]
        draws = [synth.draw_cpu(n, wl.seed, k, kind) if (t.touched or kind == W.KIND_P_PREV)
                 else np.zeros(n, np.float32)
                 for kind in (W.KIND_P_PREV, W.KIND_M_PREV, W.KIND_V_PREV, W.KIND_GRAD)]
        p, m, v = torch_step(*draws, hp)
        for key, x in expected_counts(draws[0], p, m, v, ev).items():
            want[key] += x
        ours = np.array([ev.forward(*(float(d[i]) for d in draws))[0] for i in range(n)],
                        np.float32)
        differ += int(np.count_nonzero(p.view(np.uint32) != ours.view(np.uint32)))
    assert differ > 0                          # torch rounds the step differently
    assert got == want
    assert want["fp32_recon_mismatch"] > 0 and want["changed"] > 0
    # the oracle-stepped state of the same sample reconstructs differently
    assert as_dict(mode_b.diagnostics(wl, hp, 0, "oracle")) != got
