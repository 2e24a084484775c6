"""The Python layer refuses buffers that the library, which takes raw
addresses and element counts, would read or write out of bounds: wrong
dtype, device, layout or length.  Nothing is launched for them."""
import sys

import pytest
import torch

from paper_2608_00455_amd import layouts
from paper_2608_00455_amd.pipeline import DeltaPipeline
from synth import workloads as W

pytestmark = pytest.mark.gpu


def test_pipeline_refuses_unsafe_buffers():
    print("case: pipeline buffer checks", flush=True)
    sys.stdout.flush()
    wl = W.scaled_dense(layers=1, tp=2)
    spec = layouts.build_spec(wl)
    n = wl.numel
    pipe = DeltaPipeline(spec, capacity=1024)
    hp = W.StepHP(lr=1e-5)
    good = [torch.zeros(n, dtype=torch.float32, device="cuda") for _ in range(3)]
    p, m, v = good
    with pytest.raises(ValueError, match="dtype"):
        pipe.extract(p.double(), m, v, hp)
    with pytest.raises(ValueError, match="on cpu"):
        pipe.extract(p, m.cpu(), v, hp)
    with pytest.raises(ValueError, match="contiguous"):
        pipe.extract(p, m, torch.zeros(2 * n, device="cuda")[::2], hp)
    with pytest.raises(ValueError, match="needed"):
        pipe.extract(p, m, v, hp, n=n + 1)
    with pytest.raises(ValueError, match="out_prev"):
        pipe.extract(p, m, v, hp, out_prev=torch.zeros(n - 1, device="cuda"))
    with pytest.raises(ValueError, match="needed"):
        pipe.extract_remap(p[:-1], m[:-1], v[:-1], hp, n=n)
    with pytest.raises(TypeError):
        pipe.extract(p.cpu().numpy(), m, v, hp)
    torch.cuda.synchronize()
    assert int(pipe.cursor.item()) == 0          # nothing ran
    short = [torch.zeros(k, dtype=torch.int16, device="cuda") for k in spec.rank_numel]
    short[-1] = short[-1][:-1]
    with pytest.raises(ValueError, match="shards"):
        DeltaPipeline(spec, capacity=16, shards=short)
    with pytest.raises(ValueError, match="shards"):
        DeltaPipeline(spec, capacity=16, shards=short[:-1])
    # the good buffers still run
    pipe.step(p, m, v, hp)
    torch.cuda.synchronize()
    pipe.close()
