"""Seeded input generator: Philox4x32-10 known answers and draw properties."""
import numpy as np
import pytest

import synth
from synth import workloads as W

# Known-answer vectors published with the Random123 reference implementation
# of Philox4x32-10 (Salmon et al., SC 2011): (counter, key) -> output.
KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,want", KAT)
def test_philox_known_answers(ctr, key, want):
    assert synth.philox_block(ctr, key) == want


def test_draw_moments_and_bounds():
    n = 1 << 20
    for kind, sigma in W.SIGMA.items():
        x = synth.draw_cpu(n, 12345, 7, kind).astype(np.float64)
        bound = 2 * np.sqrt(3.0) * sigma
        assert np.all(np.abs(x) <= bound * (1 + 1e-6))
        if W.ABSVAL[kind]:
            assert np.all(x >= 0)
            # E|X| of the standardised Irwin-Hall(4) variate: 0.80829 (integral of
            # |s - 2| against the piecewise-cubic Irwin-Hall(4) density)
            assert abs(x.mean() / sigma - 0.80829) < 0.005
        else:
            assert abs(x.mean()) < 0.01 * sigma
            assert abs(x.std() / sigma - 1.0) < 0.01


def test_draw_window_consistency_and_determinism():
    full = synth.draw_cpu(100_000, 99, 3, W.KIND_P_PREV)
    part = synth.draw_cpu(1000, 99, 3, W.KIND_P_PREV, index_base=54_321)
    assert np.array_equal(full[54_321:55_321].view(np.uint32), part.view(np.uint32))
    again = synth.draw_cpu(100_000, 99, 3, W.KIND_P_PREV, threads=4)
    assert np.array_equal(full.view(np.uint32), again.view(np.uint32))
    other = synth.draw_cpu(100_000, 99, 4, W.KIND_P_PREV)
    assert np.count_nonzero(full == other) < 10


def test_workload_sizes():
    assert W.tiny_block().numel == 11_274_240
    assert W.qwen3_8b().numel == 8_190_735_360
    moe = W.qwen3_30b_a3b_share(synth.word)
    assert moe.numel == 7_477_447_680
    assert len(moe.tensors) == 4716
    assert W.qwen3_8b_layers_sweep(1e-6).numel == 771_785_728
    # 96 of the 128 experts of every layer are untouched
    for layer in range(12):
        roles = [t for t in moe.tensors if t.layer == layer and t.role == "expert_up"]
        assert sum(not t.touched for t in roles) == 96


def test_2d_fill_equals_slices_of_the_canonical_draw():
    rows, cols = 37, 53
    full = synth.draw_cpu(rows * cols, 99, 5, 1).reshape(rows, cols)
    out = np.full((40, 30), np.float32(-7.0))
    # a 9 x 11 block of the canonical tensor at (12, 20) written into rows
    # 3.. of a wider buffer (row stride 30) at column 4
    synth.fill_cpu_2d(out[3:12, 4:15], 99, 5, 1, 12, 20, cols)
    assert np.array_equal(out[3:12, 4:15].view(np.uint32), full[12:21, 20:31].view(np.uint32))
    untouched = np.ones(out.shape, bool)
    untouched[3:12, 4:15] = False
    assert np.all(out[untouched] == np.float32(-7.0))
