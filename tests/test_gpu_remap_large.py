"""Remap and apply at a scale where the remap grid is capped (more than
128 blocks per CU of 4096 entries), so a block takes its slice in three or
more 2048-entry groups: 200 M shuffled entries of a 20000 x 16384 matrix
split by rows between two receivers.

The expected buckets have a closed form here (rank r holds the entries of
its rows, offset by r * 10000 * 16384; each value is a fixed hash of its
offset), so they are checked on the device with torch sorts and scatters
rather than with the oracle.
"""
import sys

import pytest
import torch

from paper_2608_00455_amd import binding as B

pytestmark = pytest.mark.gpu

ROWS, COLS = 20000, 16384
HALF = ROWS // 2
M = 200_000_000


def value_of(flat):
    h = (flat * 40503 + 12345) & 0xFFFF
    return torch.where(h >= 32768, h - 65536, h).to(torch.int16)


def plan():
    seg = B.dte_segment()
    seg.flat_begin, seg.ndim = 0, 2
    seg.shape[0], seg.shape[1] = ROWS, COLS
    ops = []
    for r in range(2):
        o = B.dte_op()
        o.segment, o.rank, o.dst_base = 0, r, 0
        o.src_origin[0], o.src_origin[1] = r * HALF, 0
        o.extent[0], o.extent[1] = HALF, COLS
        o.dst_origin[0], o.dst_origin[1] = 0, 0
        o.dst_shape[0], o.dst_shape[1] = HALF, COLS
        ops.append(o)
    return B.dte_plan_create([seg], ops, 2, [HALF * COLS, HALF * COLS])


def test_remap_and_apply_with_capped_grid():
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert M > cus * 128 * 4096, "the grid cap must bind for this test"
    print("case: large remap, %d entries, %d CUs" % (M, cus), flush=True)
    sys.stdout.flush()
    dev = torch.device("cuda")
    g = torch.Generator(device=dev)
    g.manual_seed(26080455)
    idx = torch.randperm(ROWS * COLS, generator=g, device=dev)[:M].contiguous()
    val = value_of(idx)
    count = torch.tensor([M], dtype=torch.int64, device=dev)
    off = [torch.empty(M, dtype=torch.int64, device=dev) for _ in range(2)]
    rval = [torch.empty(M, dtype=torch.int16, device=dev) for _ in range(2)]
    rank_count = torch.zeros(2, dtype=torch.int64, device=dev)
    shards = [torch.zeros(HALF * COLS, dtype=torch.int16, device=dev) for _ in range(2)]
    h = plan()
    try:
        s = torch.cuda.current_stream().cuda_stream
        B.dte_remap(h, idx.data_ptr(), val.data_ptr(), count.data_ptr(), M,
                    [t.data_ptr() for t in off], [t.data_ptr() for t in rval], [M, M],
                    rank_count.data_ptr(), s)
        B.dte_apply(h, [t.data_ptr() for t in shards], [t.data_ptr() for t in off],
                    [t.data_ptr() for t in rval], rank_count.data_ptr(), [M, M], s)
        torch.cuda.synchronize()
    finally:
        B.dte_plan_destroy(h)
    low = idx < HALF * COLS
    want_count = [int(low.sum().item()), M - int(low.sum().item())]
    assert rank_count.cpu().tolist() == want_count
    for r in range(2):
        k = want_count[r]
        mine, order = torch.sort(off[r][:k])
        want = torch.sort(idx[low if r == 0 else ~low] - r * HALF * COLS).values
        assert torch.equal(mine, want), r
        assert torch.equal(rval[r][:k][order], value_of(want + r * HALF * COLS)), r
        expect = torch.zeros_like(shards[r])
        expect[want] = value_of(want + r * HALF * COLS)
        assert torch.equal(shards[r], expect), r


def test_remap_and_apply_on_the_largest_segment():
    """A 65536 x 65535 matrix (4,294,901,760 elements, just under the
    2^32 limit of a segment): segment-local indices near the top of their
    32-bit range, the first and last elements and both sides of the row
    split, 50 M random entries in all."""
    rows, cols = 65536, 65535
    half = rows // 2
    total = rows * cols
    print("case: largest segment, %d elements" % total, flush=True)
    sys.stdout.flush()
    dev = torch.device("cuda")
    g = torch.Generator(device=dev)
    g.manual_seed(26080456)
    edges = torch.tensor([0, 1, cols - 1, half * cols - 1, half * cols, total - cols, total - 2,
                          total - 1], dtype=torch.int64, device=dev)
    rnd = torch.randint(0, total, (50_000_000,), generator=g, device=dev, dtype=torch.int64)
    idx = torch.unique(torch.cat([rnd, edges]))
    idx = idx[torch.randperm(idx.numel(), generator=g, device=dev)].contiguous()
    m = idx.numel()
    val = value_of(idx)
    seg = B.dte_segment()
    seg.flat_begin, seg.ndim = 0, 2
    seg.shape[0], seg.shape[1] = rows, cols
    ops = []
    for r in range(2):
        o = B.dte_op()
        o.segment, o.rank, o.dst_base = 0, r, 0
        o.src_origin[0], o.src_origin[1] = r * half, 0
        o.extent[0], o.extent[1] = half, cols
        o.dst_origin[0], o.dst_origin[1] = 0, 0
        o.dst_shape[0], o.dst_shape[1] = half, cols
        ops.append(o)
    h = B.dte_plan_create([seg], ops, 2, [half * cols, half * cols])
    count = torch.tensor([m], dtype=torch.int64, device=dev)
    off = [torch.empty(m, dtype=torch.int64, device=dev) for _ in range(2)]
    rval = [torch.empty(m, dtype=torch.int16, device=dev) for _ in range(2)]
    rank_count = torch.zeros(2, dtype=torch.int64, device=dev)
    shards = [torch.zeros(half * cols, dtype=torch.int16, device=dev) for _ in range(2)]
    try:
        s = torch.cuda.current_stream().cuda_stream
        B.dte_remap(h, idx.data_ptr(), val.data_ptr(), count.data_ptr(), m,
                    [t.data_ptr() for t in off], [t.data_ptr() for t in rval], [m, m],
                    rank_count.data_ptr(), s)
        B.dte_apply(h, [t.data_ptr() for t in shards], [t.data_ptr() for t in off],
                    [t.data_ptr() for t in rval], rank_count.data_ptr(), [m, m], s)
        torch.cuda.synchronize()
    finally:
        B.dte_plan_destroy(h)
    low = idx < half * cols
    want_count = [int(low.sum().item()), m - int(low.sum().item())]
    assert rank_count.cpu().tolist() == want_count
    for r in range(2):
        k = want_count[r]
        mine, order = torch.sort(off[r][:k])
        want = torch.sort(idx[low if r == 0 else ~low] - r * half * cols).values
        assert torch.equal(mine, want), r
        assert torch.equal(rval[r][:k][order], value_of(want + r * half * cols)), r
        expect = torch.zeros_like(shards[r])
        expect[want] = value_of(want + r * half * cols)
        assert torch.equal(shards[r], expect), r
        del expect
    # the extremes went where they belong
    last = shards[1][half * cols - 1].item()
    assert last == int(value_of(torch.tensor([total - 1]))[0])
