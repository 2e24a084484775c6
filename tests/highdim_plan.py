"""A transfer plan whose segments have one to four dimensions, written out
both as the oracle's Plan and as the C-ABI structs (test helper; the model
workloads only have vectors and matrices).  Replication, splits along every
dimension, a sub-box placed inside a larger receiver view, unit dimensions.
"""
from oracle import plan as oplan
from paper_2608_00455_amd import binding as B

NRANKS = 3


def _prod(s):
    n = 1
    for x in s:
        n *= x
    return n


def _boxes():
    """Segments and (segment, rank, src_origin, extent, view shape,
    dst_origin) boxes: replication, splits along every dimension, a
    sub-box placed inside a larger view, and unit dimensions."""
    segs = [(100000,), (370, 530), (6, 70, 110), (5, 40, 30, 9), (3, 1, 2, 1)]
    boxes = []
    for r in range(NRANKS):                       # 1-D: replicated
        boxes.append((0, r, (0,), (100000,), (100000,), (0,)))
    rows = [(0, 130), (130, 250), (250, 370)]     # 2-D: row split
    for r, (a, b) in enumerate(rows):
        boxes.append((1, r, (a, 0), (b - a, 530), (b - a, 530), (0, 0)))
    mids = [(0, 30), (30, 50), (50, 70)]          # 3-D: split along dimension 1
    for r, (a, b) in enumerate(mids):
        boxes.append((2, r, (0, a, 0), (6, b - a, 110), (6, b - a, 110), (0, 0, 0)))
    boxes.append((3, 0, (0, 0, 0, 0), (5, 40, 30, 4), (5, 40, 30, 4), (0, 0, 0, 0)))
    boxes.append((3, 1, (0, 0, 0, 4), (5, 40, 30, 5), (5, 40, 30, 5), (0, 0, 0, 0)))
    # rank 2: a sub-box of the 4-D segment placed at an offset in a larger view
    boxes.append((3, 2, (1, 3, 2, 2), (2, 30, 20, 5), (3, 34, 21, 7), (1, 2, 1, 1)))
    boxes.append((4, 1, (0, 0, 0, 0), (3, 1, 2, 1), (3, 1, 2, 1), (0, 0, 0, 0)))
    return segs, boxes


class HighDimSpec:
    """The plan as oracle Plan and as C structs (duck type of PlanSpec)."""

    def __init__(self):
        segs, boxes = _boxes()
        self.seg_shape = segs
        self.seg_begin = []
        pos = 0
        for s in segs:
            self.seg_begin.append(pos)
            pos += _prod(s)
        self.numel = pos
        self.nranks = NRANKS
        size = [0] * NRANKS
        self.boxes = []
        views = [[] for _ in range(NRANKS)]
        for seg, r, a_s, e, view, a_r in boxes:
            base = size[r]
            size[r] += _prod(view)
            views[r].append(("view%d" % len(self.boxes), base, view))
            self.boxes.append((seg, r, base, a_s, e, a_r, view))
        self.rank_numel = size
        self.oracle_plan = oplan.Plan(
            self.seg_begin, [tuple(s) for s in segs],
            [oplan.Op(seg, r, base, tuple(a_s), tuple(e), tuple(a_r), tuple(view))
             for seg, r, base, a_s, e, a_r, view in self.boxes],
            size, views)

    def c_segments(self):
        out = []
        for begin, shape in zip(self.seg_begin, self.seg_shape):
            sg = B.dte_segment()
            sg.flat_begin = begin
            sg.ndim = len(shape)
            for d in range(B.DTE_MAX_DIMS):
                sg.shape[d] = shape[d] if d < len(shape) else 1
            out.append(sg)
        return out

    def c_ops(self):
        out = []
        for seg, r, base, a_s, e, a_r, view in self.boxes:
            o = B.dte_op()
            o.segment, o.rank, o.dst_base = seg, r, base
            for d in range(B.DTE_MAX_DIMS):
                used = d < len(e)
                o.src_origin[d] = a_s[d] if used else 0
                o.extent[d] = e[d] if used else 1
                o.dst_origin[d] = a_r[d] if used else 0
                o.dst_shape[d] = view[d] if used else 1
            out.append(o)
        return out
