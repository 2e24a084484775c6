"""Storage-mediated publication (paper sec. 4.4), host side, no GPU.

The stored files are checked by a reader written here from the format's
description (Python struct, the `xxhash` package for XXH64, libzstd through
ctypes), independent of the library's own reader; the payload is the
oracle's delta, and the destination's result (oracle remap and apply of
what was read) is the receiver layout of the new BF16 weights.  Commit
rules: no version without a changed entry, a missing writer part publishes
nothing, several writers may hold entries of one tensor (tensor-parallel
Megatron-Core ranks publish their pieces of it), the version chain is
followed from parents, and corrupted or truncated chunks are rejected.
"""
import ctypes
import json
import os
import struct

import numpy as np
import pytest
import xxhash

from oracle import core as ocore
from oracle import plan as oplan
from oracle import remap as oremap
from oracle import run as orun
from paper_2608_00455_amd import binding as B
from paper_2608_00455_amd import store as S
from synth import workloads as W


def _zstd_decompress(data: bytes, size: int) -> bytes:
    lib = ctypes.CDLL("libzstd.so.1")
    lib.ZSTD_decompress.restype = ctypes.c_size_t
    lib.ZSTD_decompress.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                    ctypes.c_size_t]
    lib.ZSTD_isError.restype = ctypes.c_uint
    lib.ZSTD_isError.argtypes = [ctypes.c_size_t]
    out = ctypes.create_string_buffer(size)
    src = ctypes.create_string_buffer(data, len(data))
    got = lib.ZSTD_decompress(out, size, src, len(data))
    assert not lib.ZSTD_isError(got) and got == size
    return out.raw[:size]


def independent_read(d, version):
    """Parse a committed version from its files alone."""
    man = json.load(open(os.path.join(d, "v%d" % version, "manifest.json")))
    idx, val = [], []
    for c in man["chunks"]:
        raw = open(os.path.join(d, "v%d" % version, c["file"]), "rb").read()
        assert len(raw) == c["bytes"]
        assert xxhash.xxh64(raw, seed=0).intdigest() == int(c["xxh64"], 16)
        magic, fmt, seg, transform, first, count, payload = struct.unpack("<4sIiIqqq", raw[:40])
        assert (magic, fmt, seg, first, count) == (b"DTEC", 1, c["segment"], c["first"], c["count"])
        assert payload == 6 * count
        body = raw[40:] if man["codec"] == "none" else _zstd_decompress(raw[40:], payload)
        words = np.frombuffer(body[:4 * count], dtype="<u4").astype(np.int64)
        local = np.cumsum(words) if transform == 1 else words
        idx.append(man["segments"][seg]["flat_begin"] + local)
        val.append(np.frombuffer(body[4 * count:], dtype="<u2"))
    return (man, np.concatenate(idx) if idx else np.zeros(0, np.int64),
            np.concatenate(val) if val else np.zeros(0, np.uint16))


def segs_of(wl):
    return S.segments_of([t.name for t in wl.tensors], wl.flat_begins(),
                         [t.numel for t in wl.tensors])


@pytest.fixture(scope="module")
def delta():
    wl = W.scaled_dense(layers=2, tp=2, lr=1e-5)
    res = orun.extract(wl, keep=("ph", "p"), threads=2)
    return wl, res


def test_xxh64_matches_reference_implementation():
    rng = np.random.default_rng(5)
    for n in list(range(0, 80)) + [255, 256, 1000, 4099]:
        data = rng.integers(0, 256, n, dtype=np.uint8).tobytes()
        assert S.xxh64(data) == xxhash.xxh64(data, seed=0).intdigest(), n
    data = b"delta transfer engine"
    for seed in (1, 2**32 + 7, 2**64 - 1):
        assert S.xxh64(data, seed) == xxhash.xxh64(data, seed=seed).intdigest()


@pytest.mark.parametrize("codec,transform,chunk", [
    (S.CODEC_ZSTD, 1, 500), (S.CODEC_ZSTD, 0, 1 << 20), (S.CODEC_NONE, 1, 777),
    (S.CODEC_NONE, 0, 64)])
def test_round_trip_and_independent_reader(tmp_path, delta, codec, transform, chunk):
    wl, res = delta
    d = tmp_path / "store"
    opt = S.Options(codec=codec, level=3, threads=4, index_transform=transform,
                    chunk_entries=chunk)
    st = S.write_part_host(d, 1, 0, segs_of(wl), res.idx, res.val, opt)
    assert st.entries == res.idx.size and st.chunks >= 1
    assert S.commit(d, 1, 0, 1)
    assert S.latest(d) == 1
    idx, val, rs = S.read_host(d, 1, 0)
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    assert rs.stored_bytes == st.stored_bytes
    man, idx2, val2 = independent_read(str(d), 1)
    assert man["version"] == 1 and man["parent"] == 0 and man["entries"] == res.idx.size
    assert np.array_equal(idx2, res.idx) and np.array_equal(val2, res.val)
    if codec == S.CODEC_ZSTD and transform == 1:
        assert st.stored_bytes < st.raw_bytes


def test_destination_apply_gives_new_layout(tmp_path, delta):
    wl, res = delta
    d = tmp_path / "store"
    S.write_part_host(d, 1, 0, segs_of(wl), res.idx, res.val)
    assert S.commit(d, 1, 0, 1)
    idx, val, _ = S.read_host(d, 1, 0)
    pl = oplan.build_plan(wl)
    old = oremap.layout(pl, ocore.bf16(orun.flat(res.parts, "ph")))
    new = oremap.layout(pl, ocore.bf16(orun.flat(res.parts, "p")))
    got = oremap.apply(old, oremap.remap(pl, idx, val))
    for r in range(pl.nranks):
        assert np.array_equal(got[r], new[r])


def test_no_change_publishes_no_version(tmp_path, delta):
    wl, res = delta
    d = tmp_path / "store"
    S.write_part_host(d, 1, 0, segs_of(wl), res.idx, res.val)
    assert S.commit(d, 1, 0, 1)
    for w in range(2):
        S.write_part_host(d, 2, w, segs_of(wl), np.zeros(0, np.int64), np.zeros(0, np.uint16))
    assert not S.commit(d, 2, 1, 2)
    assert S.latest(d) == 1
    assert not os.path.exists(d / "v2")


def test_two_writers_disjoint_partitions(tmp_path, delta):
    wl, res = delta
    d = tmp_path / "store"
    begins = wl.flat_begins()
    cut = begins[len(wl.tensors) // 2]
    lo = res.idx < cut
    S.write_part_host(d, 1, 0, segs_of(wl), res.idx[lo], res.val[lo])
    with pytest.raises(B.DteError) as e:         # writer 1 has not reported yet
        S.commit(d, 1, 0, 2)
    assert e.value.status == B.DTE_ERR_IO
    assert S.latest(d) == 0
    S.write_part_host(d, 1, 1, segs_of(wl), res.idx[~lo], res.val[~lo])
    assert S.commit(d, 1, 0, 2)
    idx, val, _ = S.read_host(d, 1, 0)
    assert np.array_equal(idx, res.idx) and np.array_equal(val, res.val)
    # both writers with entries of every segment (even / odd entries): the
    # version holds the union, grouped by segment then writer
    even = np.arange(res.idx.size) % 2 == 0
    S.write_part_host(d, 2, 0, segs_of(wl), res.idx[even], res.val[even])
    S.write_part_host(d, 2, 1, segs_of(wl), res.idx[~even], res.val[~even])
    assert S.commit(d, 2, 1, 2)
    idx, val, _ = S.read_host(d, 2, 1)
    srt = np.argsort(idx, kind="stable")
    assert np.array_equal(idx[srt], res.idx) and np.array_equal(val[srt], res.val)
    seg = np.searchsorted(np.array(begins), idx, side="right") - 1
    assert np.all(np.diff(seg) >= 0)


def test_version_chain(tmp_path, delta):
    wl, res = delta
    d = tmp_path / "store"
    for v in (1, 2, 3):
        k = res.idx.size * v // 3
        S.write_part_host(d, v, 0, segs_of(wl), res.idx[:k], res.val[:k])
        assert S.commit(d, v, v - 1, 1)
    assert S.latest(d) == 3
    assert S.chain(d, 0, 3) == [1, 2, 3]
    assert S.chain(d, 2, 3) == [3]
    assert S.chain(d, 3, 3) == []
    with pytest.raises(B.DteError) as e:
        S.read_host(d, 3, 1)                      # 3 extends 2, not 1
    assert e.value.status == B.DTE_ERR_CHAIN
    idx, _, _ = S.read_host(d, 2, 1)
    assert idx.size == res.idx.size * 2 // 3


def test_corrupted_and_truncated_chunks_are_rejected(tmp_path, delta):
    wl, res = delta
    d = tmp_path / "store"
    S.write_part_host(d, 1, 0, segs_of(wl), res.idx, res.val, S.Options(chunk_entries=1000))
    assert S.commit(d, 1, 0, 1)
    man = json.load(open(d / "v1" / "manifest.json"))
    path = d / "v1" / man["chunks"][1]["file"]
    good = path.read_bytes()
    bad = bytearray(good)
    bad[len(bad) // 2] ^= 0x40
    path.write_bytes(bytes(bad))
    with pytest.raises(B.DteError) as e:
        S.read_host(d, 1, 0)
    assert e.value.status == B.DTE_ERR_CORRUPT
    path.write_bytes(good[:-3])
    with pytest.raises(B.DteError) as e:
        S.read_host(d, 1, 0)
    assert e.value.status == B.DTE_ERR_CORRUPT
    path.write_bytes(good)
    idx, _, _ = S.read_host(d, 1, 0)
    assert idx.size == res.idx.size


def test_writer_rejects_bad_input(tmp_path, delta):
    wl, res = delta
    d = tmp_path / "store"
    segs = segs_of(wl)
    with pytest.raises(B.DteError):               # not ascending
        S.write_part_host(d, 1, 0, segs, res.idx[::-1], res.val)
    with pytest.raises(B.DteError):               # outside every segment
        S.write_part_host(d, 1, 0, segs, np.array([wl.numel + 5]), np.array([1], np.uint16))
    with pytest.raises(B.DteError):               # bad options
        S.write_part_host(d, 1, 0, segs, res.idx, res.val, S.Options(threads=0))
    with pytest.raises(B.DteError):               # version 0
        S.write_part_host(d, 0, 0, segs, res.idx, res.val)


def _mcore_delta_in_sender_offsets(wl):
    """The oracle's delta of the rank's elements (sec. 4.2.1, in canonical
    offsets) expressed as offsets of the rank's own shard, ascending."""
    from oracle import mcore
    ci = mcore.canonical_index(wl)
    res = mcore.extract(wl)
    order = np.argsort(ci, kind="stable")
    sender = order[np.searchsorted(ci[order], res.idx)]
    srt = np.argsort(sender, kind="stable")
    return sender[srt], res.val[srt]


def test_megatron_core_writers_publish_the_canonical_delta(tmp_path):
    """Two tensor-parallel trainer ranks of a Megatron-Core shard publish
    their changes mapped to canonical tensors (norms by rank 0 only); the
    committed version holds exactly the canonical model's delta."""
    from paper_2608_00455_amd import layouts
    wl0 = W.scaled_mcore(trainer_tp=2, trainer_rank=0, vocab=64, lr=1e-5)
    twin = W.canonical_twin(wl0)
    segs = segs_of(twin)
    d = tmp_path / "store"
    for r in range(2):
        wl = W.with_sender_rank(wl0, r)
        idx, val = _mcore_delta_in_sender_offsets(wl)
        pieces = S.pieces_of(layouts.store_pieces(wl))
        S.write_part_host(d, 1, r, segs, idx, val, S.Options(chunk_entries=300), pieces=pieces)
    assert S.commit(d, 1, 0, 2)
    idx, val, _ = S.read_host(d, 1, 0)
    want = orun.extract(twin, threads=2)
    srt = np.argsort(idx, kind="stable")
    assert np.array_equal(idx[srt], want.idx) and np.array_equal(val[srt], want.val)
    man, idx2, val2 = independent_read(str(d), 1)
    assert sorted({c["writer"] for c in man["chunks"]}) == [0, 1]
    srt2 = np.argsort(idx2, kind="stable")
    assert np.array_equal(idx2[srt2], want.idx)


def test_mapped_writer_rejects_overlapping_or_unmapped_entries(tmp_path, delta):
    wl, res = delta
    segs = segs_of(wl)
    n0 = wl.tensors[0].numel
    # two pieces claiming the same sender range
    bad = S.pieces_of([(0, n0, 0, n0, n0, 0, 0), (0, n0, 0, n0, n0, 0, 0)])
    with pytest.raises(B.DteError):
        S.write_part_host(tmp_path / "a", 1, 0, segs, res.idx[:1], res.val[:1], pieces=bad)
    # entries outside every piece
    only_first = S.pieces_of([(0, n0, 0, n0, n0, 0, 0)])
    with pytest.raises(B.DteError):
        S.write_part_host(tmp_path / "b", 1, 0, segs, res.idx, res.val, pieces=only_first)
