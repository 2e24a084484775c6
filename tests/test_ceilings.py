"""The benchmark's reference kernels (libceilings.so, outside the C ABI of
include/dte.h): exported entry points, argument checks made before any
device work, and, on the GPU, the bytes each reference kernel writes."""
import ctypes
import os

import numpy as np
import pytest

from paper_2608_00455_amd import build as dte_build

P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
TILE = 2048   # elements per wave tile of the read kernels


def lib():
    if not os.path.exists(dte_build.CEIL_LIB):
        pytest.skip("libceilings.so not built")
    L = ctypes.CDLL(dte_build.CEIL_LIB)
    L.ceil_read3_waves.restype = I64
    L.ceil_read3_waves.argtypes = [I32]
    L.ceil_read3.restype = ctypes.c_int
    L.ceil_read3.argtypes = [P, P, P, I64, I32, P, P]
    L.ceil_read3_dynamic.restype = ctypes.c_int
    L.ceil_read3_dynamic.argtypes = [P, P, P, I64, P, P, P]
    L.ceil_read3_write.restype = ctypes.c_int
    L.ceil_read3_write.argtypes = [P, P, P, I64, I64, P, P, I32, P, P]
    L.ceil_write_entries.restype = ctypes.c_int
    L.ceil_write_entries.argtypes = [I64, P, P, I32, P]
    L.ceil_line_writes.restype = ctypes.c_int
    L.ceil_line_writes.argtypes = [I32, P, P, P, P, P, I32, P]
    return L


def test_bad_arguments_are_refused_before_device_work():
    L = lib()
    fake = 4096   # never dereferenced: every call below fails its checks first
    assert L.ceil_read3(None, fake, fake, 1 << 20, 3, fake, None) == 1
    assert L.ceil_read3(fake, fake, fake, -1, 3, fake, None) == 1
    assert L.ceil_read3(fake + 4, fake, fake, 1 << 20, 3, fake, None) == 1     # misaligned
    assert L.ceil_read3(fake, fake, fake, 1 << 20, 0, fake, None) == 1
    assert L.ceil_read3_dynamic(fake, fake, fake, 1 << 20, None, fake, None) == 1
    assert L.ceil_read3_dynamic(fake, fake + 8, fake, 1 << 20, fake, fake, None) == 1
    assert L.ceil_read3_dynamic(fake, fake, fake, -1, fake, fake, None) == 1
    assert L.ceil_read3_write(fake, fake, fake, 1 << 20, 10, None, fake, 3, fake, None) == 1
    assert L.ceil_read3_write(fake, fake, fake, 1 << 20, -1, fake, fake, 3, fake, None) == 1
    assert L.ceil_read3_write(fake, fake, fake, 1 << 20, 10, fake + 4, fake, 3, fake, None) == 1
    assert L.ceil_read3_write(fake, fake, fake, 1 << 20, 10, fake, fake + 1, 3, fake, None) == 1
    # E (t + 1) would not fit 64 bits
    assert L.ceil_read3_write(fake, fake, fake, TILE << 30, 1 << 40, fake, fake, 3, fake,
                              None) == 1
    assert L.ceil_write_entries(10, None, fake, 4, None) == 1
    assert L.ceil_write_entries(-1, fake, fake, 4, None) == 1
    assert L.ceil_write_entries(10, fake, fake, 0, None) == 1
    assert L.ceil_write_entries(0, fake, fake, 4, None) == 0                   # nothing to do
    assert L.ceil_line_writes(0, None, None, None, None, None, 4, None) == 1
    assert L.ceil_line_writes(17, None, None, None, None, None, 4, None) == 1


@pytest.mark.gpu
def test_reference_kernels_write_what_they_state():
    import torch
    L = lib()
    s = torch.cuda.current_stream()
    n = 37 * TILE + 100                    # whole tiles only are read
    a, b, c = (torch.randn(n, device="cuda") for _ in range(3))
    sink = torch.zeros(64 * L.ceil_read3_waves(3), dtype=torch.int32, device="cuda")
    assert L.ceil_read3(a.data_ptr(), b.data_ptr(), c.data_ptr(), n, 3, sink.data_ptr(),
                        s.cuda_stream) == 0
    counter = torch.zeros(1, dtype=torch.int64, device="cuda")
    assert L.ceil_read3_dynamic(a.data_ptr(), b.data_ptr(), c.data_ptr(), n, counter.data_ptr(),
                                sink.data_ptr(), s.cuda_stream) == 0
    torch.cuda.synchronize()
    # every block takes chunks of 48 tiles until one starts past the end
    chunks = -(-(n // TILE) // 48)
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    assert int(counter.item()) == chunks + blocks
    tiles, e = n // TILE, 1001
    idx = torch.full((e + 8,), -7, dtype=torch.int64, device="cuda")
    val = torch.full((e + 8,), 7, dtype=torch.int16, device="cuda")
    assert L.ceil_read3_write(a.data_ptr(), b.data_ptr(), c.data_ptr(), n, e, idx.data_ptr(),
                              val.data_ptr(), 2, sink.data_ptr(), s.cuda_stream) == 0
    torch.cuda.synchronize()
    want = np.empty(e, np.int64)
    for t in range(tiles):                 # tile t: entries [E t / tiles, E (t+1) / tiles)
        e0, e1 = e * t // tiles, e * (t + 1) // tiles
        want[e0:e1] = t * TILE + np.arange(e1 - e0)
    got = idx.cpu().numpy()
    assert np.array_equal(got[:e], want) and (got[e:] == -7).all()
    gv = val.cpu().numpy().view(np.uint16)
    assert np.array_equal(gv[:e], np.arange(e, dtype=np.uint16)) and (gv[e:] == 7).all()
    idx.fill_(-7)
    val.fill_(7)
    assert L.ceil_write_entries(e, idx.data_ptr(), val.data_ptr(), 4, s.cuda_stream) == 0
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    assert np.array_equal(got[:e], np.arange(e)) and (got[e:] == -7).all()
    gv = val.cpu().numpy().view(np.uint16)
    assert np.array_equal(gv[:e], np.arange(e, dtype=np.uint16)) and (gv[e:] == 7).all()
    # whole 64-byte lines of the pattern 0x3F80 at the lines of the offsets
    numel = [4096, 1000]
    dst = [torch.zeros(k, dtype=torch.int16, device="cuda") for k in numel]
    offs = [torch.tensor([5, 40, 41, 4095], dtype=torch.int64, device="cuda"),
            torch.tensor([990, 3], dtype=torch.int64, device="cuda")]
    count = torch.tensor([4, 2], dtype=torch.int64, device="cuda")
    arr = lambda T, xs: (T * 2)(*xs)       # noqa: E731
    assert L.ceil_line_writes(2, arr(P, [t.data_ptr() for t in dst]),
                              arr(P, [t.data_ptr() for t in offs]), count.data_ptr(),
                              arr(I64, [4, 2]), arr(I64, numel), 4, s.cuda_stream) == 0
    torch.cuda.synchronize()
    for k, (d, o) in enumerate(zip(dst, offs)):
        want = np.zeros(numel[k], np.uint16)
        for j in o.cpu().tolist():
            line = j // 32
            if (line + 1) * 32 <= numel[k]:    # lines not whole inside the buffer: skipped
                want[line * 32:(line + 1) * 32] = 0x3F80
        assert np.array_equal(d.cpu().numpy().view(np.uint16), want), k
