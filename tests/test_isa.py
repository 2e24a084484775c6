"""Instruction-level checks of the device code as built (AMD assembly of
this repository's own sources, gfx950):

* no matrix-core (MFMA) instructions: nothing on the path is a contraction;
* no packed-FP32 arithmetic (the build disables it);
* no scalar-cache writes (scalar stores, scalar atomics, scalar cache
  write-back or discard): outputs go through vector stores only;
* no scratch memory (no register spills) in any kernel;
* the hot extract kernels (full tiles, vector loads, no theta_hat output)
  fit three waves per SIMD as one 12-wave block per CU: at most 168 VGPRs
  and the CU's 160 KB of LDS per block.
"""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2608_00455_amd import build as B  # noqa: E402

SOURCES = ["extract.hip", "remap.hip", "store.hip", "ceilings.hip"]


def _hipcc_ok():
    try:
        return os.path.exists(B.hipcc())
    except Exception:
        return False


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    if not _hipcc_ok():
        pytest.skip("hipcc not available")
    d = tmp_path_factory.mktemp("asm")
    procs, outs = [], {}
    for src in SOURCES:
        out = str(d / src.replace(".hip", ".s"))
        cmd = [B.hipcc()] + [f for f in B.HIPCC_FLAGS if f not in ("-shared", "-fPIC")] + \
            ["--cuda-device-only", "-S", "-o", out, os.path.join(B.SRC, src)]
        procs.append(subprocess.Popen(cmd, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE))
        outs[src] = out
    for p in procs:
        err = p.communicate(timeout=900)[1]
        assert p.returncode == 0, err.decode()[-2000:]
    return {src: open(path).read() for src, path in outs.items()}


def kernels(text):
    """(name, fields) of every kernel in the code object metadata."""
    start = text.index("amdhsa.kernels:")
    end = text.find("\namdhsa.", start)        # the next top-level metadata key
    meta = text[start:end if end > 0 else len(text)]
    out = []
    for entry in meta.split("\n  - ")[1:]:
        fields = dict(re.findall(r"\.(\w+):\s+(\S+)", entry))
        out.append((fields["name"], fields))
    return out


def test_no_matrix_core_or_packed_fp32_instructions(assembly):
    for src, text in assembly.items():
        assert not re.search(r"^\s+v_mfma", text, re.M), src
        assert not re.search(r"^\s+v_pk_(add|mul|fma)_f32\b", text, re.M), src


def test_no_scalar_cache_writes(assembly):
    pat = re.compile(r"^\s+s_(store|atomic|buffer_store|scratch_store|dcache_wb|dcache_discard)",
                     re.M)
    for src, text in assembly.items():
        assert not pat.search(text), src


def test_no_kernel_uses_scratch(assembly):
    n = 0
    for src, text in assembly.items():
        for name, f in kernels(text):
            assert int(f["private_segment_fixed_size"]) == 0, (src, name)
            n += 1
    assert n > 20


def test_hot_extract_kernels_fit_three_waves_per_simd(assembly):
    hot = []
    for name, f in kernels(assembly["extract.hip"]):
        m = re.search(r"extract_kernelILb(\d)ELb(\d)ELb(\d)ELb(\d)ELb(\d)ELb(\d)E", name)
        if not m:
            continue
        full, vec, _, prev, _, _ = (int(x) for x in m.groups())
        if full and vec and not prev:
            hot.append(name)
            assert int(f["vgpr_count"]) <= 168, (name, f["vgpr_count"])
            assert int(f["agpr_count"]) == 0, name
            assert int(f["group_segment_fixed_size"]) <= 160 * 1024, name
    # decay == 1 or not, folded or literal order, with or without routing
    assert len(hot) == 8
