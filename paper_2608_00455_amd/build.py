"""Build libdte.so (HIP, gfx950) in-tree, and libceilings.so (the
benchmark's reference kernels: a plain read stream and whole-line scattered
writes, outside the C ABI).

Floating-point flags: no contraction into fused multiply-add, IEEE
subnormals, correctly rounded binary32 divide and square root, no packed
FP32 instructions.
"""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libdte.so")
SOURCES = ["dte_api.hip", "extract.hip", "remap.hip", "store.hip"]
CEIL_LIB = os.path.join(HERE, "libceilings.so")
CEIL_SOURCES = ["ceilings.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc():
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(extra=()):
    cmds = [[hipcc()] + HIPCC_FLAGS + list(extra) + ["-o", out] + [os.path.join(SRC, s) for s in srcs]
            for out, srcs in ((LIB, SOURCES), (CEIL_LIB, CEIL_SOURCES))]
    procs = [subprocess.Popen(c) for c in cmds]
    for p, c in zip(procs, cmds):
        if p.wait() != 0:
            raise subprocess.CalledProcessError(p.returncode, c)
    return LIB


def asm(source="extract.hip", out=None):
    """Device assembly of one source, for instruction inspection."""
    out = out or os.path.join(tempfile.gettempdir(), source.replace(".hip", ".s"))
    cmd = [hipcc()] + [f for f in HIPCC_FLAGS if f not in ("-shared", "-fPIC")] + \
        ["--cuda-device-only", "-S", "-o", out, os.path.join(SRC, source)]
    subprocess.check_call(cmd)
    return out


if __name__ == "__main__":
    print(asm(sys.argv[2]) if len(sys.argv) > 2 and sys.argv[1] == "asm" else build())
