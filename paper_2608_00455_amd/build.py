"""Build libdte.so (HIP, gfx950) in-tree.

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
    cmd = [hipcc()] + HIPCC_FLAGS + list(extra) + ["-o", LIB] + \
        [os.path.join(SRC, s) for s in SOURCES]
    subprocess.check_call(cmd)
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
