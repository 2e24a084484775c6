"""Build the host (gcc) and device (hipcc, gfx950) generator libraries."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "csrc")

HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
               "-ffp-contract=off", "-fno-fast-math",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build_cpu():
    out = os.path.join(HERE, "libsynth_cpu.so")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-fno-fast-math", "-o", out, os.path.join(SRC, "synth_cpu.c"), "-lm"])
    return out


def build_hip():
    out = os.path.join(HERE, "libsynth_hip.so")
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    subprocess.check_call([hipcc] + HIPCC_FLAGS +
                          ["-o", out, os.path.join(SRC, "synth_hip.hip")])
    return out


def build_all():
    return build_cpu(), build_hip()


if __name__ == "__main__":
    print(build_all())
