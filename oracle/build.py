"""Build the oracle's C library with gcc (test infrastructure only)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")


def build():
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-fno-fast-math", "-o", LIB,
                           os.path.join(HERE, "dte_oracle.c"), "-lm"])
    return LIB


if __name__ == "__main__":
    print(build())
