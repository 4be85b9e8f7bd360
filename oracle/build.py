"""Build the CPU oracle library (test infrastructure) with gcc.

gcc -O2 -ffp-contract=off -mfma: explicit fma() only, no implicit contraction, no
fast-math, so every fp64 operation is the IEEE operation the source names.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
CMD = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-mfma", "-fPIC",
       "-shared", "-Wall", "-Wextra", "-Werror", SRC, "-o", LIB, "-lm"]


def build(force=False):
    if (not force and os.path.exists(LIB)
            and os.path.getmtime(LIB) >= max(os.path.getmtime(SRC),
                                             os.path.getmtime(os.path.join(HERE, "oracle.h")))):
        return LIB
    subprocess.run(CMD, check=True)
    return LIB


if __name__ == "__main__":
    build(force=True)
    print(LIB)
