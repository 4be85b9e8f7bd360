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


def build_variant(source_text, lib_path):
    """Compile `source_text` (a modified copy of oracle.c, written next to `lib_path`) with
    the oracle's own flags into `lib_path`. The tests use this to check that each pin
    rejects a deliberately broken oracle; the real library is untouched."""
    src = os.path.splitext(lib_path)[0] + ".c"
    with open(src, "w") as f:
        f.write(source_text)
    cmd = [a for a in CMD]
    cmd[cmd.index(SRC)] = src
    cmd[cmd.index(LIB)] = lib_path
    subprocess.run(cmd + ["-I", HERE], check=True)
    return lib_path
