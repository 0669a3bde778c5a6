"""Compiles the C oracle (ts_ref.c) into oracle/libts_ref.so with gcc and OpenMP.

Test infrastructure only (see ts_ref.c).  Plain -O2: no -ffast-math, so every sum keeps the
left-to-right order written in the source.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ts_ref.c")
LIB = os.path.join(HERE, "libts_ref.so")


def build(src=SRC, out=LIB):
    """Compile src into the shared library out; returns out."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
