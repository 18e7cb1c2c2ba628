"""Compile the C oracle (``qdref.c``) into ``libqdref.so`` with gcc.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "qdref.c")
LIB = os.path.join(HERE, "libqdref.so")


def build(force: bool = True) -> str:
    """Build ``libqdref.so`` next to its source and return its path."""
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.run(
        ["gcc", "-O2", "-fPIC", "-shared", "-std=c99", "-o", tmp, SRC, "-lpthread", "-lm"],
        check=True,
    )
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
