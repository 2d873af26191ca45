"""Build the CPU oracle library (plain C, gcc, OpenMP) next to its source.

Test infrastructure only: the oracle is what the GPU path is checked against.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "kvlink_oracle.c")
LIB = os.path.join(HERE, "libkvlink_oracle.so")

CFLAGS = ["-std=c99", "-O2", "-fPIC", "-shared", "-fopenmp",
          "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra"]


def build(verbose=False):
    """Compile the oracle every time it is called; return the library path."""
    tmp = LIB + ".tmp"
    cmd = ["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
