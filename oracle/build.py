"""Builds the oracle's shared library with gcc (test infrastructure only)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "fxpq_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


CFLAGS = ["-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
          "-fno-fast-math", "-ffp-contract=off"]


def build(verbose: bool = False) -> str:
    cmd = ["gcc"] + CFLAGS + ["-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
