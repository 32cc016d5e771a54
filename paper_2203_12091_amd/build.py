"""Builds libfxpq.so (gfx950) in-tree with hipcc."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libfxpq.so")
SOURCES = ["fxpq_api.hip", "k_stream.hip", "k_flsearch.hip", "k_conv.hip", "k_teacher.hip",
           "k_wide.hip"]


def build(verbose: bool = False) -> str:
    # -z defs: an undefined symbol (e.g. a kernel stub the host pass did not
    # emit) fails the build instead of the first dlopen
    cmd = ["hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wl,-z,defs",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include"), "-o", LIB + ".tmp"]
    cmd += [os.path.join(CSRC, s) for s in SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True, stdout=subprocess.DEVNULL if not verbose else None,
                   stderr=subprocess.PIPE if not verbose else None)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
