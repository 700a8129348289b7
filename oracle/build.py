"""Compile the fp64 C oracle into ``oracle/liboracle.so`` with gcc.

The oracle is test infrastructure: it is built next to the GPU library so the
checker exists wherever the library is built, but the GPU library never links
or loads it.  Strict IEEE semantics: no fast-math and no FMA contraction.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRCS = [os.path.join(HERE, "bhtsne_oracle.c"), os.path.join(HERE, "bhtsne_oracle3d.c")]
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O3", "-std=c11", "-fPIC", "-shared", "-fopenmp",
           "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
           *SRCS, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
