"""Compile the CPU oracle (test infrastructure) into oracle/liboracle.so and,
from the same source with OpenMP on, oracle/liboracle_omp.so.

The oracle is plain C built without floating-point contraction or fast-math so
that each operation is one correctly rounded IEEE-754 operation.  The OpenMP
build runs the loops whose iterations are independent over several host
threads (used only to time the oracle on all host cores); its results are
identical.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "termezo_oracle.c")
OUT = os.path.join(HERE, "liboracle.so")
OUT_OMP = os.path.join(HERE, "liboracle_omp.so")
FLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fno-builtin", "-Wall",
         "-Wextra", "-shared", "-fPIC"]


def build(verbose: bool = False) -> str:
    for out, extra in ((OUT, ["-Wno-unknown-pragmas"]), (OUT_OMP, ["-fopenmp"])):
        cmd = ["gcc", *FLAGS, *extra, SRC, "-o", out + ".tmp", "-lm"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(out + ".tmp", out)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
