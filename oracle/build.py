"""Build the CPU oracle (plain C, gcc) into ``oracle/liboracle_aqlm.so``.

Test infrastructure only; see ``aqlm_oracle.c``.  The flags keep every fp32
operation a single IEEE operation in source order: no contraction into FMA,
no fast-math reassociation.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "aqlm_oracle.c")
LIB = os.path.join(HERE, "liboracle_aqlm.so")

CFLAGS = ["-std=c11", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
          "-fno-fast-math", "-fexcess-precision=standard", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    cmd = ["gcc", *CFLAGS, "-o", LIB + ".tmp", SRC]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
