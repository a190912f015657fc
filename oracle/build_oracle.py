"""Build step for the CPU oracle: compiles mg_oracle.c into liboracle_mg.so (gcc, OpenMP).

Test infrastructure only.  -ffp-contract=off keeps every product and sum a separate
IEEE rounding unless the source writes fmaf(); no -ffast-math, so no reassociation,
no flush-to-zero and no approximate libm calls.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mg_oracle.c")
LIB = os.path.join(HERE, "liboracle_mg.so")

CFLAGS = ["-O3", "-mfma", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
          "-fno-fast-math", "-fno-finite-math-only", "-Wall", "-Wno-unknown-pragmas"]


def build(verbose: bool = False) -> str:
    cmd = ["gcc", *CFLAGS, SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
