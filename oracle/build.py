"""Builds the oracle's C part (liboracle.so) with gcc.

TEST INFRASTRUCTURE ONLY: the oracle is the independent CPU reference that the
tests, the smoke check and the benchmark's CPU-baseline leg compare against.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "noise_ref.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(verbose: bool = False) -> str:
    """Compile oracle/noise_ref.c into oracle/liboracle.so and return its path.

    -ffp-contract=off keeps every multiply and add a separately rounded IEEE
    operation; no -ffast-math.  OpenMP parallelises over rows and words.
    """
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-o", tmp, SRC, "-lquadmath", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
