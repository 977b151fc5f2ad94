"""Build the CPU oracle library (test infrastructure; see mosa_oracle.c)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mosa_oracle.c")
LIB = os.path.join(HERE, "liboracle_mosa.so")


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, strict IEEE double: no -ffast-math,
    no FMA contraction so every product and sum is rounded exactly as written)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
