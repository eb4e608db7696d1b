"""Builds the CPU oracle library (test infrastructure; never linked by the GPU path)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libsdd_oracle.so")


def build(verbose: bool = False) -> str:
    """Compiles oracle/sdd_oracle.c with gcc (IEEE semantics: no fast-math, no FMA contraction)."""
    src = os.path.join(HERE, "sdd_oracle.c")
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off", "-fno-semantic-interposition",
           "-fno-fast-math", "-Wall", "-Wno-unknown-pragmas", "-o", LIB + ".tmp", src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
