"""Builds the oracle shared library (plain C, gcc).  Test infrastructure only."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liborc.so")


def build(verbose: bool = False) -> str:
    """Compile attn_oracle.c into liborc.so next to it and return its path.

    Plain FP64 C: no fused multiply-add contraction and no fast-math, so the
    oracle's arithmetic is the arithmetic written in the source on any x86-64
    host; OpenMP only splits independent rows across threads."""
    src = os.path.join(HERE, "attn_oracle.c")
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, src, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
