"""Builds the fp64 CPU oracle (plain C, OpenMP). Test infrastructure only."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))


def build() -> str:
    out = os.path.join(HERE, "liboracle.so")
    # No -ffast-math: the oracle keeps IEEE fp64 semantics.
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                           os.path.join(HERE, "oracle.c"), "-lm", "-o", out + ".tmp"])
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build()
