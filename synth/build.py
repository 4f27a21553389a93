"""Builds the generator's two native twins in place (host C and gfx950 HIP)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
HIP_FLAGS = ["-O3", "--offload-arch=gfx950", "-fPIC", "-shared", "-ffp-contract=off",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build_host() -> str:
    out = os.path.join(HERE, "libsynth_host.so")
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
                           os.path.join(HERE, "csrc", "synth_host.c"), "-lm", "-o", out + ".tmp"])
    os.replace(out + ".tmp", out)
    return out


def build_dev() -> str:
    out = os.path.join(HERE, "libsynth_dev.so")
    subprocess.check_call(["hipcc", *HIP_FLAGS, os.path.join(HERE, "csrc", "synth_dev.hip"), "-o", out + ".tmp"])
    os.replace(out + ".tmp", out)
    return out


def build() -> None:
    build_host()
    build_dev()


if __name__ == "__main__":
    build()
