"""Builds libdcp.so (the C-ABI library of include/dcp.h) in place for gfx950."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["dcp_api.hip", "fast.hip", "proj.hip", "generic.hip", "merge.hip", "sparse.hip", "knn.hip", "transition.hip", "scatter.hip"]
FLAGS = ["-O3", "--offload-arch=gfx950", "-fPIC", "-shared", "-std=c++17",
         # hipcc's host pass warns that it does not know this feature; harmless
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]


def build(verbose: bool = False) -> str:
    out = os.path.join(HERE, "libdcp.so")
    cmd = ["hipcc", *FLAGS, *[os.path.join(HERE, "csrc", s) for s in SOURCES], "-o", out + ".tmp"]
    if verbose:
        cmd.insert(1, "-Rpass-analysis=kernel-resource-usage")
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
