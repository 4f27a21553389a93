"""Builds libdcp.so (the C-ABI library of include/dcp.h) in place for gfx950.

Each source is compiled on its own (in parallel) and the objects are linked
into one shared library; no device code crosses translation units.
"""
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["dcp_api.hip", "fast.hip", "proj.hip", "generic.hip", "merge.hip", "sparse.hip", "knn.hip", "transition.hip", "scatter.hip"]
ARCH = ["--offload-arch=gfx950"]
FLAGS = ["-O3", *ARCH, "-fPIC", "-std=c++17",
         # hipcc's host pass warns that it does not know this feature; harmless
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
# Per-source additions. The fused transition issues its matrix-core products
# from a queue of LDS reads; LLVM's ILP-first machine scheduler orders that
# loop 1.7% faster than the default occupancy-first one (same bits; measured
# side by side on an 8000 x 8000 pair tensor). The other kernels gain nothing
# or lose with it, so it stays on this one source.
EXTRA = {"transition.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"]}


def build(verbose: bool = False) -> str:
    out = os.path.join(HERE, "libdcp.so")
    tmp = tempfile.mkdtemp(prefix="dcp_build_")
    try:
        def compile_one(src):
            obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
            cmd = ["hipcc", *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(HERE, "csrc", src), "-o", obj]
            if verbose:
                cmd.insert(1, "-Rpass-analysis=kernel-resource-usage")
            subprocess.check_call(cmd)
            return obj

        workers = min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
        with ThreadPoolExecutor(max_workers=workers) as ex:
            objs = list(ex.map(compile_one, SOURCES))
        subprocess.check_call(["hipcc", *ARCH, "-fPIC", "-shared", *objs, "-o", out + ".tmp"])
        os.replace(out + ".tmp", out)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
