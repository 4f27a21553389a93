"""AddressSanitizer + UndefinedBehaviorSanitizer runs on the CPU: the fp64
oracle (every entry point, edge cases included, leak checking on) and the
C-ABI's host-side argument checks (the library's host code instrumented; no
kernel is launched). A mutated copy of the oracle with a one-element-short
allocation must be caught, which shows the instrumented build is real."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ORACLE_C = os.path.join(ROOT, "oracle", "oracle.c")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def have(tool):
    return shutil.which(tool) is not None


def build_oracle_driver(tmp_path, oracle_src):
    exe = str(tmp_path / "oracle_driver")
    subprocess.check_call(["gcc", "-std=c99", *SAN, "-fopenmp", oracle_src,
                           os.path.join(HERE, "sanitize", "oracle_driver.c"), "-lm", "-o", exe])
    return exe


def run(exe, leaks):
    env = dict(os.environ, OMP_NUM_THREADS="2", ASAN_OPTIONS=f"detect_leaks={1 if leaks else 0}:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    return subprocess.run([exe], env=env, capture_output=True, text=True, timeout=300)


@pytest.mark.skipif(not have("gcc"), reason="gcc not available")
def test_oracle_clean_under_asan_and_ubsan(tmp_path):
    r = run(build_oracle_driver(tmp_path, ORACLE_C), leaks=True)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "all entry points ran" in r.stdout


@pytest.mark.skipif(not have("gcc"), reason="gcc not available")
def test_sanitizer_catches_a_planted_overflow(tmp_path):
    src = open(ORACLE_C).read()
    planted = "calloc((size_t)(n_tokens > 0 ? n_tokens - 1 : 1), sizeof(int64_t))"
    original = "calloc((size_t)(n_tokens > 0 ? n_tokens : 1), sizeof(int64_t))"
    assert src.count(original) == 1
    mutant = tmp_path / "oracle_mutant.c"
    mutant.write_text(src.replace(original, planted))
    r = run(build_oracle_driver(tmp_path, str(mutant)), leaks=True)
    assert r.returncode != 0
    assert "AddressSanitizer" in r.stderr


@pytest.mark.skipif(not (have("hipcc") and os.path.exists("/opt/rocm/llvm/bin/clang")), reason="ROCm not available")
def test_c_abi_argument_checks_clean_under_asan_and_ubsan(tmp_path):
    lib_dir = tmp_path / "lib"
    lib_dir.mkdir()
    srcs = sorted(os.path.join(ROOT, "paper_2607_05439_amd", "csrc", f)
                  for f in os.listdir(os.path.join(ROOT, "paper_2607_05439_amd", "csrc")) if f.endswith(".hip"))
    # each sanitizer flag applies to the host pass only; the device code is
    # built at -O0 (the driver launches no kernel)
    subprocess.check_call(["hipcc", "--offload-arch=gfx950", "-Xarch_device", "-O0", "-O1", "-g", "-fPIC", "-shared",
                           "-std=c++17",
                           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                           "-Xarch_host", "-fno-sanitize-recover=all", "-I" + os.path.join(ROOT, "include"),
                           *srcs, "-o", str(lib_dir / "libdcp.so")],
                          stderr=subprocess.DEVNULL)
    exe = str(tmp_path / "boundary_driver")
    subprocess.check_call(["/opt/rocm/llvm/bin/clang", "-g", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-I" + os.path.join(ROOT, "include"),
                           os.path.join(HERE, "sanitize", "boundary_driver.c"), "-L" + str(lib_dir), "-ldcp",
                           "-Wl,-rpath," + str(lib_dir), "-o", exe])
    # the HIP runtime keeps allocations until exit: no leak check here
    r = run(exe, leaks=False)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "all checks behaved" in r.stdout
