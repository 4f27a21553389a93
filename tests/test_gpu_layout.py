"""In-bounds checks of the gfx950 builtin lane layouts the fused kernels use
(one wave each; GPU)."""
import ctypes
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def probe():
    import torch
    assert torch.cuda.is_available()
    torch.zeros(1, device="cuda")
    lib = ctypes.CDLL(os.path.join(HERE, "probes", "libprobe.so"))
    for f in ("probe_mfma32", "probe_mfma16", "probe_swaps", "probe_transpose"):
        getattr(lib, f).argtypes = [ctypes.c_void_p]
    lib.probe_exp2.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    lib.probe_dma.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    return lib, torch


def run(probe, name, n):
    lib, torch = probe
    out = torch.full((n,), -1.0, device="cuda")
    assert getattr(lib, name)(out.data_ptr()) == 0
    return out.cpu().numpy()


L = np.arange(64)
N, G = L % 16, L // 16


@pytest.mark.parametrize("name", ["probe_mfma32", "probe_mfma16"])
def test_accumulator_layout(probe, name):
    d = run(probe, name, 256).reshape(64, 4)
    want = ((4 * G[:, None] + np.arange(4)[None, :]) * 16 + N[:, None]).astype(np.float32)
    assert np.array_equal(d, want)


def test_swaps_and_reductions(probe):
    o = run(probe, "probe_swaps", 64 * 6).reshape(64, 6)
    lo = L < 32
    assert np.array_equal(o[:, 0], np.where(lo, L, 100 + L - 32))
    assert np.array_equal(o[:, 1], np.where(lo, L + 32, 100 + L))
    even = (G % 2) == 0
    assert np.array_equal(o[:, 2], np.where(even, L, 100 + L - 16))
    assert np.array_equal(o[:, 3], np.where(even, L + 16, 100 + L))
    assert np.array_equal(o[:, 4], 4 * N + 96)
    f = (37 * L) % 64
    assert np.array_equal(o[:, 5], np.array([max(f[n + 16 * k] for k in range(4)) for n in N]))


def test_bias_transpose(probe):
    o = run(probe, "probe_transpose", 64 * 64).reshape(64, 16, 4)
    want = np.empty_like(o)
    for lane in range(64):
        n, g = lane % 16, lane // 16
        for a in range(4):
            for r in range(4):
                for i in range(4):
                    want[lane, 4 * a + r, i] = (n + 16 * a) * 64 + (4 * g + r) * 4 + i
    assert np.array_equal(o, want)


def test_exp2_of_integers_is_exact(probe):
    lib, torch = probe
    k = np.arange(-140, 128, dtype=np.float32)
    x = torch.from_numpy(k).cuda()
    y = torch.empty_like(x)
    assert lib.probe_exp2(x.data_ptr(), y.data_ptr(), len(k)) == 0
    want = np.ldexp(np.float32(1.0), k.astype(np.int32)).astype(np.float32)
    want[k < -126] = 0.0  # the hardware flushes denormal results to zero
    assert np.array_equal(y.cpu().numpy(), want)


def test_direct_to_lds_loads(probe):
    lib, torch = probe
    src = torch.arange(192 * 4, dtype=torch.int32, device="cuda") * 7 + 1
    out = torch.zeros(256 * 4, dtype=torch.int32, device="cuda")
    assert lib.probe_dma(src.data_ptr(), out.data_ptr()) == 0
    s = src.cpu().numpy().reshape(192, 4)
    o = out.cpu().numpy().reshape(256, 4)
    lane = np.arange(64)
    assert np.array_equal(o[:64], s[lane ^ 5])                    # lane L lands at base + 16 L
    assert np.array_equal(o[64:128], s[64 + (lane ^ 9)])          # destination above 64 KB
    assert np.array_equal(o[192:256], s[128 + (lane ^ 3)])        # near the top of 160 KB
    oob = o[128:192]
    zeros = np.all(oob == 0)
    untouched = np.all(oob[:, 0].astype(np.uint32) == (0xDEAD0000 + 102400 // 16 + lane).astype(np.uint32))
    print("out-of-range DMA:", "writes zeros" if zeros else "leaves LDS untouched" if untouched else "other")
    assert zeros or untouched
