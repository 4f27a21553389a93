"""The kNN kernel rejects a candidate without computing its distance when
e = |c|^2 - 2 c.q (three fp32 multiply-adds) exceeds a per-query limit
(T - |q|^2) + 2^-19 (T + rho^2), rho = |q| + 1.001 sqrt(T), where T is the
current k-th distance. This checks, with the same fp32 operation order on the
host, that no candidate whose distance (as the definition rounds it) is at most
T is rejected, over coordinates near and far from the origin and thresholds
from the nearest neighbour to the 2000th. It does not run the kernel; the GPU
tests compare the kernel's lists with the oracle."""
import numpy as np
import pytest

import synth

F = np.float32


def fma(a, b, c):
    # one rounding of a*b + c: the fp32 product is exact in fp64
    return (np.float64(a) * np.float64(b) + np.float64(c)).astype(F)


def d2_definition(q, c):
    dx, dy, dz = (F(q[0]) - c[:, 0]), (F(q[1]) - c[:, 1]), (F(q[2]) - c[:, 2])
    return ((dx * dx) + (dy * dy)) + (dz * dz)


@pytest.mark.parametrize("scale,shift", [(1.0, 0.0), (1.0, 3000.0), (1.0, -250000.0), (1e-4, 7.0), (1e5, 0.0)])
def test_no_candidate_within_the_kth_distance_is_rejected(scale, shift):
    x = (synth.coords(synth.KNN_WORKLOADS["knn5000"]).astype(np.float64) * scale + shift).astype(F)
    cc = fma(x[:, 0], x[:, 0], fma(x[:, 1], x[:, 1], x[:, 2] * x[:, 2]))
    rng = np.random.default_rng(5)
    for qi in rng.integers(0, len(x), 30):
        q = x[qi]
        d = d2_definition(q, x)
        e = fma(x[:, 0], F(-2) * q[0], fma(x[:, 1], F(-2) * q[1], fma(x[:, 2], F(-2) * q[2], cc)))
        qq = fma(q[0], q[0], fma(q[1], q[1], q[2] * q[2]))
        qn = np.sqrt(qq)
        ds = np.sort(d)
        for k in (1, 2, 64, 128, 256, 2000):
            T = ds[k - 1]
            rho = qn + F(1.001) * np.sqrt(T)
            lim = (T - qq) + F(2.0**-19) * (T + rho * rho)
            inside = d <= T
            assert inside.sum() >= k
            assert not np.any(e[inside] > lim), (qi, k)
