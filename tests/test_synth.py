"""The seeded input generator: the C twin equals the numpy definition (CPU only)."""
import numpy as np

import synth


def test_normal_twins_bit_identical():
    k = synth.key(3, synth.T_Z)
    for start, count in ((0, 1000), (2**40 + 17, 5000)):
        a = synth.normal_np(k, start, count)
        b = synth.normal(k, start, count)
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
        assert np.array_equal(synth.bf16_round(a), synth.normal(k, start, count, bf16=True))


def test_normal_moments():
    x = synth.normal(synth.key(0, synth.T_S), 0, 1 << 20).astype(np.float64)
    assert abs(x.mean()) < 5e-3 and abs(x.std() - 1.0) < 5e-3
    assert np.all(np.abs(x) <= 6.0)
    # exact fp32 values on the 2^-16 grid
    assert np.array_equal(x * 65536, np.round(x * 65536))


def test_z_rows_twins_bit_identical():
    for period in (0, 7):
        for bf16 in (False, True):
            a = synth.z_rows_np(11, 12, period, 30, 16, [0, 9, 29], bf16)
            b = synth.z_rows(11, 12, period, 30, 16, [0, 9, 29], bf16)
            assert a.dtype == b.dtype and np.array_equal(a, b)


def test_structured_z_has_period():
    wl = synth.WORKLOADS["ico4800_bf16"]
    z = synth.z_host(wl, [0, 80])  # rows 0 and 80 share base rows
    a, b = synth.bf16_to_f32(z[0]), synth.bf16_to_f32(z[1])
    # base is shared, the 0.1*noise term differs: |a - b| is small relative to |a|
    assert np.std(a - b) < 0.2 and np.std(a) > 0.9
    assert np.std(synth.bf16_to_f32(z[0, :80]) - synth.bf16_to_f32(z[0, 80:160])) < 0.2


def test_bf16_round_ties_to_even():
    x = np.array([1.0 + 2**-8, 1.0 + 3 * 2**-8, -(1.0 + 2**-8), 1.0 + 2**-8 + 2**-20], np.float32)
    got = synth.bf16_to_f32(synth.bf16_round(x))
    assert list(got) == [1.0, 1.0 + 4 * 2**-8, -1.0, 1.0 + 2 * 2**-8]


def test_masks():
    m2 = synth.mask_host(synth.WORKLOADS["pad1024_bf16"])
    assert m2.sum() == 1020 and np.all(m2[-4:] == 0)
    m3 = synth.mask_host(synth.WORKLOADS["ico4800_bf16"])
    assert m3.sum() == 4560
    assert np.array_equal(m3, synth.mask_host(synth.WORKLOADS["ico4800_bf16"]))
    m5 = synth.mask_host(synth.WORKLOADS["asm24000_bf16"])
    assert m5.sum() == 23520 and np.all(m5[-480:] == 0)
    assert synth.mask_host(synth.WORKLOADS["grid12000_bf16"]) is None


def test_weights_scale():
    wl = synth.WORKLOADS["asm24000_bf16"]
    w = synth.weights(wl)
    assert w["w_q"].shape == (384, 384) and w["w_b"].shape == (16, 128)
    assert abs(w["w_q"].std() * np.sqrt(384) - 1.0) < 0.02
    assert abs(w["w_b"].std() * np.sqrt(128) - 1.0) < 0.05
    assert not np.array_equal(w["w_q"], w["w_k"])
