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


def test_neighbour_lists_properties():
    """The kNN stand-in: in range, no repeats, the sequence-local atoms first,
    the inter-chain quota when there are more than three chains, deterministic."""
    wl = synth.ATOM_WORKLOADS["atoms5000_bf16"]
    nb = synth.neighbours(wl, 0, wl.n_atoms)
    assert nb.shape == (wl.n_atoms, wl.k) and nb.dtype == np.int32
    assert ((nb >= -1) & (nb < wl.n_atoms)).all()
    for i in (0, 1, 998, 999, 1000, 2345, 4999):
        row = nb[i][nb[i] >= 0]
        assert len(row) == len(set(row.tolist()))
        c0 = i // wl.per_chain * wl.per_chain
        r = (i - c0) // wl.per_res
        local = list(range(c0 + max(r - 1, 0) * wl.per_res, min(c0 + (r + 2) * wl.per_res, c0 + wl.per_chain)))
        assert row[:len(local)].tolist() == local
        if len(row) == wl.k:  # not one of the ragged rows
            assert (row // wl.per_chain != i // wl.per_chain).sum() == wl.q_inter
    assert np.array_equal(nb[100:200], synth.neighbours(wl, 100, 100))
    # ragged rows: some budgets left partly empty, filled slots stay in front
    valid = nb >= 0
    assert (valid.sum(1) < wl.k).any() and (valid.sum(1) == wl.k).mean() > 0.8
    assert all(not valid[i, t] or valid[i, :t].all() for i in range(0, 5000, 37) for t in range(wl.k))


def test_neighbour_lists_small_pools():
    """Fewer candidates than slots: every candidate once, the rest empty."""
    wl = synth.ATOM_WORKLOADS["atoms200_f32"]
    nb = synth.neighbours(wl, 0, wl.n_atoms)
    for i in (0, 77, 199):
        row = nb[i][nb[i] >= 0]
        own = row[row // wl.per_chain == i // wl.per_chain]
        assert sorted(own.tolist()) == list(range(i // 50 * 50, i // 50 * 50 + 50))
        assert len(row) - len(own) == wl.q_inter


def test_pair_slices_match_dense_rows():
    wl = synth.ATOM_WORKLOADS["atoms200_f32"]
    rows = [3, 150]
    nb = synth.neighbours(wl, 0, wl.n_atoms)[rows]
    got = synth.p_gathered_host(wl, rows, nb)
    dense = synth.p_rows_host(wl, rows)
    for r in range(2):
        for t in range(wl.k):
            if nb[r, t] >= 0:
                assert np.array_equal(got[r, t], dense[r, nb[r, t]])
            else:
                assert not got[r, t].any()
