"""Deterministic atom -> token mean pooling on the GPU against the fp64 oracle,
through the C-ABI (GPU)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import DCP_BF16, DCP_F32, log, rel_err

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to("cuda:0")
    return torch.from_numpy(a).to("cuda:0")


def pool(a, idx, n_tokens, out_dtype=DCP_F32):
    """dcp_scatter_mean; a, idx host arrays. Returns the output as fp32 numpy."""
    import torch
    import paper_2607_05439_amd as dcp
    n_atoms, c = a.shape
    in_dtype = DCP_BF16 if a.dtype == np.uint16 else DCP_F32
    out = torch.full((max(n_tokens, 1), c), 7.0, dtype=torch.float32 if out_dtype == DCP_F32 else torch.bfloat16,
                     device="cuda:0")
    ws_bytes = dcp.dcp_scatter_mean_workspace_size(n_tokens, c)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda:0")
    dcp.dcp_scatter_mean(n_atoms, n_tokens, c, in_dtype, out_dtype, dev(a) if n_atoms else None,
                         dev(idx) if n_atoms else None, out, ws, ws.numel())
    return out.float().cpu().numpy()[:n_tokens]


def test_sorted_tokens_bf16_features():
    n_tok, c, _ = synth.SCATTER_WORKLOADS["pool300_f32"]
    idx = synth.token_index(n_tok)
    a = synth.atom_features(len(idx), c, bf16=True)
    ref = oracle.scatter_mean(a, idx, n_tok)
    err = rel_err(pool(a, idx, n_tok), ref)
    log(f"case sorted bf16 in, f32 out: rel err {err:.3e}")
    assert err <= 1e-6
    err = rel_err(pool(a, idx, n_tok, DCP_BF16), ref)
    assert err <= 1e-2


def test_any_order_is_bit_identical():
    """Random (unsorted) indices; permuting the atoms (with their indices)
    gives the same bits: the reduction does not depend on order."""
    r = np.random.default_rng(3)
    n_atoms, n_tok, c = 5000, 700, 96
    a = r.standard_normal((n_atoms, c)).astype(np.float32)
    idx = r.integers(0, n_tok, n_atoms).astype(np.int32)
    base = pool(a, idx, n_tok)
    ref = oracle.scatter_mean(a, idx, n_tok)
    assert rel_err(base, ref) <= 1e-6
    for seed in (4, 5):
        p = np.random.default_rng(seed).permutation(n_atoms)
        assert np.array_equal(pool(a[p], idx[p], n_tok), base)
    assert np.array_equal(pool(a, idx, n_tok), base)


def ordered_case(name):
    """Atoms in token order (the usual layout), with the structures a run-based
    reduction has to stitch together: tokens across run boundaries, gaps,
    out-of-range indices, long runs."""
    r = np.random.default_rng(len(name))
    if name == "gaps_and_out_of_range":
        n_tok, c = 400, 72
        idx = np.sort(np.concatenate([r.integers(-3, 0, 40), r.choice(np.arange(400)[::3], 900),
                                      r.integers(400, 405, 30)])).astype(np.int32)
    elif name == "one_token_over_many_runs":
        n_tok, c = 50, 128
        idx = np.sort(np.concatenate([np.full(3000, 7), r.integers(0, 50, 500), np.full(1000, 49)])).astype(np.int32)
    elif name == "long_runs":  # more than 64 atoms per token on average: runs of 384 atoms
        n_tok, c = 3, 512
        idx = np.sort(r.integers(0, 3, 1000)).astype(np.int32)
    elif name == "run_boundaries":  # tokens of exactly 64 and 65 atoms, aligned and not
        n_tok, c = 40, 64
        idx = np.repeat(np.arange(40), [64, 65, 1, 63] * 10).astype(np.int32)
    elif name == "end_gap_at_tile_edge":  # 128 atoms (two 64-atom tiles exactly), trailing empty tokens
        n_tok, c = 50, 32
        idx = np.sort(r.integers(0, 21, 128)).astype(np.int32)
    elif name == "single_atom":
        n_tok, c = 5, 8
        idx = np.array([2], dtype=np.int32)
    elif name == "odd_channel_count":
        n_tok, c = 30, 33
        idx = np.sort(r.integers(0, 30, 200)).astype(np.int32)
    else:  # all out of range
        n_tok, c = 6, 16
        idx = np.array([-1, -1, 6, 9], dtype=np.int32)
    a = (r.standard_normal((len(idx), c)) * 3).astype(np.float32)
    return a, idx, n_tok


@pytest.mark.parametrize("name", ["gaps_and_out_of_range", "one_token_over_many_runs", "long_runs", "run_boundaries",
                                  "end_gap_at_tile_edge", "single_atom", "all_out_of_range", "odd_channel_count"])
def test_ordered_atoms_match_oracle_and_shuffled_atoms(name):
    """Ordered atoms against the oracle, and bit for bit against a shuffled
    copy of the same atoms."""
    a, idx, n_tok = ordered_case(name)
    assert np.all(np.diff(idx) >= 0)
    got = pool(a, idx, n_tok)
    ref = oracle.scatter_mean(a, idx, n_tok)
    err = rel_err(got, ref) if np.abs(ref).max() > 0 else float(np.abs(got).max())
    log(f"case ordered {name}: {len(idx)} atoms, {n_tok} tokens, rel err {err:.3e}")
    assert err <= 1e-6
    present = np.zeros(n_tok, bool)
    present[idx[(idx >= 0) & (idx < n_tok)]] = True
    assert np.all(got[~present] == 0.0)
    if len(idx) > 1:
        p = np.random.default_rng(1).permutation(len(idx))
        while np.all(np.diff(idx[p]) >= 0):
            p = np.random.default_rng(int(p[0]) + 2).permutation(len(idx))
        assert np.array_equal(pool(a[p], idx[p], n_tok), got)
    assert np.array_equal(pool(a, idx, n_tok, DCP_BF16), pool(a[::-1][::-1].copy(), idx, n_tok, DCP_BF16))
    # bf16 features (rows of 2c bytes) through the same paths
    ab = synth.bf16_round(a)
    got_b = pool(ab, idx, n_tok)
    ref_b = oracle.scatter_mean(ab, idx, n_tok)
    assert (rel_err(got_b, ref_b) if np.abs(ref_b).max() > 0 else float(np.abs(got_b).max())) <= 1e-6
    if len(idx) > 1:
        assert np.array_equal(pool(ab[p], idx[p], n_tok), got_b)


@pytest.mark.parametrize("c", [1, 63, 65, 300, 512])
def test_channel_counts_and_edge_indices(c):
    r = np.random.default_rng(c)
    n_atoms, n_tok = 1500, 200
    a = (r.standard_normal((n_atoms, c)) * 100).astype(np.float32)
    idx = np.sort(r.integers(0, n_tok, n_atoms)).astype(np.int32)
    idx[::97] = -1         # no token
    idx[5::89] = n_tok     # out of range
    idx[idx == 17] = 18    # token 17 has no atoms
    got = pool(a, idx, n_tok)
    ref = oracle.scatter_mean(a, idx, n_tok)
    assert rel_err(got, ref) <= 1e-6
    assert np.all(got[17] == 0.0)


def test_one_crowded_token_and_empty_inputs():
    r = np.random.default_rng(9)
    a = r.standard_normal((20000, 128)).astype(np.float32)
    idx = np.zeros(20000, dtype=np.int32)
    idx[::1000] = 1
    got = pool(a, idx, 3)
    assert rel_err(got, oracle.scatter_mean(a, idx, 3)) <= 1e-6
    assert np.all(got[2] == 0.0)
    assert np.all(pool(np.zeros((0, 128), np.float32), np.zeros(0, np.int32), 5) == 0.0)


def test_pool24000_whole_workload():
    """The whole 24000-token assembly (about 216 000 atoms, bf16 features):
    every token against the oracle, and repeatable bits."""
    n_tok, c, dt = synth.SCATTER_WORKLOADS["pool24000_bf16"]
    idx = synth.token_index(n_tok)
    a = synth.atom_features(len(idx), c, bf16=dt == "bf16")
    log(f"case pool24000_bf16: {len(idx)} atoms")
    got = pool(a, idx, n_tok)
    err = rel_err(got, oracle.scatter_mean(a, idx, n_tok))
    log(f"  rel err {err:.3e}")
    assert err <= 1e-6
    assert np.array_equal(pool(a, idx, n_tok), got)


@pytest.mark.parametrize("c,bf16", [(8, True), (16, True), (24, True), (40, True), (136, True), (264, True),
                                    (512, True), (4, False), (12, False), (300, False), (512, False)])
def test_ordered_row_widths(c, bf16):
    """Ordered atoms with feature rows of 1 to 128 sixteen-byte chunks (lane
    groups of every width, and rows split over two slices): against the oracle
    and bit for bit against a shuffled copy."""
    r = np.random.default_rng(c + bf16)
    n_tok = 90
    idx = np.sort(np.concatenate([r.integers(0, n_tok, 700), [0, n_tok - 1]])).astype(np.int32)
    idx[idx == 33] = 34  # one empty token inside
    a = r.standard_normal((len(idx), c)).astype(np.float32)
    if bf16:
        a = synth.bf16_round(a)
    got = pool(a, idx, n_tok)
    ref = oracle.scatter_mean(a, idx, n_tok)
    log(f"case ordered width c={c} bf16={bf16}: rel err {rel_err(got, ref):.3e}")
    assert rel_err(got, ref) <= 1e-6
    assert np.all(got[33] == 0.0)
    p = np.random.default_rng(7).permutation(len(idx))
    assert np.array_equal(pool(a[p], idx[p], n_tok), got)


@pytest.mark.parametrize("bf16", [False, True])
def test_wide_magnitudes_every_feature_within_fixed_point_bound(bf16):
    """Features from 1e-12 to 2^28 in magnitude (rounding of tiny values, the
    exact conversion for large ones): every output within the fixed-point
    rounding (2^-33 per feature) plus the output rounding of the oracle's fp64
    mean, and bit-identical to a shuffled copy (the any-order path)."""
    r = np.random.default_rng(11 + bf16)
    n_tok, c = 300, 64
    idx = np.sort(r.integers(0, n_tok, 700)).astype(np.int32)
    mag = 10.0 ** r.uniform(-12, 8.4, (len(idx), c))
    a = np.clip(r.choice([-1.0, 1.0], (len(idx), c)) * mag, -2.0**28, 2.0**28).astype(np.float32)
    if bf16:
        a = synth.bf16_round(a)
    got = pool(a, idx, n_tok).astype(np.float64)
    ref = oracle.scatter_mean(a, idx, n_tok)
    bound = 2.0**-33 + 2.0**-24 * np.abs(ref)
    worst = float(np.max(np.abs(got - ref) / bound))
    log(f"case wide magnitudes bf16={bf16}: worst error / bound {worst:.3f}")
    assert worst <= 1.0
    p = np.random.default_rng(3).permutation(len(idx))
    assert np.array_equal(pool(a[p], idx[p], n_tok), got.astype(np.float32))


def test_one_inversion_takes_the_any_order_path():
    """A sorted index with one adjacent pair swapped deep inside a long array
    (one order-check flag of many set): still the exact means, bit-identical
    to the fully sorted atoms."""
    r = np.random.default_rng(21)
    n_tok, c = 9000, 32
    idx = np.sort(r.integers(0, n_tok, 80000)).astype(np.int32)
    a = r.standard_normal((len(idx), c)).astype(np.float32)
    k = int(np.nonzero(np.diff(idx[60000:]) > 0)[0][0]) + 60000  # idx[k] < idx[k + 1]
    p = np.arange(len(idx))
    p[k], p[k + 1] = k + 1, k
    assert np.any(np.diff(idx[p]) < 0)
    sorted_out = pool(a, idx, n_tok)
    swapped = pool(a[p], idx[p], n_tok)
    assert rel_err(swapped, oracle.scatter_mean(a, idx, n_tok)) <= 1e-6
    assert np.array_equal(swapped, sorted_out)


def test_workspace_contents_do_not_matter():
    """The order flags and the per-token plan are written, never cleared: a
    workspace full of arbitrary bytes, or one left by a larger call with other
    atoms, gives the same bits as a fresh one (ordered and shuffled atoms)."""
    import torch
    import paper_2607_05439_amd as dcp
    r = np.random.default_rng(31)

    def call(a, idx, n_tok, ws):
        out = torch.full((n_tok, a.shape[1]), 7.0, dtype=torch.float32, device="cuda:0")
        dcp.dcp_scatter_mean(len(idx), n_tok, a.shape[1], DCP_BF16 if a.dtype == np.uint16 else DCP_F32, DCP_F32,
                             dev(a), dev(idx), out, ws, ws.numel())
        return out.cpu().numpy()

    n_tok, c = 500, 64
    idx = np.sort(r.integers(0, n_tok, 4000)).astype(np.int32)
    idx[idx == 100] = 101  # an empty token
    a = r.standard_normal((len(idx), c)).astype(np.float32)
    ref = pool(a, idx, n_tok)
    ws_bytes = dcp.dcp_scatter_mean_workspace_size(2000, c)
    for fill in (0xFF, 0x00, 0x7F):
        ws = torch.full((ws_bytes,), fill, dtype=torch.uint8, device="cuda:0")
        assert np.array_equal(call(a, idx, n_tok, ws), ref)
    # a larger ordered call, then an unordered one, then the original, on one workspace
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda:0")
    idx_big = np.sort(r.integers(0, 2000, 9000)).astype(np.int32)
    a_big = r.standard_normal((len(idx_big), c)).astype(np.float32)
    assert rel_err(call(a_big, idx_big, 2000, ws), oracle.scatter_mean(a_big, idx_big, 2000)) <= 1e-6
    p = r.permutation(len(idx))
    assert np.array_equal(call(a[p], idx[p], n_tok, ws), ref)
    assert np.array_equal(call(a, idx, n_tok, ws), ref)
    assert np.all(ref[100] == 0.0)


def test_token_rows_spread_over_more_than_a_gib():
    """One token of 1.1 million atoms with 1 KiB feature rows: its rows span
    more than 2^30 bytes, beyond a 32-bit buffer offset, so the ordered path
    takes its 64-bit row loop. Against the oracle, next to a small token
    before it, one after it and an empty one."""
    r = np.random.default_rng(41)
    n_tok, c = 4, 256
    idx = np.repeat(np.arange(3, dtype=np.int32), [10, 1_100_000, 1000])
    a = r.standard_normal((len(idx), c), dtype=np.float32)
    assert int(np.sum(idx == 1)) * c * 4 > 2**30
    got = pool(a, idx, n_tok)
    ref = oracle.scatter_mean(a, idx, n_tok)
    log(f"case 1.1M-atom token: rel err {rel_err(got, ref):.3e}")
    assert rel_err(got, ref) <= 1e-6
    assert np.all(got[3] == 0.0)


def test_graph_capture_replays():
    """The pooling captured into a graph (the order check, the ordered sum
    and the gated any-order kernels) and replayed three times, with eager
    work, eager calls and synchronisations between the replays: every replay
    gives the eager bits, for ordered and for shuffled atoms."""
    import torch
    import paper_2607_05439_amd as dcp
    r = np.random.default_rng(51)
    n_tok, c = 700, 64
    idx = np.sort(r.integers(0, n_tok, 5000)).astype(np.int32)
    a = r.standard_normal((len(idx), c)).astype(np.float32)
    p = r.permutation(len(idx))
    for name, (aa, ii) in (("ordered", (a, idx)), ("shuffled", (a[p], idx[p]))):
        log(f"case graph capture, {name} atoms")
        ad, idd = dev(aa), dev(ii)
        ws_bytes = dcp.dcp_scatter_mean_workspace_size(n_tok, c)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda:0")
        out = torch.zeros((n_tok, c), dtype=torch.float32, device="cuda:0")

        def call():
            dcp.dcp_scatter_mean(len(ii), n_tok, c, DCP_F32, DCP_F32, ad, idd, out, ws, ws_bytes)

        call()
        torch.cuda.synchronize()
        ref = out.clone()
        assert rel_err(ref.cpu().numpy(), oracle.scatter_mean(aa, ii, n_tok)) <= 1e-6
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            call()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            call()
        torch.cuda.synchronize()
        for rep in range(3):
            out.fill_(-1.0)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, ref), (name, rep)
            out.fill_(5.0)
            call()
            torch.cuda.synchronize()
            assert torch.equal(out, ref), (name, rep)
