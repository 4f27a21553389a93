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
