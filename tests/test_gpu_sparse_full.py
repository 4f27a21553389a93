"""Sparse atom attention at full size: L = 96000 atoms (60 chains x 1600), a
24000-row stripe of P (73.7 GB bf16) in the launch configuration the
benchmark times (4 key blocks), checked on sampled query atoms against the
fp64 oracle, plus full-size properties (GPU)."""
import numpy as np
import pytest

import oracle
from gpu_helpers import DCP_BF16, AtomDevice, atom_workload, log, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def big():
    import torch
    assert torch.cuda.is_available()
    wl = atom_workload("atoms96k_bf16")
    log("allocating and generating P rows for atoms96k_bf16 (73.7 GB)")
    d = AtomDevice(wl)
    yield d
    del d
    torch.cuda.empty_cache()


def sampled(wl, n_random=256, seed=0):
    """First and last query of the stripe, queries at the key-block edges (their
    neighbours straddle two blocks) and random queries."""
    rows = {0, wl.n_q - 1}
    for p in range(wl.n_key_blocks):
        size, start = oracle.chunk(wl.n_atoms, wl.n_key_blocks, p)
        for atom in (start - 1, start, start + size - 1):
            if wl.q_row0 <= atom < wl.q_row0 + wl.n_q:
                rows.add(atom - wl.q_row0)
    rows.update(int(x) for x in np.random.default_rng(seed).choice(wl.n_q, n_random, replace=False))
    return sorted(rows)


def test_atoms96k_sampled_rows(big):
    wl = big.wl
    log("case atoms96k_bf16 n_kb=4 bf16 out (the benchmark's call), sampled query atoms")
    got = big.attention(wl.n_key_blocks, out_dtype=DCP_BF16).float().cpu().numpy()
    rows = sampled(wl)
    ref = big.oracle_rows(rows, n_blocks=wl.n_key_blocks)
    err = rel_err(got[rows], ref)
    log(f"  {len(rows)} rows rel err {err:.3e}")
    assert err <= 1e-2


def test_atoms96k_blocked_and_deterministic(big):
    import torch
    wl = big.wl
    log("case atoms96k_bf16 fp32 out: n_kb=4 twice, n_kb=1")
    a = big.attention(wl.n_key_blocks)
    b = big.attention(wl.n_key_blocks)
    assert torch.equal(a, b)
    c = big.attention(1)
    err = rel_err(c.cpu().numpy(), a.cpu().numpy())
    log(f"  blocked vs unblocked rel diff {err:.3e}")
    assert err <= 1e-6
    assert torch.isfinite(a).all()
