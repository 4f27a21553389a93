"""Sparse (kNN) pair-biased atom attention on the GPU against the fp64 oracle,
through the C-ABI (GPU)."""
import numpy as np
import pytest

from gpu_helpers import DCP_BF16, DCP_F32, AtomDevice, atom_workload, log, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    import torch
    assert torch.cuda.is_available()
    return AtomDevice(atom_workload("atoms200_f32"), affine=True)


@pytest.fixture(scope="module")
def mid():
    log("generating atoms5000_bf16 (P rows 800 MB)")
    return AtomDevice(atom_workload("atoms5000_bf16"))


def test_tiny_f32_matches_oracle(tiny):
    """fp32 path, affine LayerNorm and projection bias (which the kernel may
    drop: per-head constants), budgets with empty slots, 4 chains."""
    n = tiny.wl.n_q
    ref = tiny.oracle_rows(np.arange(n))
    for n_kb in (1, 3, 200):
        log(f"case atoms200_f32 n_kb={n_kb}")
        got = tiny.attention(n_kb).cpu().numpy()
        err = rel_err(got, ref)
        log(f"  rel err {err:.3e}")
        assert err <= 1e-5


def test_tiny_blocked_equals_unblocked(tiny):
    a = tiny.attention(1).cpu().numpy()
    for n_kb in (2, 7, 200):
        b = tiny.attention(n_kb).cpu().numpy()
        assert rel_err(b, a) <= 1e-6, n_kb


def test_mid_bf16_matches_oracle(mid):
    n = mid.wl.n_q
    ref = mid.oracle_rows(np.arange(n))
    log("case atoms5000_bf16 n_kb=1 fp32 out")
    got = mid.attention(1).cpu().numpy()
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= 1e-2
    log("case atoms5000_bf16 n_kb=5 bf16 out")
    got = mid.attention(5, out_dtype=DCP_BF16).float().cpu().numpy()
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= 1e-2


def test_mid_blocked_deterministic(mid):
    import torch
    a = mid.attention(1)
    b = mid.attention(5)
    c = mid.attention(5)
    assert torch.equal(b, c)
    err = rel_err(b.cpu().numpy(), a.cpu().numpy())
    log(f"  blocked vs unblocked rel diff {err:.3e}")
    assert err <= 1e-6


def test_gathered_slices_equal_dense_rows(mid):
    """p_gathered = 1 (P_sparse given) reads the same values as the gather
    from the dense rows: identical bits."""
    import torch
    pg = mid.gathered_p()
    a = mid.attention(3)
    b = mid.attention(3, p=pg, p_gathered=1)
    assert torch.equal(a, b)


def test_sub_stripe_and_empty_call(mid):
    """A call on part of the stripe gives those rows of the full call; n_q = 0 is a no-op."""
    import torch
    full = mid.attention(2)
    part = mid.attention(2, row0=1234, n_q=777)
    assert torch.equal(part, full[1234:1234 + 777])
    mid.attention(2, row0=10, n_q=0)
    torch.cuda.synchronize()


def test_edge_neighbour_lists(tiny):
    """Empty rows, out-of-range indices, repeats, one neighbour, blocks with a
    single slot."""
    import torch
    wl = tiny.wl
    nb = tiny.nbr_host.copy()
    nb[0, :] = -1                 # all empty: 0
    nb[1, :] = 1000               # out of range: empty
    nb[2, :] = 17                 # one atom in every slot
    nb[3, 5:] = -1                # 5 slots
    nb[4, :] = np.arange(wl.k) % 3  # heavy repeats
    nb[5, :] = -1
    nb[5, 0] = wl.n_atoms - 1     # a single neighbour: the last atom
    nb[6, ::2] = -7               # negative but not -1
    ref = tiny.oracle_rows(np.arange(wl.n_q), nbr=nb)
    got = tiny.attention(4, nbr=torch.from_numpy(nb).to(tiny.dev)).cpu().numpy()
    assert np.all(got[0] == 0) and np.all(got[1] == 0)
    err = rel_err(got, ref)
    log(f"  edge lists rel err {err:.3e}")
    assert err <= 1e-5


def test_edge_neighbour_lists_bf16():
    """Edge lists on the bf16 path: empty, out-of-range and negative slots,
    one atom in every slot, heavy repeats, 16 consecutive query atoms without
    neighbours, two queries with the same list, every neighbour listed twice."""
    import torch
    wl = atom_workload("atoms5000_bf16", n_q=40, q_row0=300)
    d = AtomDevice(wl, affine=True)
    nb = d.nbr_host.copy()
    nb[0, :] = -1
    nb[1, :] = wl.n_atoms + 5
    nb[2, :] = 17
    nb[3, 5:] = -1
    nb[4, :] = np.arange(wl.k) % 3
    nb[5, :] = -1
    nb[5, 0] = wl.n_atoms - 1
    nb[6, ::2] = -7
    nb[16:32, :] = -1
    nb[33, :] = nb[34, :]
    nb[35, wl.k // 2:] = nb[35, :wl.k // 2]
    log(f"case atoms5000_bf16 edge lists, k={wl.k}, rows 300..339")
    ref = d.oracle_rows(np.arange(wl.n_q), nbr=nb)
    got = d.attention(4, nbr=torch.from_numpy(nb).to(d.dev)).cpu().numpy()
    assert np.all(got[0] == 0) and np.all(got[1] == 0) and np.all(got[16:32] == 0)
    err = rel_err(got, ref)
    log(f"  edge lists rel err {err:.3e}")
    assert err <= 1e-2


@pytest.mark.parametrize("k", [1, 63, 100, 256])
def test_slot_counts(k):
    """Budgets that are not a multiple of 64, a single slot, and the 256-slot
    maximum (the wider kernel variant)."""
    wl = atom_workload("atoms5000_bf16", k=k, n_q=700, q_row0=1500)
    d = AtomDevice(wl)
    log(f"case atoms5000_bf16 k={k} rows 1500..2199")
    ref = d.oracle_rows(np.arange(wl.n_q))
    got = d.attention(2).cpu().numpy()
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= 1e-2


def test_f32_gathered_and_k256():
    wl = atom_workload("atoms200_f32", k=256)
    d = AtomDevice(wl, affine=True)
    ref = d.oracle_rows(np.arange(wl.n_q))
    got = d.attention(3, p=d.gathered_p(), p_gathered=1).cpu().numpy()
    err = rel_err(got, ref)
    log(f"  atoms200_f32 k=256 gathered rel err {err:.3e}")
    assert err <= 1e-5
