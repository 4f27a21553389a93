"""dcp_pair_bias_attention through the C-ABI against the fp64 oracle (GPU).

Tolerances (max|err| / max|ref|): 1e-5 for fp32 inputs, 1e-2 for bf16 inputs,
1e-6 between blocked and unblocked GPU results with fp32 output.
"""
import numpy as np
import pytest

from gpu_helpers import DCP_BF16, DCP_F32, Device, log, rel_err, sample_rows, workload

pytestmark = pytest.mark.gpu

TOL_F32, TOL_BF16, TOL_BLOCKED = 1e-5, 1e-2, 1e-6


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _np(t):
    return t.float().cpu().numpy().astype(np.float64)


# ----------------------------------------------------------------------------- tiny fp32 (general path)
def test_tiny128_f32_parity(torch_cuda):
    log("case tiny128_f32 n_kb=1")
    d = Device(workload("tiny128_f32"))
    rows = np.arange(128)
    ref = d.oracle_rows(rows)
    got = _np(d.attention(0, 128, 1))
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= TOL_F32


def test_tiny128_f32_blocked(torch_cuda):
    log("case tiny128_f32 n_kb=4 vs 1")
    d = Device(workload("tiny128_f32"))
    a = _np(d.attention(0, 128, 1))
    b = _np(d.attention(0, 128, 4))
    assert rel_err(b, a) <= TOL_BLOCKED
    assert rel_err(b, d.oracle_rows(np.arange(128), n_blocks=4)) <= TOL_F32


def test_general_path_bf16_inputs(torch_cuda):
    log("case general path, bf16 inputs, c_z=64 H=4 d=16, masked, stripe")
    wl = workload(n_tok=50, c_s=40, c_z=64, n_heads=4, head_dim=16, dtype="bf16", mask="random:7")
    d = Device(wl)
    got = _np(d.attention(3, 40, 3))
    ref = d.oracle_rows(np.arange(3, 43))
    assert rel_err(got, ref) <= TOL_F32


# ----------------------------------------------------------------------------- fused bf16 path
def test_pad1024_parity(torch_cuda):
    log("case pad1024_bf16 n_kb=4 f32 out")
    d = Device(workload("pad1024_bf16"))
    ref = d.oracle_rows(np.arange(1024))
    got = _np(d.attention(0, 1024, 4))
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= TOL_BF16
    got_bf = _np(d.attention(0, 1024, 4, out_dtype=DCP_BF16))
    assert rel_err(got_bf, ref) <= TOL_BF16


def test_pad1024_blocked_vs_unblocked(torch_cuda):
    log("case pad1024_bf16 blocked vs unblocked")
    d = Device(workload("pad1024_bf16"))
    a = _np(d.attention(0, 1024, 1))
    for nb in (4, 7, 64):
        b = _np(d.attention(0, 1024, nb))
        err = rel_err(b, a)
        log(f"  n_kb={nb} rel diff {err:.3e}")
        assert err <= TOL_BLOCKED


def test_deterministic(torch_cuda):
    log("case pad1024_bf16 repeat")
    d = Device(workload("pad1024_bf16"))
    a = d.attention(0, 1024, 4)
    b = d.attention(0, 1024, 4)
    assert torch_cuda.equal(a, b)


def test_masked_keys_never_read(torch_cuda):
    log("case pad1024_bf16 masked z perturbed")
    d = Device(workload("pad1024_bf16"))
    a = d.attention(0, 1024, 4)
    masked = np.flatnonzero(d.mask_host == 0)
    z2 = d.z.clone()
    z2[:, masked, :] = 1000.0
    b = d.attention(0, 1024, 4, z=z2)
    assert torch_cuda.equal(a, b)


def test_affine_constants_irrelevant(torch_cuda):
    log("case beta and b_b change nothing")
    wl = workload(n_tok=96, mask="tail:5")
    d = Device(wl, affine=True)
    a = _np(d.attention(0, 96, 2))
    b = _np(d.attention(0, 96, 2, drop_affine=True))
    assert rel_err(a, b) <= TOL_BLOCKED
    assert rel_err(a, d.oracle_rows(np.arange(96))) <= TOL_BF16


@pytest.mark.parametrize("n_tok,q_row0,n_q,n_kb,mask", [
    (1, 0, 1, 1, "none"),
    (5, 1, 3, 2, "none"),
    (16, 0, 16, 1, "none"),
    (17, 0, 17, 17, "tail:1"),
    (37, 5, 19, 3, "random:6"),
    (100, 60, 40, 5, "random:30"),
    (333, 0, 333, 2, "tail:13"),
    # one workgroup of query rows over many keys: the launch splits the keys into
    # many short parts whose bounds do not fall on 16-key tiles (32 parts of 64
    # keys; 7 parts of 71-72 keys per block)
    (2048, 100, 50, 1, "random:200"),
    (1500, 0, 64, 3, "tail:7"),
])
def test_ragged_and_small(torch_cuda, n_tok, q_row0, n_q, n_kb, mask):
    log(f"case ragged N={n_tok} q_row0={q_row0} n_q={n_q} n_kb={n_kb} mask={mask}")
    d = Device(workload(n_tok=n_tok, mask=mask))
    got = _np(d.attention(q_row0, n_q, n_kb))[:n_q]
    ref = d.oracle_rows(np.arange(q_row0, q_row0 + n_q))
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= TOL_BF16


def test_all_keys_masked_gives_zero(torch_cuda):
    log("case all keys masked")
    wl = workload(n_tok=40)
    d = Device(wl, mask=np.zeros(40, np.uint8))
    out = d.attention(0, 40, 3)
    assert torch_cuda.count_nonzero(out).item() == 0
    wl32 = workload(n_tok=20, c_s=16, c_z=8, n_heads=2, head_dim=4, dtype="f32")
    d32 = Device(wl32, mask=np.zeros(20, np.uint8))
    assert torch_cuda.count_nonzero(d32.attention(0, 20, 2)).item() == 0


def test_one_block_entirely_masked(torch_cuda):
    log("case a whole key block masked")
    m = np.ones(200, np.uint8)
    m[50:100] = 0  # block 1 of 4
    d = Device(workload(n_tok=200), mask=m)
    got = _np(d.attention(0, 200, 4))
    assert rel_err(got, d.oracle_rows(np.arange(200))) <= TOL_BF16
    assert rel_err(got, _np(d.attention(0, 200, 1))) <= TOL_BLOCKED


def test_n_q_zero_is_noop(torch_cuda):
    import paper_2607_05439_amd as dcp
    d = Device(workload(n_tok=32))
    shape = d.shape()
    assert dcp.dcp_workspace_size(shape, 0, 1) == 0
    out = torch_cuda.full((1, 384), 7.0, device="cuda")
    dcp.dcp_pair_bias_attention(shape, d.weights(), d.s, d.z, None, 32, 0, 1, out, None, 0, None)
    torch_cuda.cuda.synchronize()
    assert torch_cuda.all(out == 7.0)


# ----------------------------------------------------------------------------- larger workloads, sampled rows
def test_ico4800_sampled(torch_cuda):
    wl = workload("ico4800_bf16")
    log("case ico4800_bf16 n_kb=10 sampled rows")
    d = Device(wl)
    got = _np(d.attention(0, wl.n_tok, wl.n_key_blocks))
    rows = sample_rows(wl.n_tok, wl.stripes, wl.n_key_blocks, 96, d.mask_host)
    err = rel_err(got[rows], d.oracle_rows(rows))
    log(f"  {len(rows)} rows rel err {err:.3e}")
    assert err <= TOL_BF16


def test_grid12000_stripes_sampled(torch_cuda):
    wl = workload("grid12000_bf16")
    log("case grid12000_bf16 4 stripes x 4 key blocks, sampled rows")
    d = Device(wl)
    for q0, nq in wl.stripes:
        got = _np(d.attention(q0, nq, wl.n_key_blocks))
        rows = sample_rows(wl.n_tok, [(q0, nq)], 1, 24, None, seed=q0)
        rows = [r for r in rows if q0 <= r < q0 + nq]
        err = rel_err(got[np.array(rows) - q0], d.oracle_rows(rows))
        log(f"  stripe {q0}: {len(rows)} rows rel err {err:.3e}")
        assert err <= TOL_BF16
