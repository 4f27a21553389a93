"""Numerical-equivalence checks of the fused path through the C-ABI (GPU).

The paper keeps the sharded computation numerically equivalent to the
single-GPU one (Introduction; Methods, "2D grid context parallelism"): here
that means (1) the key-blocked result equals the unblocked one at the
workloads whose launches split blocks differently (the 4800-token layer's 10
blocks, a 12000-token stripe's 4 blocks each cut into segments), (2) the
fused LayerNorm holds for pair vectors whose channel mean is large against
their spread, or whose scale is far from 1 (Methods, "RFDiffusion 3
preliminaries and notation": the bias is a learned projection of Z, read as
Linear(LayerNorm(z))), and (3) renumbering the tokens (s, z and the mask
together) renumbers the output rows and changes nothing else.

Tolerances (max|err| / max|ref|): 1e-6 blocked vs unblocked and 1e-5 for
the permutation (both fp32 output, the same kernels on reordered work);
1e-2 for bf16 inputs against the fp64 oracle; 1e-4 for the materialised bias.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import AtomDevice, DCP_F32, Device, atom_workload, log, rel_err, sample_rows, workload

pytestmark = pytest.mark.gpu

TOL_BLOCKED, TOL_PERM, TOL_BF16, TOL_BIAS = 1e-6, 1e-5, 1e-2, 1e-4


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _np(t):
    return t.float().cpu().numpy().astype(np.float64)


# ----------------------------------------------------------------------------- blocked = unblocked
def test_ico4800_blocked_vs_unblocked(torch_cuda):
    wl = workload("ico4800_bf16")
    log(f"case ico4800_bf16 fp32 out: n_kb={wl.n_key_blocks} vs 1")
    d = Device(wl)
    a = _np(d.attention(0, wl.n_tok, 1))
    b = _np(d.attention(0, wl.n_tok, wl.n_key_blocks))
    err = rel_err(b, a)
    log(f"  rel diff {err:.3e}")
    assert err <= TOL_BLOCKED
    rows = sample_rows(wl.n_tok, wl.stripes, wl.n_key_blocks, 24, d.mask_host, seed=3)
    assert rel_err(b[rows], d.oracle_rows(rows)) <= TOL_BF16


def test_grid12000_stripe_blocked_vs_unblocked(torch_cuda):
    wl = workload("grid12000_bf16")
    q0, nq = wl.stripes[1]
    log(f"case grid12000_bf16 stripe {q0}+{nq} fp32 out: n_kb={wl.n_key_blocks} vs 1")
    d = Device(wl)
    a = _np(d.attention(q0, nq, 1))
    b = _np(d.attention(q0, nq, wl.n_key_blocks))
    err = rel_err(b, a)
    log(f"  rel diff {err:.3e}")
    assert err <= TOL_BLOCKED
    rows = [q0, q0 + 1, q0 + nq // 2, q0 + nq - 1]
    assert rel_err(b[np.array(rows) - q0], d.oracle_rows(rows)) <= TOL_BF16


# ----------------------------------------------------------------------------- LayerNorm: shifted and scaled z
def _transformed_z(wl, alpha: float, shift: float) -> np.ndarray:
    """bf16(alpha * z + shift) on the host, from the generator's own z."""
    z = synth.bf16_to_f32(synth.z_host(wl, range(wl.n_tok)))
    z = (z * np.float32(alpha)).astype(np.float32)
    z = (z + np.float32(shift)).astype(np.float32)
    return synth.bf16_round(z)


LN_CASES = [(1.0, 4.0), (1.0, 16.0), (1.0, 64.0), (0.01, 0.0), (30.0, 0.0), (30.0, 64.0)]


@pytest.mark.parametrize("alpha,shift", LN_CASES)
def test_layernorm_shift_scale_attention(torch_cuda, alpha, shift):
    wl = workload(n_tok=300, mask="random:20")
    log(f"case fused attention on bf16({alpha} z + {shift}), N=300, 3 key blocks, stripe 7+290")
    d = Device(wl, affine=True, z_override=_transformed_z(wl, alpha, shift))
    got = _np(d.attention(7, 290, 3))
    ref = d.oracle_rows(np.arange(7, 297))
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= TOL_BF16
    # the same keys in one block: the blocked weights do not depend on the offset either
    assert rel_err(_np(d.attention(7, 290, 1)), got) <= TOL_BLOCKED


@pytest.mark.parametrize("alpha,shift", LN_CASES)
def test_layernorm_shift_scale_bias_project(torch_cuda, alpha, shift):
    import paper_2607_05439_amd as dcp
    wl = workload(n_tok=150)
    log(f"case bias_project on bf16({alpha} z + {shift}), 150 x 150 pairs")
    zt = _transformed_z(wl, alpha, shift)
    d = Device(wl, affine=True, z_override=zt)
    out = torch_cuda.empty((150, 150, 16), dtype=torch_cuda.float32, device="cuda")
    dcp.dcp_bias_project(d.shape(), d.weights(), d.z, 150, 150, 150 * 128, out)
    w = d.w_host
    ref = oracle.bias(np.ascontiguousarray(zt), w["w_b"], w["b_b"], w["ln_gamma"], w["ln_beta"], 1e-5)
    err = rel_err(out.cpu().numpy(), ref)
    log(f"  rel err {err:.3e}")
    assert err <= TOL_BIAS


@pytest.mark.parametrize("alpha,shift", [(1.0, 64.0), (0.01, 0.0), (30.0, 16.0)])
def test_layernorm_shift_scale_sparse(torch_cuda, alpha, shift):
    """The sparse atom attention's fused LayerNorm over the 16 atom-pair
    channels on shifted and scaled pair slices (gathered form)."""
    wl = atom_workload("atoms5000_bf16")
    log(f"case sparse atom attention on bf16({alpha} p + {shift}), atoms5000 gathered slices")
    d = AtomDevice(wl, affine=True)
    rows = np.arange(wl.n_q)
    pg = synth.bf16_to_f32(synth.p_gathered_host(wl, wl.q_row0 + rows, d.nbr_host))
    pg = ((pg * np.float32(alpha)).astype(np.float32) + np.float32(shift)).astype(np.float32)
    pg = synth.bf16_round(pg)
    got = _np(d.attention(wl.n_key_blocks, p=d._to_dev(pg), p_gathered=1))
    check = np.unique(np.concatenate([np.arange(0, wl.n_q, max(1, wl.n_q // 200)), [wl.n_q - 1]]))
    ref = oracle.sparse_attention(d.a_host, np.ascontiguousarray(pg[check]), d.nbr_host[check], wl.q_row0 + check,
                                  d.w_host, wl.n_heads, wl.head_dim, n_blocks=wl.n_key_blocks)
    err = rel_err(got[check], ref)
    log(f"  {len(check)} rows rel err {err:.3e}")
    assert err <= TOL_BF16


# ----------------------------------------------------------------------------- token permutation
def test_token_permutation_equivariance(torch_cuda):
    """(s, z, mask) -> (s[pi], z[pi][:, pi], mask[pi]) gives out[pi], on the
    1024-token workload (4 key blocks, 4 masked padding tokens)."""
    import paper_2607_05439_amd as dcp
    torch = torch_cuda
    wl = workload("pad1024_bf16")
    log("case pad1024_bf16 token permutation, fp32 out")
    d = Device(wl)
    n, hd = wl.n_tok, wl.n_heads * wl.head_dim
    base = _np(d.attention(0, n, wl.n_key_blocks))
    pi = np.random.default_rng(11).permutation(n)
    pt = torch.from_numpy(pi).to(d.dev)
    s_p = d.s.index_select(0, pt).contiguous()
    z_p = d.z.index_select(0, pt).index_select(1, pt).contiguous()
    m_p = d.mask.index_select(0, pt).contiguous()
    out = torch.empty((n, hd), dtype=torch.float32, device=d.dev)
    shape = d.shape(DCP_F32)
    nbytes = dcp.dcp_workspace_size(shape, n, wl.n_key_blocks)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=d.dev)
    dcp.dcp_pair_bias_attention(shape, d.weights(), s_p, z_p, m_p, 0, n, wl.n_key_blocks, out, ws, nbytes, None)
    got = _np(out)
    err = rel_err(got, base[pi])
    log(f"  rel diff {err:.3e}")
    assert err <= TOL_PERM
    # and the masked tokens, wherever they land, still give finite outputs
    assert np.isfinite(got).all()


# ----------------------------------------------------------------------------- peaked softmax (large logits)
def _scale_weights(d, q_k: float, b: float):
    """Scale W_q, W_k and W_b by powers of two (exact in fp32) on both sides."""
    import torch
    for name, f in (("w_q", q_k), ("w_k", q_k), ("w_b", b)):
        d.w_host[name] = (d.w_host[name] * np.float32(f)).astype(np.float32)
        d.w[name] = torch.from_numpy(np.ascontiguousarray(d.w_host[name])).to(d.dev)


@pytest.mark.parametrize("dtype,q_k,b,tol", [("bf16", 1.0, 8.0, TOL_BF16), ("f32", 2.0, 8.0, 1e-5)])
def test_peaked_softmax(torch_cuda, dtype, q_k, b, tol):
    """Logits far from the unit-scale workloads' range (the pair bias scaled
    up 8x, to a spread of about +-30 natural units; q and k scaled too on the
    fp32 path): most softmax weights underflow against the row maximum, and
    the running maximum moves by many units between key tiles. (On the bf16
    path q and k stay at unit scale: they enter the matrix cores as bf16, whose
    rounding grows with the logits' size and is part of that path's precision,
    not of its softmax: at 4x larger q.k logits the error against the fp64
    oracle reaches 1.3e-2.)"""
    if dtype == "bf16":
        wl = workload(n_tok=300, mask="random:20")
        q0, nq, nkb = 5, 290, 3
    else:
        wl = workload(n_tok=128, c_s=128, c_z=32, n_heads=4, head_dim=32, dtype="f32", mask="tail:6")
        q0, nq, nkb = 0, 128, 4
    log(f"case peaked softmax {dtype}: W_q, W_k x{q_k}, W_b x{b}")
    d = Device(wl, affine=True)
    _scale_weights(d, q_k, b)
    got = _np(d.attention(q0, nq, nkb))[:nq]
    ref = d.oracle_rows(np.arange(q0, q0 + nq))
    err = rel_err(got, ref)
    log(f"  rel err {err:.3e}")
    assert err <= tol
    assert rel_err(_np(d.attention(q0, nq, 1))[:nq], got) <= (TOL_BLOCKED if dtype == "bf16" else 1e-5)
