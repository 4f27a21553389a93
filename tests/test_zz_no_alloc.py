"""dcp_pair_bias_attention_noalloc (scratch from the library's static device
array) against dcp_pair_bias_attention (scratch from a workspace) through the
C-ABI (GPU): two calls in a row, the second smaller, each giving the same
bits as the workspace form; then the first again, as the array keeps the
previous call's contents."""
import numpy as np
import pytest

from gpu_helpers import DCP_BF16, DCP_F32, Device, log, rel_err, workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch


def _noalloc(d, q_row0, n_q, n_kb, out_dtype):
    import paper_2607_05439_amd as dcp
    torch = d.torch
    wl = d.wl
    out = torch.empty((n_q, wl.n_heads * wl.head_dim), dtype=torch.float32 if out_dtype == DCP_F32 else torch.bfloat16,
                      device=d.dev)
    z_ptr = d.z.data_ptr() + q_row0 * wl.n_tok * wl.c_z * d.z.element_size()
    dcp.dcp_pair_bias_attention_noalloc(d.shape(out_dtype), d.weights(), d.s, z_ptr, d.mask, q_row0, n_q, n_kb, out)
    return out


def test_noalloc_matches_workspace_form(torch_cuda):
    torch = torch_cuda
    big = Device(workload("pad1024_bf16"))
    small = Device(workload(n_tok=300, mask="random:20"))
    cases = [(big, 0, 1024, 4, DCP_F32), (small, 7, 250, 3, DCP_BF16), (big, 0, 1024, 4, DCP_F32),
             (small, 0, 300, 1, DCP_F32)]
    for d, q0, nq, nkb, odt in cases:
        log(f"case noalloc N={d.wl.n_tok} q_row0={q0} n_q={nq} n_kb={nkb} out={odt}")
        ref = d.attention(q0, nq, nkb, out_dtype=odt)
        got = _noalloc(d, q0, nq, nkb, odt)
        torch.cuda.synchronize()
        assert torch.equal(got, ref[:nq])
        err = rel_err(got.float().cpu().numpy(), d.oracle_rows(np.arange(q0, q0 + nq)))
        log(f"  bit-identical to the workspace form; rel err vs oracle {err:.3e}")
        assert err <= 1e-2
