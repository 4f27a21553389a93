"""The whole-assembly workload at full size (N = 24000, bf16 z = 147 GB) in the
launch configuration bench.py times (6 key blocks), checked on sampled rows
against the fp64 oracle, plus full-size properties (GPU)."""
import numpy as np
import pytest

from gpu_helpers import DCP_BF16, DCP_F32, Device, log, rel_err, sample_rows, workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def big():
    import torch
    assert torch.cuda.is_available()
    wl = workload("asm24000_bf16")
    log("allocating and generating z for asm24000_bf16 (147 GB)")
    d = Device(wl)
    yield d
    del d
    torch.cuda.empty_cache()


def test_asm24000_sampled_rows(big):
    wl = big.wl
    log("case asm24000_bf16 n_kb=6 bf16 out (the benchmark's call), sampled rows")
    got = big.attention(0, wl.n_tok, wl.n_key_blocks, out_dtype=DCP_BF16).float().cpu().numpy()
    rows = sample_rows(wl.n_tok, wl.stripes, wl.n_key_blocks, 96, big.mask_host)
    ref = big.oracle_rows(rows)
    err = rel_err(got[rows], ref)
    log(f"  {len(rows)} rows rel err {err:.3e}")
    assert err <= 1e-2


def test_asm24000_blocked_and_deterministic(big):
    import torch
    wl = big.wl
    log("case asm24000_bf16 fp32 out: n_kb=6 twice, n_kb=1")
    a = big.attention(0, wl.n_tok, wl.n_key_blocks)
    b = big.attention(0, wl.n_tok, wl.n_key_blocks)
    assert torch.equal(a, b)
    c = big.attention(0, wl.n_tok, 1)
    err = rel_err(c.cpu().numpy(), a.cpu().numpy())
    log(f"  blocked vs unblocked rel diff {err:.3e}")
    assert err <= 1e-6
    # padding (masked) query rows still produce outputs; masked keys are never used
    assert torch.isfinite(a).all()


@pytest.mark.parametrize("r0", [0, 11990, 23980])
def test_asm24000_bias_project_full_rows(big, r0):
    """dcp_bias_project over whole rows of the 147 GB tensor (all 24000 columns,
    the last rows masked padding tokens, which the bias does not skip) against
    the oracle."""
    import torch
    import oracle
    import paper_2607_05439_amd as dcp
    import synth
    wl = big.wl
    nr, nc = 20, wl.n_tok
    log(f"case asm24000_bf16 bias_project rows {r0}..{r0 + nr - 1} x {nc} columns")
    out = torch.empty((nr, nc, wl.n_heads), dtype=torch.float32, device="cuda")
    dcp.dcp_bias_project(big.shape(), big.weights(), big.z[r0].data_ptr(), nr, nc, nc * wl.c_z, out)
    z_host = synth.z_host(wl, range(r0, r0 + nr))
    w = big.w_host
    ref = oracle.bias(np.ascontiguousarray(z_host), w["w_b"], w["b_b"], w["ln_gamma"], w["ln_beta"], 1e-5)
    err = rel_err(out.cpu().numpy(), ref)
    log(f"  rel err {err:.3e}")
    assert err <= 1e-4


@pytest.mark.parametrize("q_row0,n_q", [(0, 16384), (7000, 16400)])
def test_asm24000_stripes_numbered_per_xcd(big, q_row0, n_q):
    """Stripes of 256 and 257 row groups of 64: the smallest for which the
    attention numbers its workgroups per XCD, and one that leaves XCD 0 one row
    group more than the others. Against the whole-layer call (fp32 out, 1e-6:
    the stripe's own segment count may differ) and the fp64 oracle (1e-2, bf16
    inputs) on the first and last rows of the stripe and of its last row
    groups."""
    wl = big.wl
    log(f"case asm24000_bf16 stripe q_row0={q_row0} n_q={n_q} n_kb={wl.n_key_blocks} (per-XCD numbering)")
    full = big.attention(0, wl.n_tok, wl.n_key_blocks).cpu().numpy()
    got = big.attention(q_row0, n_q, wl.n_key_blocks).cpu().numpy()
    err = rel_err(got, full[q_row0:q_row0 + n_q])
    log(f"  stripe vs whole layer rel diff {err:.3e}")
    assert err <= 1e-6
    local = [0, 1, 63, 64, n_q - 129, n_q - 65, n_q - 64, n_q - 17, n_q - 1]
    ref = big.oracle_rows([q_row0 + r for r in local])
    err = rel_err(got[local], ref)
    log(f"  {len(local)} rows against the oracle rel err {err:.3e}")
    assert err <= 1e-2
