"""Pair transition (LayerNorm + SwiGLU + residual) on the GPU against the fp64
oracle, through the C-ABI (GPU)."""
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


def run(z, w, dtype, n_pairs=None, in_place=False, eps=1e-5):
    """dcp_pair_transition on device tensor z (flattened pairs); returns the output tensor."""
    import torch
    import paper_2607_05439_amd as dcp
    c_z = z.shape[-1]
    hidden = w["w1"].shape[0]
    n = z.numel() // c_z if n_pairs is None else n_pairs
    ws_bytes = dcp.dcp_transition_workspace_size(c_z, hidden, dtype)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda:0")
    out = z if in_place else torch.empty_like(z)
    W = {k: (None if v is None else dev(v)) for k, v in w.items()}
    dcp.dcp_pair_transition(n, c_z, hidden, dtype, eps, W["w1"], W["w2"], W["w3"], W["gamma"], W["beta"], z, out,
                            ws, ws.numel())
    return out


def host_f64(t):
    import torch
    return t.float().cpu().numpy().astype(np.float64)


def test_f32_whole_output():
    wl, hidden = synth.transition_workload("trans40_f32")
    z = synth.z_host(wl, range(wl.n_tok))  # [40, 40, 32] fp32
    for affine in (False, True):
        w = synth.transition_weights(wl, hidden, affine=affine)
        ref = oracle.transition(z, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
        zt = dev(z)
        got = host_f64(run(zt, w, DCP_F32))
        err = rel_err(got, ref)
        log(f"case trans40_f32 affine={affine}: rel err {err:.3e}")
        assert err <= 1e-5
        inplace = run(zt, w, DCP_F32, in_place=True)
        assert np.array_equal(host_f64(inplace), got)


def test_bf16_whole_output():
    wl, hidden = synth.transition_workload("trans192_bf16")
    z = synth.z_host(wl, range(wl.n_tok))  # [192, 192, 128] bf16 bits
    for affine in (False, True):
        w = synth.transition_weights(wl, hidden, affine=affine)
        ref = oracle.transition(z, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
        got = host_f64(run(dev(z), w, DCP_BF16))
        err = rel_err(got, ref)
        log(f"case trans192_bf16 affine={affine}: rel err {err:.3e}")
        assert err <= 1e-2


def test_bf16_ragged_inplace_deterministic():
    """Pair counts that are not a multiple of the 256-pair group, in place
    against out of place, repeated calls, and pairs past n_pairs untouched."""
    import torch
    wl, hidden = synth.transition_workload("trans192_bf16")
    z = synth.z_host(wl, range(8))  # 8 rows x 192 pairs
    w = synth.transition_weights(wl, hidden, affine=True)
    flat = z.reshape(-1, 128)
    for n in (1, 255, 257, 1000, len(flat)):
        ref = oracle.transition(flat[:n], w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
        zt = dev(flat)
        a = run(zt, w, DCP_BF16, n_pairs=n)
        b = run(zt, w, DCP_BF16, n_pairs=n)
        assert torch.equal(a[:n], b[:n])
        err = rel_err(host_f64(a[:n]), ref)
        assert err <= 1e-2, (n, err)
        zc = zt.clone()
        run(zc, w, DCP_BF16, n_pairs=n, in_place=True)
        assert torch.equal(zc[:n], a[:n])
        assert torch.equal(zc[n:], zt[n:])
    run(dev(flat), w, DCP_BF16, n_pairs=0)


def test_bf16_full_size_in_place_sampled():
    """The 24000-token pair tensor (147 GB, bf16) updated in place in one call,
    as the benchmark does; sampled pairs against the oracle on the generator's
    host copy of the same values."""
    import torch
    wl, hidden = synth.transition_workload("trans24000_bf16")
    n = wl.n_tok
    log("allocating and generating z for asm24000_bf16 (147 GB)")
    z = torch.empty((n, n, 128), dtype=torch.bfloat16, device="cuda:0")
    synth.z_fill_device(wl, z.data_ptr(), 0, n, torch.cuda.current_stream().cuda_stream)
    w = synth.transition_weights(wl, hidden)
    log("case trans24000_bf16 in place")
    run(z, w, DCP_BF16, in_place=True)
    rng = np.random.default_rng(0)
    rows = [0, 1, 12345, n - 1]
    cols = np.concatenate([[0, 1, 255, 256, n - 1], rng.choice(n, 300, replace=False)])
    zh = synth.z_host(wl, rows)[:, cols]  # [4, len(cols), 128]
    ref = oracle.transition(zh, w["w1"], w["w2"], w["w3"])
    got = host_f64(z[rows][:, torch.from_numpy(cols).to("cuda:0")])
    err = rel_err(got, ref)
    log(f"  {zh.shape[0] * zh.shape[1]} pairs rel err {err:.3e}")
    assert err <= 1e-2
    del z
    torch.cuda.empty_cache()
