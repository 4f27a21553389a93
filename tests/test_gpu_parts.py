"""dcp_bias_project and dcp_block_merge against the oracle, and the device
input generator against its host twin (GPU)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import DCP_BF16, DCP_F32, Device, log, rel_err, workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available()
    return torch


@pytest.mark.parametrize("dtype,c_z,h,tol", [("bf16", 128, 16, 1e-4), ("f32", 32, 4, 1e-5), ("bf16", 48, 3, 1e-5)])
def test_bias_project(torch_cuda, dtype, c_z, h, tol):
    import paper_2607_05439_amd as dcp
    log(f"case bias_project {dtype} c_z={c_z} H={h}")
    wl = workload(n_tok=70, c_z=c_z, n_heads=h, head_dim=8, c_s=32, dtype=dtype)
    d = Device(wl, affine=True)
    r0, c0, nr, nc = 3, 5, 37, 61  # a tile of the full z
    tile = d.z[r0:r0 + nr, c0:c0 + nc]
    out = torch_cuda.empty((nr, nc, h), dtype=torch_cuda.float32, device="cuda")
    dcp.dcp_bias_project(d.shape(), d.weights(), tile.data_ptr(), nr, nc, wl.n_tok * c_z, out)
    z_host = synth.z_host(wl, range(r0, r0 + nr))[:, c0:c0 + nc]
    w = d.w_host
    ref = oracle.bias(np.ascontiguousarray(z_host), w["w_b"], w["b_b"], w["ln_gamma"], w["ln_beta"], 1e-5)
    err = rel_err(out.cpu().numpy(), ref)
    log(f"  rel err {err:.3e}")
    assert err <= tol


def test_bias_project_column_chunks(torch_cuda):
    """The fused bias kernel: workgroups of 64 rows (here one full group and a
    partial one) over column chunks (131 columns: 9 chunks, a short last one)."""
    import paper_2607_05439_amd as dcp
    log("case bias_project bf16 c_z=128 H=16, 75 rows x 131 columns")
    wl = workload(n_tok=200, c_z=128, n_heads=16, head_dim=24, c_s=384, dtype="bf16")
    d = Device(wl, affine=True)
    r0, c0, nr, nc = 7, 60, 75, 131
    tile = d.z[r0:r0 + nr, c0:c0 + nc]
    out = torch_cuda.empty((nr, nc, 16), dtype=torch_cuda.float32, device="cuda")
    dcp.dcp_bias_project(d.shape(), d.weights(), tile.data_ptr(), nr, nc, wl.n_tok * 128, out)
    z_host = synth.z_host(wl, range(r0, r0 + nr))[:, c0:c0 + nc]
    w = d.w_host
    ref = oracle.bias(np.ascontiguousarray(z_host), w["w_b"], w["b_b"], w["ln_gamma"], w["ln_beta"], 1e-5)
    err = rel_err(out.cpu().numpy(), ref)
    log(f"  rel err {err:.3e}")
    assert err <= 1e-4


def test_bias_project_long_row_stride(torch_cuda):
    """Row strides too long for 32-bit offsets over 16 rows take the
    register-load kernel; it gives the same bits as the LDS-ring kernel on the
    same pairs (17 rows 2^26 elements apart: a 2.3 GB allocation)."""
    import paper_2607_05439_amd as dcp
    log("case bias_project bf16, row stride 2^26 elements (fallback kernel) vs contiguous")
    wl = workload(n_tok=40, c_z=128, n_heads=16, head_dim=24, c_s=384, dtype="bf16")
    d = Device(wl, affine=True)
    nr, nc = 17, 40
    stride = 1 << 26
    big = torch_cuda.empty(nr * stride, dtype=torch_cuda.bfloat16, device="cuda")
    rows = big.view(nr, stride)[:, :nc * 128]
    rows.copy_(d.z[:nr].reshape(nr, nc * 128))
    got = torch_cuda.empty((nr, nc, 16), dtype=torch_cuda.float32, device="cuda")
    ref = torch_cuda.empty((nr, nc, 16), dtype=torch_cuda.float32, device="cuda")
    dcp.dcp_bias_project(d.shape(), d.weights(), big.data_ptr(), nr, nc, stride, got)
    dcp.dcp_bias_project(d.shape(), d.weights(), d.z.data_ptr(), nr, nc, nc * 128, ref)
    torch_cuda.cuda.synchronize()
    del big, rows
    assert torch_cuda.equal(got, ref)


@pytest.mark.parametrize("D", [6, 8, 24])
def test_block_merge(torch_cuda, D):
    """Head sizes 6 (one channel per thread) and 8, 24 (four channels of a
    head per thread)."""
    import paper_2607_05439_amd as dcp
    log(f"case block_merge D={D}")
    r = np.random.default_rng(5)
    P, R, H = 5, 33, 4
    m = (3 * r.standard_normal((P, H, R))).astype(np.float32)
    m[1, :, ::3] = -np.inf
    m[:, 0, 7] = -np.inf  # a fully empty (row, head)
    l = (r.random((P, H, R)) + 0.5).astype(np.float32)
    l[np.isneginf(m)] = 0
    acc = r.standard_normal((P, R, H, D)).astype(np.float32)
    acc[np.isneginf(m).transpose(0, 2, 1)] = 0
    gate = r.random((R, H * D)).astype(np.float32)
    T = lambda a: torch_cuda.from_numpy(np.ascontiguousarray(a)).cuda()
    mo = torch_cuda.empty((H, R), device="cuda")
    lo = torch_cuda.empty((H, R), device="cuda")
    ao = torch_cuda.empty((R, H, D), device="cuda")
    out = torch_cuda.empty((R, H * D), device="cuda")
    dcp.dcp_block_merge(P, R, H, D, T(m), T(l), T(acc), mo, lo, ao, T(gate), out, DCP_F32)
    m_ref, l_ref, a_ref, o_ref = oracle.merge(m, l, acc, gate)
    assert np.array_equal(mo.cpu().numpy(), m_ref.astype(np.float32))
    assert rel_err(lo.cpu().numpy(), l_ref) <= 1e-6
    assert rel_err(ao.cpu().numpy(), a_ref) <= 1e-6
    assert rel_err(out.cpu().numpy(), o_ref) <= 1e-6
    assert np.all(out.cpu().numpy()[7, 0:D] == 0.0)
    out_bf = torch_cuda.empty((R, H * D), dtype=torch_cuda.bfloat16, device="cuda")
    dcp.dcp_block_merge(P, R, H, D, T(m), T(l), T(acc), None, None, None, None, out_bf, DCP_BF16)
    _, _, _, o_nogate = oracle.merge(m, l, acc, None)
    assert rel_err(out_bf.float().cpu().numpy(), o_nogate) <= 1e-2


@pytest.mark.parametrize("period,bf16", [(0, True), (80, True), (0, False), (7, False)])
def test_device_generator_matches_host(torch_cuda, period, bf16):
    log(f"case device generator period={period} bf16={bf16}")
    wl = workload(n_tok=90, c_z=32, dtype="bf16" if bf16 else "f32", z_period=period)
    rows = [0, 1, 45, 89]
    dt = torch_cuda.bfloat16 if bf16 else torch_cuda.float32
    z = torch_cuda.empty((90, 90, 32), dtype=dt, device="cuda")
    synth.z_fill_device(wl, z.data_ptr(), 0, 90, torch_cuda.cuda.current_stream().cuda_stream)
    host = synth.z_host(wl, rows)
    dev = z[rows].cpu()
    dev = dev.view(torch_cuda.int16).numpy().view(np.uint16) if bf16 else dev.numpy()
    assert np.array_equal(dev.view(np.uint8), host.view(np.uint8))


def test_block_merge_forms_agree_bit_for_bit(torch_cuda):
    """The same merge through the four-channel kernel (16-byte aligned
    buffers) and through the one-channel kernel (buffers one element off
    alignment): identical bits, with and without the gate, fp32 and bf16."""
    import paper_2607_05439_amd as dcp
    r = np.random.default_rng(8)
    P, R, H, D = 6, 257, 16, 24
    m = np.floor(8 * r.standard_normal((P, H, R))).astype(np.float32)
    m[2, :, ::5] = -np.inf
    l = (r.random((P, H, R)) + 0.5).astype(np.float32)
    l[np.isneginf(m)] = 0
    acc = r.standard_normal((P, R, H, D)).astype(np.float32)
    gate = r.random((R, H * D)).astype(np.float32)

    def dev_at(a, shift):  # device copy whose data starts `shift` floats into a fresh buffer
        flat = torch_cuda.zeros(a.size + 4, dtype=torch_cuda.float32, device="cuda")
        flat[shift:shift + a.size] = torch_cuda.from_numpy(np.ascontiguousarray(a).ravel()).cuda()
        return flat[shift:shift + a.size].view(a.shape)

    for with_gate in (True, False):
        outs = []
        for shift in (0, 1):
            for dt in (DCP_F32, DCP_BF16):
                o = torch_cuda.zeros(R * H * D + 8, dtype=torch_cuda.float32 if dt == DCP_F32 else torch_cuda.bfloat16,
                                     device="cuda")[shift:shift + R * H * D].view(R, H * D)
                ao = dev_at(np.zeros((R, H, D), np.float32), shift)
                dcp.dcp_block_merge(P, R, H, D, dev_at(m, shift), dev_at(l, shift), dev_at(acc, shift), None, None,
                                    ao, dev_at(gate, shift) if with_gate else None, o, dt)
                outs.append((o.float().cpu().numpy(), ao.cpu().numpy()))
        for i in range(2):  # fp32 and bf16 outputs: aligned against shifted
            assert np.array_equal(outs[i][0], outs[2 + i][0])
            assert np.array_equal(outs[i][1], outs[2 + i][1])
