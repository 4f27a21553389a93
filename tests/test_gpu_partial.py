"""One ring step through the C-ABI (dcp_pair_bias_attention_partial): the
partial states of key ranges, merged in ring order with dcp_block_merge, give
the full call's output; each range's state matches the oracle's blocked
partial; empty and fully masked ranges give the empty state (GPU)."""
import numpy as np
import pytest

import oracle
from gpu_helpers import DCP_F32, Device, log, rel_err, workload

pytestmark = pytest.mark.gpu


def partial(d, q_row0, n_q, k0, k1):
    import torch
    import paper_2607_05439_amd as dcp
    wl = d.wl
    hd = wl.n_heads * wl.head_dim
    f32 = dict(dtype=torch.float32, device=d.dev)
    m, l = torch.full((wl.n_heads, n_q), 7.0, **f32), torch.full((wl.n_heads, n_q), 7.0, **f32)
    acc, g = torch.full((n_q, hd), 7.0, **f32), torch.full((n_q, hd), 7.0, **f32)
    shape = d.shape(DCP_F32)
    ws = torch.empty(max(dcp.dcp_workspace_size(shape, n_q, 1), 256), dtype=torch.uint8, device=d.dev)
    z_ptr = d.z.data_ptr() + q_row0 * wl.n_tok * wl.c_z * d.z.element_size()
    dcp.dcp_pair_bias_attention_partial(shape, d.weights(), d.s, z_ptr, d.mask, q_row0, n_q, k0, k1, m, l, acc, g,
                                        ws, ws.numel(), None)
    return m, l, acc, g


def ring(d, q_row0, n_q, bounds):
    """Partials of [bounds[i], bounds[i+1]) merged in increasing order."""
    import torch
    import paper_2607_05439_amd as dcp
    wl = d.wl
    hd = wl.n_heads * wl.head_dim
    parts = [partial(d, q_row0, n_q, a, b) for a, b in zip(bounds[:-1], bounds[1:])]
    m = torch.stack([p[0] for p in parts]).contiguous()
    l = torch.stack([p[1] for p in parts]).contiguous()
    acc = torch.stack([p[2] for p in parts]).contiguous()
    out = torch.empty((n_q, hd), dtype=torch.float32, device=d.dev)
    dcp.dcp_block_merge(len(parts), n_q, wl.n_heads, wl.head_dim, m, l, acc, None, None, None, parts[0][3], out,
                        DCP_F32)
    return out.cpu().numpy()


# The exported states are in natural-log units: on the fused path the
# internal base-2 maxima are converted ((m - 192) ln 2, rounded to fp32) and
# the public merge rescales with expf, a few fp32 ulps per part, where the
# internal blocked path rescales by exact powers of two (bar 1e-6).
@pytest.mark.parametrize("name,q_row0,n_q,tol", [("tiny128_f32", 0, 128, 1e-6), ("pad1024_bf16", 100, 200, 1e-5)])
def test_ring_of_partials_equals_the_full_call(name, q_row0, n_q, tol):
    d = Device(workload(name))
    n = d.wl.n_tok
    full = d.attention(q_row0, n_q, 1).cpu().numpy()
    for bounds in ([0, n], [0, 37, 37, 300 if n > 300 else n // 2, n], [0, 1, n - 1, n]):
        got = ring(d, q_row0, n_q, bounds)
        err = rel_err(got, full)
        log(f"case {name} rows {q_row0}+{n_q} ring {bounds}: rel err vs full call {err:.3e}")
        assert err <= tol


@pytest.mark.parametrize("name,tol", [("tiny128_f32", 1e-5), ("pad1024_bf16", 1e-2)])
def test_partials_match_the_oracle_blocks(name, tol):
    d = Device(workload(name))
    wl = d.wl
    n, nb = wl.n_tok, 4
    rows = list(range(0, n, max(1, n // 24)))[:24]
    _, (om, ol, oacc) = oracle.attention(d.s_host, __import__("synth").z_host(wl, rows), rows, d.mask_host,
                                          d.w_host, wl.n_heads, wl.head_dim, n_blocks=nb, return_parts=True)
    for b in range(nb):
        size, start = oracle.chunk(n, nb, b)
        got = [t.cpu().numpy() for t in partial(d, 0, n, start, start + size)[:3]]
        gm, gl, gacc = got[0][:, rows], got[1][:, rows], got[2][rows].reshape(len(rows), wl.n_heads, wl.head_dim)
        # what a state means, independent of its reference point m: the
        # log-sum-exp m + log l and the normalised sum acc / l
        lse_ref = om[b] + np.log(ol[b])
        lse_got = gm.astype(np.float64) + np.log(gl.astype(np.float64))
        out_ref = oacc[b] / ol[b].T[:, :, None]
        out_got = gacc / gl.T[:, :, None]
        e1 = float(np.max(np.abs(lse_got - lse_ref)) / max(1.0, np.max(np.abs(lse_ref))))
        e2 = rel_err(out_got, out_ref)
        log(f"case {name} block {b} [{start}, {start + size}): log-sum-exp err {e1:.3e}, normalised acc err {e2:.3e}")
        assert e1 <= tol and e2 <= tol


def test_empty_and_fully_masked_ranges_give_the_empty_state():
    d = Device(workload("pad1024_bf16"))  # the last 4 tokens are masked
    for k0, k1 in ((500, 500), (1020, 1024)):
        m, l, acc, g = (t.cpu().numpy() for t in partial(d, 0, 64, k0, k1))
        log(f"case empty range [{k0}, {k1})")
        assert np.all(np.isneginf(m)) and np.all(l == 0.0) and np.all(acc == 0.0)
        assert np.all(np.isfinite(g)) and np.all((g > 0) & (g < 1))
