"""Shared plumbing for the GPU tests: device inputs from the seeded generator,
calls through the C-ABI binding, and the oracle on the same inputs."""
from __future__ import annotations

import dataclasses
import sys
from typing import Optional, Sequence

import numpy as np

import oracle
import synth

DCP_F32, DCP_BF16 = 0, 1


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max |got - ref| / max |ref| (the acceptance metric)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def workload(name: str = "", **kw) -> synth.Workload:
    """A registered workload, or an ad-hoc one with the given fields."""
    if name in synth.WORKLOADS and not kw:
        return synth.WORKLOADS[name]
    base = dict(name=name or "adhoc", n_tok=64, c_s=384, c_z=128, n_heads=16, head_dim=24, dtype="bf16",
                n_key_blocks=1, stripes=((0, 64),), mask="none", z_period=0, seed=0, note="")
    if name in synth.WORKLOADS:
        base.update(dataclasses.asdict(synth.WORKLOADS[name]))
    base.update(kw)
    return synth.Workload(**base)


class Device:
    """Device-resident inputs of one workload."""

    def __init__(self, wl: synth.Workload, affine: bool = False, mask: Optional[np.ndarray] = "default",
                 z_override: Optional[np.ndarray] = None, s_override: Optional[np.ndarray] = None):
        import torch
        self.torch = torch
        self.wl = wl
        self.dev = torch.device("cuda:0")
        self.w_host = synth.weights(wl, affine=affine)
        self.s_host = synth.s_host(wl) if s_override is None else np.ascontiguousarray(s_override)
        self.mask_host = synth.mask_host(wl) if isinstance(mask, str) else mask
        self.s = self._to_dev(self.s_host)
        self.w = {k: (None if v is None else torch.from_numpy(np.ascontiguousarray(v)).to(self.dev))
                  for k, v in self.w_host.items()}
        self.mask = None if self.mask_host is None else torch.from_numpy(self.mask_host).to(self.dev)
        n = wl.n_tok
        self.z_host_override = z_override
        if z_override is not None:
            self.z = self._to_dev(z_override)
        else:
            dt = torch.bfloat16 if wl.bf16 else torch.float32
            self.z = torch.empty((n, n, wl.c_z), dtype=dt, device=self.dev)
            synth.z_fill_device(wl, self.z.data_ptr(), 0, n, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()

    def _to_dev(self, a: np.ndarray):
        torch = self.torch
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(self.dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)

    def shape(self, out_dtype: int = DCP_F32, eps: float = 1e-5):
        import paper_2607_05439_amd as dcp
        wl = self.wl
        return dcp.make_shape(wl.n_tok, wl.c_s, wl.c_z, wl.n_heads, wl.head_dim,
                              DCP_BF16 if wl.bf16 else DCP_F32, out_dtype, eps)

    def weights(self, drop_affine: bool = False):
        import paper_2607_05439_amd as dcp
        w = self.w
        if drop_affine:
            return dcp.make_weights(w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"], None, w["ln_gamma"], None)
        return dcp.make_weights(w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"], w["b_b"], w["ln_gamma"],
                                w["ln_beta"])

    def attention(self, q_row0: int, n_q: int, n_kb: int, out_dtype: int = DCP_F32, drop_affine: bool = False,
                  z=None, mask="default", workspace=None):
        """Run dcp_pair_bias_attention; returns the output as a device tensor."""
        import paper_2607_05439_amd as dcp
        torch = self.torch
        shape = self.shape(out_dtype)
        wl = self.wl
        hd = wl.n_heads * wl.head_dim
        out = torch.empty((max(n_q, 1), hd), dtype=torch.float32 if out_dtype == DCP_F32 else torch.bfloat16,
                          device=self.dev)
        nbytes = dcp.dcp_workspace_size(shape, n_q, n_kb)
        ws = workspace if workspace is not None else torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                                                 device=self.dev)
        zt = self.z if z is None else z
        z_ptr = zt.data_ptr() + q_row0 * wl.n_tok * wl.c_z * zt.element_size()
        m = self.mask if isinstance(mask, str) else mask
        dcp.dcp_pair_bias_attention(shape, self.weights(drop_affine), self.s, z_ptr, m, q_row0, n_q, n_kb, out,
                                    ws, ws.numel(), None)
        return out

    def oracle_rows(self, rows: Sequence[int], n_blocks: int = 1, drop_affine: bool = False) -> np.ndarray:
        """fp64 oracle on the generator's host copy of the same inputs (or on
        the host array the device z was uploaded from)."""
        if self.z_host_override is not None:
            z_rows = np.ascontiguousarray(self.z_host_override[np.asarray(rows, dtype=np.int64)])
        else:
            z_rows = synth.z_host(self.wl, rows)
        w = dict(self.w_host)
        if drop_affine:
            w["b_b"] = None
            w["ln_beta"] = None
        return oracle.attention(self.s_host, z_rows, rows, self.mask_host, w, self.wl.n_heads,
                                self.wl.head_dim, n_blocks=n_blocks)


def sample_rows(n_tok: int, stripes, n_kb: int, n_random: int, mask: Optional[np.ndarray], seed: int = 0):
    """Rows the oracle checks at full size: the first and last row of every
    stripe and key block, some masked (padding) rows, and random rows."""
    rows = set()
    for q0, nq in stripes:
        rows.update({q0, q0 + nq - 1})
    for p in range(n_kb):
        size, start = oracle.chunk(n_tok, n_kb, p)
        rows.update({start, start + size - 1})
    if mask is not None:
        masked = np.flatnonzero(mask == 0)
        if len(masked):
            rows.update(int(x) for x in masked[:: max(1, len(masked) // 8)][:8])
            rows.add(int(masked[-1]))
    r = np.random.default_rng(seed)
    rows.update(int(x) for x in r.choice(n_tok, size=min(n_random, n_tok), replace=False))
    return sorted(rows)


# ----------------------------------------------------------------------------- sparse atom attention
def atom_workload(name: str, **kw) -> synth.AtomWorkload:
    wl = synth.ATOM_WORKLOADS[name]
    return dataclasses.replace(wl, **kw) if kw else wl


class AtomDevice:
    """Device-resident inputs of one atom workload: A, the query stripe's rows
    of P (dense), and the neighbour lists."""

    def __init__(self, wl: synth.AtomWorkload, affine: bool = False):
        import torch
        self.torch = torch
        self.wl = wl
        self.dev = torch.device("cuda:0")
        self.w_host = synth.atom_weights(wl, affine=affine)
        self.a_host = synth.a_host(wl)
        self.a = self._to_dev(self.a_host)
        self.w = {k: (None if v is None else torch.from_numpy(np.ascontiguousarray(v)).to(self.dev))
                  for k, v in self.w_host.items()}
        self.nbr_host = synth.neighbours(wl, wl.q_row0, wl.n_q)
        self.nbr = torch.from_numpy(self.nbr_host).to(self.dev)
        dt = torch.bfloat16 if wl.bf16 else torch.float32
        self.p = torch.empty((wl.n_q, wl.n_atoms, wl.c_ap), dtype=dt, device=self.dev)
        synth.p_fill_device(wl, self.p.data_ptr(), wl.q_row0, wl.n_q, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()

    def _to_dev(self, a: np.ndarray):
        torch = self.torch
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(self.dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)

    def shape(self, out_dtype: int = DCP_F32, p_gathered: int = 0, k: Optional[int] = None, eps: float = 1e-5):
        import paper_2607_05439_amd as dcp
        wl = self.wl
        return dcp.make_sparse_shape(wl.n_atoms, wl.c_atom, wl.c_ap, wl.n_heads, wl.head_dim, k or wl.k,
                                     DCP_BF16 if wl.bf16 else DCP_F32, out_dtype, p_gathered, eps)

    def weights(self, drop_affine: bool = False):
        import paper_2607_05439_amd as dcp
        w = self.w
        if drop_affine:
            return dcp.make_weights(w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"], None, w["ln_gamma"], None)
        return dcp.make_weights(w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"], w["b_b"], w["ln_gamma"],
                                w["ln_beta"])

    def attention(self, n_kb: int, out_dtype: int = DCP_F32, row0: int = 0, n_q: Optional[int] = None, nbr=None,
                  p=None, p_gathered: int = 0, workspace=None):
        """dcp_sparse_pair_bias_attention for stripe rows [row0, row0 + n_q)
        (query atoms q_row0 + row0 ...); returns the output as a device tensor."""
        import paper_2607_05439_amd as dcp
        torch = self.torch
        wl = self.wl
        n_q = wl.n_q - row0 if n_q is None else n_q
        nb = self.nbr if nbr is None else nbr
        k = nb.shape[1]
        shape = self.shape(out_dtype, p_gathered, k)
        out = torch.empty((max(n_q, 1), wl.n_heads * wl.head_dim),
                          dtype=torch.float32 if out_dtype == DCP_F32 else torch.bfloat16, device=self.dev)
        nbytes = dcp.dcp_sparse_workspace_size(shape, n_q)
        ws = workspace if workspace is not None else torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                                                 device=self.dev)
        pt = self.p if p is None else p
        p_ptr = pt.data_ptr() + row0 * pt.shape[1] * pt.shape[2] * pt.element_size()
        nbr_ptr = nb.data_ptr() + row0 * k * 4
        dcp.dcp_sparse_pair_bias_attention(shape, self.weights(), self.a, p_ptr, nbr_ptr, wl.q_row0 + row0, n_q, n_kb,
                                           out, ws, ws.numel(), None)
        return out

    def gathered_p(self, nbr: Optional[np.ndarray] = None):
        """P_sparse [n_q, k, c_ap] on the device, from the host generator."""
        nb = self.nbr_host if nbr is None else nbr
        rows = self.wl.q_row0 + np.arange(self.wl.n_q)
        return self._to_dev(synth.p_gathered_host(self.wl, rows, nb))

    def oracle_rows(self, local_rows: Sequence[int], n_blocks: int = 1, nbr: Optional[np.ndarray] = None,
                    drop_affine: bool = False) -> np.ndarray:
        """fp64 oracle for stripe rows ``local_rows`` on the generator's host copy
        of the same inputs."""
        local_rows = np.asarray(local_rows, dtype=np.int64)
        nb = (self.nbr_host if nbr is None else nbr)[local_rows]
        atoms = self.wl.q_row0 + local_rows
        p = synth.p_gathered_host(self.wl, atoms, nb)
        w = dict(self.w_host)
        if drop_affine:
            w["b_b"] = None
            w["ln_beta"] = None
        return oracle.sparse_attention(self.a_host, p, nb, atoms, w, self.wl.n_heads, self.wl.head_dim,
                                       n_blocks=n_blocks)
