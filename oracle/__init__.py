"""fp64 CPU oracle for pair-biased, gated multi-head attention.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. It shares no code
with the GPU path (``paper_2607_05439_amd``) and neither imports the other.

The arithmetic lives in ``oracle.c`` (its header states the definition and the
paper passages it follows); this module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_lib = None


def _configure(lib: ctypes.CDLL) -> ctypes.CDLL:
    i64, i32, vp, f64 = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_double
    lib.oracle_chunk.argtypes = [i64, i64, i64, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.oracle_linear.argtypes = [i64, i32, i32, vp, vp, vp]
    lib.oracle_bias.argtypes = [i64, i64, i32, i32, vp, i32, i64, vp, vp, vp, vp, f64, vp]
    lib.oracle_attend.argtypes = [i64, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_merge.argtypes = [i32, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_attention.argtypes = [i64, i32, i32, i32, i32, vp, vp, i32, vp, i64, vp,
                                     vp, vp, vp, vp, vp, vp, vp, vp, f64, i32, vp, vp, vp, vp]
    lib.oracle_sparse_attention.argtypes = [i64, i32, i32, i32, i32, i32, vp, vp, i32, vp, vp, i64,
                                            vp, vp, vp, vp, vp, vp, vp, vp, f64, i32, vp]
    lib.oracle_knn.argtypes = [vp, i64, vp, i64, i64, vp, vp, i32, i32, vp, vp]
    lib.oracle_transition.argtypes = [i64, i32, i32, vp, i32, vp, vp, vp, vp, vp, f64, vp]
    lib.oracle_scatter_mean.argtypes = [i64, i64, i32, vp, i32, vp, vp]
    lib.oracle_topk_merge.argtypes = [i64, i32, vp, vp, vp, vp, vp, vp]
    lib.oracle_knn_blocked.argtypes = [vp, i64, vp, i64, vp, vp, i32, i32, i32, vp, vp]
    for f in (lib.oracle_bias, lib.oracle_attend, lib.oracle_merge, lib.oracle_attention,
              lib.oracle_sparse_attention, lib.oracle_knn, lib.oracle_topk_merge, lib.oracle_knn_blocked,
              lib.oracle_transition, lib.oracle_scatter_mean):
        f.restype = ctypes.c_int
    return lib


def _load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        path = os.path.join(_HERE, "liboracle.so")
        if not os.path.exists(path):
            from . import build as _b
            _b.build()
        _lib = _configure(ctypes.CDLL(path))
    return _lib


def _f64(a: Optional[np.ndarray]) -> Optional[np.ndarray]:
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _zbuf(z: np.ndarray) -> Tuple[np.ndarray, int]:
    """Pair-tensor buffer: uint16 holds bf16 bit patterns (dtype 1); float32 is dtype 0."""
    if z.dtype == np.uint16:
        return np.ascontiguousarray(z), 1
    if z.dtype == np.float32:
        return np.ascontiguousarray(z), 0
    raise TypeError("z must be bf16 bits (uint16) or float32")


def decode(x: np.ndarray) -> np.ndarray:
    """Exact fp64 value of an fp32 array or of bf16 bit patterns (uint16)."""
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float64)


def chunk(total: int, parts: int, p: int) -> Tuple[int, int]:
    size, start = ctypes.c_int64(), ctypes.c_int64()
    _load().oracle_chunk(total, parts, p, ctypes.byref(size), ctypes.byref(start))
    return size.value, start.value


def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    x, w = _f64(x), _f64(w)
    y = np.empty((x.shape[0], w.shape[0]))
    _load().oracle_linear(x.shape[0], w.shape[1], w.shape[0], _p(x), _p(w), _p(y))
    return y


def bias(z: np.ndarray, w_b: np.ndarray, b_b=None, gamma=None, beta=None, eps: float = 1e-5) -> np.ndarray:
    """bias[r, c, h] for z[r, c, :] (shape [n_rows, n_cols, c_z])."""
    zb, dt = _zbuf(z)
    n_rows, n_cols, c_z = zb.shape
    w_b, b_b, gamma, beta = _f64(w_b), _f64(b_b), _f64(gamma), _f64(beta)
    out = np.empty((n_rows, n_cols, w_b.shape[0]))
    rc = _load().oracle_bias(n_rows, n_cols, c_z, w_b.shape[0], zb.ctypes.data, dt, n_cols * c_z,
                             _p(w_b), _p(b_b), _p(gamma), _p(beta), eps, _p(out))
    assert rc == 0
    return out


def attend(q, k, v, g_pre, bias_rows, mask, n_heads: int, head_dim: int) -> np.ndarray:
    """Attention from explicit ingredients; bias_rows is [n_rows, n_tok, H]."""
    q, k, v, g_pre, bias_rows = _f64(q), _f64(k), _f64(v), _f64(g_pre), _f64(bias_rows)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    out = np.empty((q.shape[0], n_heads * head_dim))
    rc = _load().oracle_attend(q.shape[0], k.shape[0], n_heads, head_dim, _p(q), _p(k), _p(v), _p(g_pre),
                               _p(bias_rows), _p(m), _p(out))
    assert rc == 0
    return out


def merge(m, l, acc, gate=None):
    """Merge partials m, l [P, H, R], acc [P, R, H, d]; returns (m, l, acc, out)."""
    m, l, acc, gate = _f64(m), _f64(l), _f64(acc), _f64(gate)
    n_parts, n_heads, n_rows = m.shape
    d = acc.shape[3]
    mo, lo = np.empty((n_heads, n_rows)), np.empty((n_heads, n_rows))
    ao, out = np.empty((n_rows, n_heads, d)), np.empty((n_rows, n_heads * d))
    rc = _load().oracle_merge(n_parts, n_rows, n_heads, d, _p(m), _p(l), _p(acc), _p(gate),
                              _p(mo), _p(lo), _p(ao), _p(out))
    assert rc == 0
    return mo, lo, ao, out


def attention(s: np.ndarray, z_rows: np.ndarray, rows: Sequence[int], mask: Optional[np.ndarray],
              w: Dict[str, Optional[np.ndarray]], n_heads: int, head_dim: int, eps: float = 1e-5,
              n_blocks: int = 1, return_parts: bool = False):
    """The whole definition for query tokens ``rows``.

    s: [N, c_s] (fp32, or bf16 bits as uint16); z_rows: [len(rows), N, c_z]
    (z[rows[r], :, :]); w: fp32 weights in nn.Linear layout (keys w_q, w_k,
    w_v, w_g, w_b and optional ln_gamma, ln_beta, b_b).
    """
    s64 = decode(s) if s.dtype == np.uint16 else _f64(s)
    n_tok, c_s = s64.shape
    zb, dt = _zbuf(z_rows)
    assert zb.shape[0] == len(rows) and zb.shape[1] == n_tok
    c_z = zb.shape[2]
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    ws = {k_: _f64(w.get(k_)) for k_ in ("w_q", "w_k", "w_v", "w_g", "w_b", "b_b", "ln_gamma", "ln_beta")}
    hd = n_heads * head_dim
    out = np.empty((len(r), hd))
    parts = None
    if return_parts and n_blocks > 1:
        parts = (np.empty((n_blocks, n_heads, len(r))), np.empty((n_blocks, n_heads, len(r))),
                 np.empty((n_blocks, len(r), n_heads, head_dim)))
    rc = _load().oracle_attention(
        n_tok, c_s, c_z, n_heads, head_dim, _p(s64), zb.ctypes.data, dt, _p(r), len(r), _p(m),
        _p(ws["w_q"]), _p(ws["w_k"]), _p(ws["w_v"]), _p(ws["w_g"]), _p(ws["w_b"]), _p(ws["b_b"]),
        _p(ws["ln_gamma"]), _p(ws["ln_beta"]), eps, n_blocks, _p(out),
        _p(parts[0]) if parts else None, _p(parts[1]) if parts else None, _p(parts[2]) if parts else None)
    if rc != 0:
        raise ValueError("oracle_attention rejected its arguments")
    return (out, parts) if return_parts else out


def sparse_attention(a: np.ndarray, p_rows: np.ndarray, nbr: np.ndarray, rows: Sequence[int],
                     w: Dict[str, Optional[np.ndarray]], n_heads: int, head_dim: int, eps: float = 1e-5,
                     n_blocks: int = 1) -> np.ndarray:
    """Sparse kNN pair-biased attention for query atoms ``rows``.

    a: [L, c_atom] (fp32 or bf16 bits); p_rows: [len(rows), k, c_ap] gathered
    pair slices (fp32 or bf16 bits); nbr: [len(rows), k] int32 neighbour atom
    indices (-1 = empty slot); w: weights as for ``attention``.
    """
    a64 = decode(a) if a.dtype == np.uint16 else _f64(a)
    n_atoms, c_atom = a64.shape
    pb, dt = _zbuf(p_rows)
    n_rows, k, c_ap = pb.shape
    nb = np.ascontiguousarray(nbr, dtype=np.int32)
    assert nb.shape == (n_rows, k) and len(rows) == n_rows
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    ws = {k_: _f64(w.get(k_)) for k_ in ("w_q", "w_k", "w_v", "w_g", "w_b", "b_b", "ln_gamma", "ln_beta")}
    out = np.empty((n_rows, n_heads * head_dim))
    rc = _load().oracle_sparse_attention(
        n_atoms, c_atom, c_ap, n_heads, head_dim, k, _p(a64), pb.ctypes.data, dt, nb.ctypes.data, _p(r), n_rows,
        _p(ws["w_q"]), _p(ws["w_k"]), _p(ws["w_v"]), _p(ws["w_g"]), _p(ws["w_b"]), _p(ws["b_b"]),
        _p(ws["ln_gamma"]), _p(ws["ln_beta"]), eps, n_blocks, _p(out))
    if rc != 0:
        raise ValueError("oracle_sparse_attention rejected its arguments")
    return out


def _f32c(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32c(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def knn(x_q: np.ndarray, x_c: np.ndarray, k: int, c_index0: int = 0, group_q=None, group_c=None, group_mode: int = 0,
        n_blocks: int = 1) -> Tuple[np.ndarray, np.ndarray]:
    """k nearest candidates of each query: (idx [n_q, k] int32, d2 [n_q, k] fp32),
    sorted by (d2, index); n_blocks > 1 uses the blocked ring form (c_index0 = 0)."""
    xq, xc = _f32c(x_q), _f32c(x_c)
    gq, gc = _i32c(group_q), _i32c(group_c)
    n_q, n_c = xq.shape[0], xc.shape[0]
    idx = np.empty((n_q, k), dtype=np.int32)
    d2 = np.empty((n_q, k), dtype=np.float32)
    gp = lambda a: None if a is None else a.ctypes.data
    if n_blocks == 1:
        rc = _load().oracle_knn(xq.ctypes.data, n_q, xc.ctypes.data, n_c, c_index0, gp(gq), gp(gc), group_mode, k,
                                idx.ctypes.data, d2.ctypes.data)
    else:
        assert c_index0 == 0
        rc = _load().oracle_knn_blocked(xq.ctypes.data, n_q, xc.ctypes.data, n_c, gp(gq), gp(gc), group_mode, k,
                                        n_blocks, idx.ctypes.data, d2.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_knn rejected its arguments")
    return idx, d2


def topk_merge(idx_a, d2_a, idx_b, d2_b) -> Tuple[np.ndarray, np.ndarray]:
    """The ring top-k combine of two sorted candidate lists [n, k]."""
    ia, ib = _i32c(idx_a), _i32c(idx_b)
    da, db = _f32c(d2_a), _f32c(d2_b)
    n, k = ia.shape
    io = np.empty((n, k), dtype=np.int32)
    do = np.empty((n, k), dtype=np.float32)
    rc = _load().oracle_topk_merge(n, k, ia.ctypes.data, da.ctypes.data, ib.ctypes.data, db.ctypes.data,
                                   io.ctypes.data, do.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_topk_merge rejected its arguments")
    return io, do


def transition(z: np.ndarray, w1: np.ndarray, w2: np.ndarray, w3: np.ndarray, gamma=None, beta=None,
               eps: float = 1e-5) -> np.ndarray:
    """z + W3 (SiLU(W1 LN(z)) * W2 LN(z)) per pair; z [..., c_z] fp32 or bf16 bits; fp64 result."""
    zb, dt = _zbuf(z)
    c_z = zb.shape[-1]
    n = zb.size // c_z
    hidden = np.asarray(w1).shape[0]
    out = np.empty(zb.shape, dtype=np.float64)
    keep = [_f64(a) for a in (w1, w2, w3, gamma, beta)]  # alive until the call returns
    rc = _load().oracle_transition(n, c_z, hidden, zb.ctypes.data, dt, *[_p(a) for a in keep], eps, _p(out))
    if rc != 0:
        raise ValueError("oracle_transition rejected its arguments")
    return out


def scatter_mean(a: np.ndarray, tok_idx: np.ndarray, n_tokens: int) -> np.ndarray:
    """Per-token mean of atom features a [n_atoms, c] (fp32 or bf16 bits); fp64 [n_tokens, c]."""
    ab, dt = _zbuf(a)
    n_atoms, c = ab.shape
    idx = np.ascontiguousarray(tok_idx, dtype=np.int32)
    assert idx.shape == (n_atoms,)
    out = np.empty((n_tokens, c), dtype=np.float64)
    rc = _load().oracle_scatter_mean(n_atoms, n_tokens, c, ab.ctypes.data, dt, idx.ctypes.data, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_scatter_mean rejected its arguments")
    return out
