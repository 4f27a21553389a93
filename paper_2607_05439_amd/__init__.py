"""Python binding of libdcp.so (include/dcp.h): argument marshalling only.

Every step of the computation runs in the library's HIP kernels; PyTorch is
used for device memory and streams. The functions carry the C names
(``dcp_pair_bias_attention``, ``dcp_pair_bias_attention_noalloc``, ``dcp_pair_bias_attention_partial``, ``dcp_bias_project``, ``dcp_block_merge``,
``dcp_workspace_size``, ``dcp_workspace_bytes``, ``dcp_sparse_pair_bias_attention``,
``dcp_sparse_workspace_size``, ``dcp_knn_topk``, ``dcp_knn_workspace_size``, ``dcp_topk_merge``,
``dcp_pair_transition``, ``dcp_transition_workspace_size``, ``dcp_scatter_mean``,
``dcp_scatter_mean_workspace_size``) and accept torch tensors (device pointers are taken
from ``data_ptr()``) or plain integer addresses. Loading fails loudly when the
library has not been built: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Union

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdcp.so")

DCP_F32, DCP_BF16 = 0, 1
DCP_OK, DCP_ERR_INVALID_ARGUMENT, DCP_ERR_UNSUPPORTED, DCP_ERR_WORKSPACE, DCP_ERR_HIP = 0, -1, -2, -3, -4
EXPORTS = ("dcp_workspace_size", "dcp_workspace_bytes", "dcp_pair_bias_attention", "dcp_pair_bias_attention_noalloc", "dcp_pair_bias_attention_partial", "dcp_bias_project",
           "dcp_block_merge",
           "dcp_sparse_workspace_size", "dcp_sparse_pair_bias_attention", "dcp_knn_topk", "dcp_knn_workspace_size", "dcp_topk_merge",
           "dcp_transition_workspace_size", "dcp_pair_transition", "dcp_scatter_mean_workspace_size",
           "dcp_scatter_mean", "dcp_set_timing_events",
           "dcp_last_error", "dcp_version")


class DcpError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"dcp error {code}: {message}")
        self.code = code


class DcpShape(ctypes.Structure):
    _fields_ = [("n_tokens", ctypes.c_int64), ("c_s", ctypes.c_int32), ("c_z", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("out_dtype", ctypes.c_int32), ("ln_eps", ctypes.c_float)]


class DcpWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w_q", "w_k", "w_v", "w_g", "w_b", "b_b", "ln_gamma", "ln_beta")]


class DcpSparseShape(ctypes.Structure):
    _fields_ = [("n_atoms", ctypes.c_int64), ("c_atom", ctypes.c_int32), ("c_ap", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("k", ctypes.c_int32),
                ("act_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32), ("p_gathered", ctypes.c_int32),
                ("ln_eps", ctypes.c_float)]


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
        P = ctypes.POINTER
        L.dcp_workspace_size.argtypes = [P(DcpShape), i64, i32, P(sz)]
        L.dcp_workspace_bytes.argtypes = [P(DcpShape), i64, i32]
        L.dcp_workspace_bytes.restype = sz
        L.dcp_pair_bias_attention.argtypes = [P(DcpShape), P(DcpWeights), vp, vp, vp, i64, i64, i32, vp, vp, sz, vp]
        L.dcp_pair_bias_attention_noalloc.argtypes = [P(DcpShape), P(DcpWeights), vp, vp, vp, i64, i64, i32, vp, vp]
        L.dcp_pair_bias_attention_partial.argtypes = [P(DcpShape), P(DcpWeights), vp, vp, vp, i64, i64, i64, i64, vp,
                                                      vp, vp, vp, vp, sz, vp]
        L.dcp_bias_project.argtypes = [P(DcpShape), P(DcpWeights), vp, i64, i64, i64, vp, vp]
        L.dcp_block_merge.argtypes = [i32, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, i32, vp]
        L.dcp_sparse_workspace_size.argtypes = [P(DcpSparseShape), i64, P(sz)]
        L.dcp_sparse_pair_bias_attention.argtypes = [P(DcpSparseShape), P(DcpWeights), vp, vp, vp, i64, i64, i32, vp,
                                                     vp, sz, vp]
        L.dcp_knn_topk.argtypes = [vp, i64, vp, i64, i64, i64, vp, vp, i32, i32, vp, vp, vp, ctypes.c_size_t, vp]
        L.dcp_knn_workspace_size.argtypes = [i64, ctypes.POINTER(ctypes.c_size_t)]
        L.dcp_topk_merge.argtypes = [i64, i32, vp, vp, vp, vp, vp, vp, vp]
        L.dcp_transition_workspace_size.argtypes = [i32, i32, i32, P(sz)]
        L.dcp_pair_transition.argtypes = [i64, i32, i32, i32, ctypes.c_float, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.dcp_scatter_mean_workspace_size.argtypes = [i64, i32, P(sz)]
        L.dcp_scatter_mean.argtypes = [i64, i64, i32, i32, i32, vp, vp, vp, vp, sz, vp]
        L.dcp_set_timing_events.argtypes = [vp, vp]
        for f in (L.dcp_workspace_size, L.dcp_pair_bias_attention, L.dcp_pair_bias_attention_noalloc,
                  L.dcp_pair_bias_attention_partial,
                  L.dcp_bias_project, L.dcp_block_merge,
                  L.dcp_sparse_workspace_size, L.dcp_sparse_pair_bias_attention, L.dcp_knn_topk, L.dcp_knn_workspace_size, L.dcp_topk_merge,
                  L.dcp_transition_workspace_size, L.dcp_pair_transition, L.dcp_scatter_mean_workspace_size,
                  L.dcp_scatter_mean, L.dcp_set_timing_events):
            f.restype = ctypes.c_int
        L.dcp_last_error.restype = ctypes.c_char_p
        L.dcp_last_error.argtypes = []
        L.dcp_version.restype = ctypes.c_char_p
        L.dcp_version.argtypes = []
        _lib = L
    return _lib


Ptr = Union[int, None, "torch.Tensor"]  # noqa: F821


def _ptr(x: Ptr) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x or None
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def _check(rc: int) -> None:
    if rc != DCP_OK:
        raise DcpError(rc, lib().dcp_last_error().decode())


def make_shape(n_tokens: int, c_s: int, c_z: int, n_heads: int, head_dim: int, act_dtype: int, out_dtype: int,
               ln_eps: float = 1e-5) -> DcpShape:
    return DcpShape(n_tokens, c_s, c_z, n_heads, head_dim, act_dtype, out_dtype, ln_eps)


def make_weights(w_q: Ptr, w_k: Ptr, w_v: Ptr, w_g: Ptr, w_b: Ptr, b_b: Ptr = None, ln_gamma: Ptr = None,
                 ln_beta: Ptr = None) -> DcpWeights:
    return DcpWeights(*[_ptr(x) for x in (w_q, w_k, w_v, w_g, w_b, b_b, ln_gamma, ln_beta)])


def dcp_workspace_size(shape: DcpShape, n_q: int, n_key_blocks: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().dcp_workspace_size(ctypes.byref(shape), n_q, n_key_blocks, ctypes.byref(out)))
    return out.value


def dcp_workspace_bytes(shape: Optional[DcpShape], n_q: int, n_key_blocks: int) -> int:
    """The size-returning query: 0 (with dcp_last_error() set) on invalid arguments."""
    return int(lib().dcp_workspace_bytes(None if shape is None else ctypes.byref(shape), n_q, n_key_blocks))


def dcp_pair_bias_attention(shape: DcpShape, weights: DcpWeights, s: Ptr, z_rows: Ptr, key_mask: Ptr, q_row0: int,
                            n_q: int, n_key_blocks: int, out: Ptr, workspace: Ptr, workspace_bytes: int,
                            stream=None) -> None:
    _check(lib().dcp_pair_bias_attention(ctypes.byref(shape), ctypes.byref(weights), _ptr(s), _ptr(z_rows),
                                         _ptr(key_mask), q_row0, n_q, n_key_blocks, _ptr(out), _ptr(workspace),
                                         workspace_bytes, _stream(stream)))


NOALLOC_SCRATCH_BYTES = 128 << 20  # DCP_NOALLOC_SCRATCH_BYTES


def dcp_pair_bias_attention_noalloc(shape: DcpShape, weights: DcpWeights, s: Ptr, z_rows: Ptr, key_mask: Ptr,
                                    q_row0: int, n_q: int, n_key_blocks: int, out: Ptr, stream=None) -> None:
    _check(lib().dcp_pair_bias_attention_noalloc(ctypes.byref(shape), ctypes.byref(weights), _ptr(s), _ptr(z_rows),
                                                 _ptr(key_mask), q_row0, n_q, n_key_blocks, _ptr(out),
                                                 _stream(stream)))


def dcp_pair_bias_attention_partial(shape: DcpShape, weights: DcpWeights, s: Ptr, z_rows: Ptr, key_mask: Ptr,
                                    q_row0: int, n_q: int, k0: int, k1: int, m_out: Ptr, l_out: Ptr, acc_out: Ptr,
                                    gate_out: Ptr, workspace: Ptr, workspace_bytes: int, stream=None) -> None:
    _check(lib().dcp_pair_bias_attention_partial(ctypes.byref(shape), ctypes.byref(weights), _ptr(s), _ptr(z_rows),
                                                 _ptr(key_mask), q_row0, n_q, k0, k1, _ptr(m_out), _ptr(l_out),
                                                 _ptr(acc_out), _ptr(gate_out), _ptr(workspace), workspace_bytes,
                                                 _stream(stream)))


def dcp_bias_project(shape: DcpShape, weights: DcpWeights, z_tile: Ptr, n_rows: int, n_cols: int,
                     row_stride_elems: int, bias_out: Ptr, stream=None) -> None:
    _check(lib().dcp_bias_project(ctypes.byref(shape), ctypes.byref(weights), _ptr(z_tile), n_rows, n_cols,
                                  row_stride_elems, _ptr(bias_out), _stream(stream)))


def dcp_block_merge(n_parts: int, n_rows: int, n_heads: int, head_dim: int, m_parts: Ptr, l_parts: Ptr,
                    acc_parts: Ptr, m_out: Ptr, l_out: Ptr, acc_out: Ptr, gate: Ptr, out: Ptr, out_dtype: int,
                    stream=None) -> None:
    _check(lib().dcp_block_merge(n_parts, n_rows, n_heads, head_dim, _ptr(m_parts), _ptr(l_parts), _ptr(acc_parts),
                                 _ptr(m_out), _ptr(l_out), _ptr(acc_out), _ptr(gate), _ptr(out), out_dtype,
                                 _stream(stream)))


def make_sparse_shape(n_atoms: int, c_atom: int, c_ap: int, n_heads: int, head_dim: int, k: int, act_dtype: int,
                      out_dtype: int, p_gathered: int = 0, ln_eps: float = 1e-5) -> DcpSparseShape:
    return DcpSparseShape(n_atoms, c_atom, c_ap, n_heads, head_dim, k, act_dtype, out_dtype, p_gathered, ln_eps)


def dcp_sparse_workspace_size(shape: DcpSparseShape, n_q: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().dcp_sparse_workspace_size(ctypes.byref(shape), n_q, ctypes.byref(out)))
    return out.value


def dcp_sparse_pair_bias_attention(shape: DcpSparseShape, weights: DcpWeights, a: Ptr, p: Ptr, nbr: Ptr, q_row0: int,
                                   n_q: int, n_key_blocks: int, out: Ptr, workspace: Ptr, workspace_bytes: int,
                                   stream=None) -> None:
    _check(lib().dcp_sparse_pair_bias_attention(ctypes.byref(shape), ctypes.byref(weights), _ptr(a), _ptr(p),
                                                _ptr(nbr), q_row0, n_q, n_key_blocks, _ptr(out), _ptr(workspace),
                                                workspace_bytes, _stream(stream)))


def dcp_knn_workspace_size(n_c: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dcp_knn_workspace_size(n_c, ctypes.byref(n)))
    return n.value


def dcp_knn_topk(x_q: Ptr, n_q: int, x_c: Ptr, n_c: int, c_index0: int, q_self0: int, group_q: Ptr, group_c: Ptr,
                 group_mode: int, k: int, idx_out: Ptr, d2_out: Ptr, workspace: Ptr, workspace_bytes: int,
                 stream=None) -> None:
    _check(lib().dcp_knn_topk(_ptr(x_q), n_q, _ptr(x_c), n_c, c_index0, q_self0, _ptr(group_q), _ptr(group_c),
                              group_mode, k, _ptr(idx_out), _ptr(d2_out), _ptr(workspace), workspace_bytes,
                              _stream(stream)))


def dcp_topk_merge(n_rows: int, k: int, idx_a: Ptr, d2_a: Ptr, idx_b: Ptr, d2_b: Ptr, idx_out: Ptr, d2_out: Ptr,
                   stream=None) -> None:
    _check(lib().dcp_topk_merge(n_rows, k, _ptr(idx_a), _ptr(d2_a), _ptr(idx_b), _ptr(d2_b), _ptr(idx_out),
                                _ptr(d2_out), _stream(stream)))


def dcp_transition_workspace_size(c_z: int, hidden: int, act_dtype: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().dcp_transition_workspace_size(c_z, hidden, act_dtype, ctypes.byref(out)))
    return out.value


def dcp_pair_transition(n_pairs: int, c_z: int, hidden: int, act_dtype: int, ln_eps: float, w1: Ptr, w2: Ptr, w3: Ptr,
                        ln_gamma: Ptr, ln_beta: Ptr, z_in: Ptr, z_out: Ptr, workspace: Ptr, workspace_bytes: int,
                        stream=None) -> None:
    _check(lib().dcp_pair_transition(n_pairs, c_z, hidden, act_dtype, ln_eps, _ptr(w1), _ptr(w2), _ptr(w3),
                                     _ptr(ln_gamma), _ptr(ln_beta), _ptr(z_in), _ptr(z_out), _ptr(workspace),
                                     workspace_bytes, _stream(stream)))


def dcp_scatter_mean_workspace_size(n_tokens: int, c: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().dcp_scatter_mean_workspace_size(n_tokens, c, ctypes.byref(out)))
    return out.value


def dcp_scatter_mean(n_atoms: int, n_tokens: int, c: int, in_dtype: int, out_dtype: int, a: Ptr, tok_idx: Ptr,
                     out: Ptr, workspace: Ptr, workspace_bytes: int, stream=None) -> None:
    _check(lib().dcp_scatter_mean(n_atoms, n_tokens, c, in_dtype, out_dtype, _ptr(a), _ptr(tok_idx), _ptr(out),
                                  _ptr(workspace), workspace_bytes, _stream(stream)))


def dcp_set_timing_events(start_event: Optional[int], stop_event: Optional[int]) -> None:
    _check(lib().dcp_set_timing_events(start_event, stop_event))


def dcp_last_error() -> str:
    return lib().dcp_last_error().decode()


def dcp_version() -> str:
    return lib().dcp_version().decode()
