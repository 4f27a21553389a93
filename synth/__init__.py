"""Seeded synthetic inputs for pair-biased attention (tests and benchmark).

This module is shared by the fp64 oracle's tests and by the GPU path's tests
and benchmark. It holds no attention arithmetic: it only draws numbers.

Definition (the numpy functions below are the reference; ``csrc/synth_host.c``
and ``csrc/synth_dev.hip`` are bit-identical twins, checked by tests):

* ``fin``: the SplitMix64 output function (Steele, Lea and Flood, 2014).
* ``key(seed, t) = fin(fin(seed + G) + t*G)`` with ``G = 0x9E3779B97F4A7C15``;
  one independent stream per tensor id ``t``.
* ``word(k, n) = fin(k + (n+1)*G)``: counter-based SplitMix64.
* ``normal(k, e)``: the twelve 16-bit fields of ``word(k, 3e..3e+2)`` summed
  (Irwin-Hall(12)), minus 393210, over 65536. Mean 0, variance 1 - 2^-32,
  range about +-6. Every value is an exact fp32 number.
* bf16 tensors take round-to-nearest-even of that fp32 value.

The workloads are the synthetic stand-ins for the paper's icosahedral RFD3
sampling runs (60 copies of a subunit, c_s = 384, c_z = 128, 16 heads); the
paper's own runs need trained weights and are not reproducible here.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
G = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# Tensor ids: one independent stream each.
T_S, T_Z, T_WQ, T_WK, T_WV, T_WG, T_WB, T_ZBASE, T_MASK, T_GAMMA, T_BETA, T_BB = range(1, 13)
# atom path: single track A, pair track P, neighbour draws, ragged draws, weights
(T_A, T_P, T_NBR, T_NBR_RAG, T_AWQ, T_AWK, T_AWV, T_AWG, T_AWB, T_AGAMMA, T_ABETA, T_ABB) = range(13, 25)
T_XYZ = 25  # atom coordinates
T_TW1, T_TW2, T_TW3, T_TGAMMA, T_TBETA = range(26, 31)  # pair transition weights
T_ATOMS_PER_TOK, T_AFEAT = 31, 32  # atom -> token pooling


# ----------------------------------------------------------------------------- numpy definition
def _fin(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.uint64)
    x = x ^ (x >> np.uint64(30))
    x = x * _M1
    x = x ^ (x >> np.uint64(27))
    x = x * _M2
    return x ^ (x >> np.uint64(31))


def key(seed: int, tensor_id: int) -> int:
    with np.errstate(over="ignore"):
        k = _fin(np.array([seed], dtype=np.uint64) + G)
        k = _fin(k + np.uint64(tensor_id) * G)
    return int(k[0])


def word_np(k: int, n: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return _fin(np.uint64(k) + (np.asarray(n, dtype=np.uint64) + np.uint64(1)) * G)


def normal_np(k: int, start: int, count: int) -> np.ndarray:
    """fp32 normals ``normal(k, start + i)`` for i < count (reference definition)."""
    return normal_np_at(k, np.arange(count, dtype=np.uint64) + np.uint64(start))


def normal_np_at(k: int, e: np.ndarray) -> np.ndarray:
    """fp32 normals ``normal(k, e[i])`` at arbitrary element indices."""
    e = np.asarray(e, dtype=np.uint64)
    s = np.zeros(e.shape, dtype=np.int64)
    for j in range(3):
        w = word_np(k, np.uint64(3) * e + np.uint64(j))
        for t in range(4):
            s += ((w >> np.uint64(16 * t)) & np.uint64(0xFFFF)).astype(np.int64)
    return ((s - 393210).astype(np.float32) * np.float32(1.0 / 65536.0)).astype(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns the 16-bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))
    return (b >> np.uint64(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def z_rows_np(k_z: int, k_base: int, period: int, n_tok: int, c_z: int, rows: Sequence[int],
              bf16: bool) -> np.ndarray:
    """Reference definition of rows of z (small sizes only)."""
    out = []
    for i in rows:
        e0 = int(i) * n_tok * c_z
        v = normal_np(k_z, e0, n_tok * c_z).reshape(n_tok, c_z)
        if period > 0:
            j = np.arange(n_tok)
            eb = ((int(i) % period) * period + (j % period))[:, None] * c_z + np.arange(c_z)[None, :]
            base = normal_np_at(k_base, eb.astype(np.uint64))
            v = (base + (np.float32(0.1) * v).astype(np.float32)).astype(np.float32)
        out.append(bf16_round(v) if bf16 else v)
    return np.stack(out)


# ----------------------------------------------------------------------------- fast C twin
_host_lib = None


def _host() -> ctypes.CDLL:
    global _host_lib
    if _host_lib is None:
        path = os.path.join(_HERE, "libsynth_host.so")
        if not os.path.exists(path):
            from . import build as _b
            _b.build_host()
        lib = ctypes.CDLL(path)
        u64, i64, i32, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.synth_key.restype = u64
        lib.synth_key.argtypes = [u64, u64]
        lib.synth_word.restype = u64
        lib.synth_word.argtypes = [u64, u64]
        lib.synth_normal_f32.argtypes = [u64, u64, i64, vp]
        lib.synth_normal_bf16.argtypes = [u64, u64, i64, vp]
        lib.synth_z_rows.argtypes = [u64, u64, i64, i64, i32, vp, i64, i32, vp]
        lib.synth_neighbours.argtypes = [u64, u64, i64, i32, i32, i32, i32, i32, i64, i64, i32, vp]
        lib.synth_coords.argtypes = [u64, i64, i32, i32, vp]
        _host_lib = lib
    return _host_lib


def normal(k: int, start: int, count: int, bf16: bool = False) -> np.ndarray:
    out = np.empty(count, dtype=np.uint16 if bf16 else np.float32)
    fn = _host().synth_normal_bf16 if bf16 else _host().synth_normal_f32
    fn(k, start, count, out.ctypes.data)
    return out


def z_rows(k_z: int, k_base: int, period: int, n_tok: int, c_z: int, rows: Sequence[int],
           bf16: bool) -> np.ndarray:
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    out = np.empty((len(r), n_tok, c_z), dtype=np.uint16 if bf16 else np.float32)
    _host().synth_z_rows(k_z, k_base, period, n_tok, c_z, r.ctypes.data, len(r), int(bf16), out.ctypes.data)
    return out


# ----------------------------------------------------------------------------- workloads
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_tok: int
    c_s: int
    c_z: int
    n_heads: int
    head_dim: int
    dtype: str                      # "f32" or "bf16": dtype of s and z
    n_key_blocks: int               # key blocks per call (the paper's ring steps)
    stripes: Tuple[Tuple[int, int], ...]  # (q_row0, n_q) per call
    mask: str = "none"              # "none" | "tail:K" | "random:K"
    z_period: int = 0               # 0: iid z; P > 0: z = base[i%P, j%P] + 0.1 noise
    seed: int = 0
    note: str = ""

    @property
    def bf16(self) -> bool:
        return self.dtype == "bf16"

    @property
    def elem_bytes(self) -> int:
        return 2 if self.bf16 else 4


def _w(name, n, c_s, c_z, h, d, dtype, n_kb, stripes, mask="none", period=0, note=""):
    return Workload(name, n, c_s, c_z, h, d, dtype, n_kb, stripes, mask, period, 0, note)


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        _w("tiny128_f32", 128, 128, 32, 4, 32, "f32", 1, ((0, 128),),
           note="tiny fp32 case; one key block (also run with 4 for the blocked check)"),
        _w("pad1024_bf16", 1024, 384, 128, 16, 24, "bf16", 4, ((0, 1024),), "tail:4",
           note="12 copies x 85-token subunit + 4 masked padding tokens; 4 key blocks of 256"),
        _w("ico4800_bf16", 4800, 384, 128, 16, 24, "bf16", 10, ((0, 4800),), "random:240", 80,
           note="60 copies x 80 tokens, 60-fold z structure, 5% random key mask, 10 key blocks of 480"),
        _w("grid12000_bf16", 12000, 384, 128, 16, 24, "bf16", 4,
           ((0, 3000), (3000, 3000), (6000, 3000), (9000, 3000)),
           note="one GPU's share of a 4x4 grid: 4 query stripes x 4 key blocks of 3000"),
        _w("asm24000_bf16", 24000, 384, 128, 16, 24, "bf16", 6, ((0, 24000),), "tail:480",
           note="whole 60 x 400 assembly, z = 147 GB bf16, last 480 tokens masked, 6 key blocks of 4000"),
    ]
}


def weights(wl: Workload, affine: bool = False) -> Dict[str, Optional[np.ndarray]]:
    """fp32 weights in nn.Linear layout [out, in], drawn N(0, 1/fan_in).

    ``affine=False`` gives the workloads' LayerNorm (gamma = 1, beta = 0, no
    projection bias); ``affine=True`` draws gamma, beta and b_b too (tests).
    """
    hd = wl.n_heads * wl.head_dim
    out: Dict[str, Optional[np.ndarray]] = {}
    for name, tid, rows, fan in (("w_q", T_WQ, hd, wl.c_s), ("w_k", T_WK, hd, wl.c_s),
                                 ("w_v", T_WV, hd, wl.c_s), ("w_g", T_WG, hd, wl.c_s),
                                 ("w_b", T_WB, wl.n_heads, wl.c_z)):
        scale = np.float32(1.0 / np.sqrt(fan))
        out[name] = (normal(key(wl.seed, tid), 0, rows * fan) * scale).astype(np.float32).reshape(rows, fan)
    if affine:
        out["ln_gamma"] = (np.float32(1.0) + np.float32(0.25) * normal(key(wl.seed, T_GAMMA), 0, wl.c_z)
                           ).astype(np.float32)
        out["ln_beta"] = normal(key(wl.seed, T_BETA), 0, wl.c_z)
        out["b_b"] = normal(key(wl.seed, T_BB), 0, wl.n_heads)
    else:
        out["ln_gamma"] = None
        out["ln_beta"] = None
        out["b_b"] = None
    return out


def s_host(wl: Workload) -> np.ndarray:
    """Single track s[N, c_s]: bf16 bit patterns (uint16) or fp32."""
    return normal(key(wl.seed, T_S), 0, wl.n_tok * wl.c_s, bf16=wl.bf16).reshape(wl.n_tok, wl.c_s)


def mask_host(wl: Workload) -> Optional[np.ndarray]:
    """Key mask [N] uint8 (1 = attend), or None when every key attends."""
    if wl.mask == "none":
        return None
    kind, k = wl.mask.split(":")
    k = int(k)
    m = np.ones(wl.n_tok, dtype=np.uint8)
    if kind == "tail":
        m[wl.n_tok - k:] = 0
    elif kind == "random":
        idx = np.arange(wl.n_tok, dtype=np.uint64)
        w = word_np(key(wl.seed, T_MASK), idx)
        order = np.lexsort((idx, w))  # by word, ties by index
        m[order[:k]] = 0
    else:
        raise ValueError(wl.mask)
    return m


def z_keys(wl: Workload) -> Tuple[int, int]:
    return key(wl.seed, T_Z), key(wl.seed, T_ZBASE)


def z_host(wl: Workload, rows: Sequence[int]) -> np.ndarray:
    """Rows of z[N, N, c_z] on the host, shape [len(rows), N, c_z]."""
    kz, kb = z_keys(wl)
    return z_rows(kz, kb, wl.z_period, wl.n_tok, wl.c_z, rows, wl.bf16)


# ----------------------------------------------------------------------------- atom workloads
@dataclasses.dataclass(frozen=True)
class AtomWorkload:
    """Sparse (kNN) pair-biased atom attention: L atoms with single track
    A[L, c_atom] and pair track P[L, L, c_ap]; the query atoms
    [q_row0, q_row0 + n_q) attend to k neighbour slots each."""
    name: str
    n_atoms: int
    c_atom: int
    c_ap: int
    n_heads: int
    head_dim: int
    k: int
    dtype: str                 # "f32" or "bf16": dtype of A and P
    n_key_blocks: int
    q_row0: int
    n_q: int
    per_res: int = 8           # atoms per residue
    per_chain: int = 1600      # atoms per chain
    win: int = 16              # residue window of the spatial draws
    q_inter: int = 32          # inter-chain quota, max(32, k/4) at k = 128
    ragged: bool = False
    seed: int = 0
    note: str = ""

    @property
    def bf16(self) -> bool:
        return self.dtype == "bf16"

    @property
    def elem_bytes(self) -> int:
        return 2 if self.bf16 else 4


ATOM_WORKLOADS: Dict[str, AtomWorkload] = {
    w.name: w
    for w in [
        AtomWorkload("atoms200_f32", 200, 128, 16, 4, 32, 128, "f32", 1, 0, 200, per_chain=50, ragged=True,
                     note="4 chains of 50 atoms: budgets larger than the candidate pools leave empty slots"),
        AtomWorkload("atoms5000_bf16", 5000, 128, 16, 4, 32, 128, "bf16", 1, 0, 5000, per_chain=1000,
                     ragged=True, note="RFD3's 5000-atom training crop as 5 chains of 1000; full P = 800 MB"),
        AtomWorkload("atoms96k_bf16", 96000, 128, 16, 4, 32, 128, "bf16", 4, 24000, 24000,
                     note="60 chains x 1600 atoms (200 residues x 8); one 24000-row stripe of P "
                          "(73.7 GB bf16) against 4 column blocks of 24000"),
    ]
}


def neighbours(wl: AtomWorkload, row0: int, n_rows: int) -> np.ndarray:
    """Neighbour lists nbr[n_rows, k] int32 of query atoms row0 .. row0+n_rows-1."""
    out = np.empty((n_rows, wl.k), dtype=np.int32)
    _host().synth_neighbours(key(wl.seed, T_NBR), key(wl.seed, T_NBR_RAG), wl.n_atoms, wl.per_res, wl.per_chain,
                             wl.k, wl.win, wl.q_inter, row0, n_rows, int(wl.ragged), out.ctypes.data)
    return out


def atom_weights(wl: AtomWorkload, affine: bool = False) -> Dict[str, Optional[np.ndarray]]:
    """fp32 weights [out, in] ~ N(0, 1/fan_in); ``affine`` also draws gamma, beta, b_b."""
    hd = wl.n_heads * wl.head_dim
    out: Dict[str, Optional[np.ndarray]] = {}
    for name, tid, rows, fan in (("w_q", T_AWQ, hd, wl.c_atom), ("w_k", T_AWK, hd, wl.c_atom),
                                 ("w_v", T_AWV, hd, wl.c_atom), ("w_g", T_AWG, hd, wl.c_atom),
                                 ("w_b", T_AWB, wl.n_heads, wl.c_ap)):
        scale = np.float32(1.0 / np.sqrt(fan))
        out[name] = (normal(key(wl.seed, tid), 0, rows * fan) * scale).astype(np.float32).reshape(rows, fan)
    if affine:
        out["ln_gamma"] = (np.float32(1.0) + np.float32(0.25) * normal(key(wl.seed, T_AGAMMA), 0, wl.c_ap)
                           ).astype(np.float32)
        out["ln_beta"] = normal(key(wl.seed, T_ABETA), 0, wl.c_ap)
        out["b_b"] = normal(key(wl.seed, T_ABB), 0, wl.n_heads)
    else:
        out["ln_gamma"] = out["ln_beta"] = out["b_b"] = None
    return out


def a_host(wl: AtomWorkload) -> np.ndarray:
    """Atom single track A[L, c_atom]: bf16 bit patterns (uint16) or fp32."""
    return normal(key(wl.seed, T_A), 0, wl.n_atoms * wl.c_atom, bf16=wl.bf16).reshape(wl.n_atoms, wl.c_atom)


def p_gathered_host(wl: AtomWorkload, rows: Sequence[int], nbr: np.ndarray) -> np.ndarray:
    """P[i, nbr[r, t], :] for i = rows[r] (zeros at empty slots), shape [len(rows), k, c_ap].

    P[i, j, c] = normal(key_P, (i*L + j)*c_ap + c), the same element numbering
    as the device generator of the pair tensor."""
    rows = np.asarray(rows, dtype=np.int64)
    nb = np.asarray(nbr, dtype=np.int64)
    valid = (nb >= 0) & (nb < wl.n_atoms)
    j = np.where(valid, nb, 0)
    e = ((rows[:, None] * wl.n_atoms + j)[:, :, None] * wl.c_ap + np.arange(wl.c_ap)[None, None, :])
    v = normal_np_at(key(wl.seed, T_P), e.astype(np.uint64).ravel()).reshape(e.shape)
    v = np.where(valid[:, :, None], v, np.float32(0.0)).astype(np.float32)
    return bf16_round(v) if wl.bf16 else v


def p_rows_host(wl: AtomWorkload, rows: Sequence[int]) -> np.ndarray:
    """Dense rows of P on the host, shape [len(rows), L, c_ap] (small L only)."""
    return z_rows(key(wl.seed, T_P), 0, 0, wl.n_atoms, wl.c_ap, rows, wl.bf16)


def p_fill_device(wl: AtomWorkload, ptr: int, row0: int, n_rows: int, stream: int) -> None:
    """Write rows [row0, row0+n_rows) of P into device memory at ``ptr``."""
    rc = _dev().synth_dev_z_rows(key(wl.seed, T_P), 0, 0, wl.n_atoms, wl.c_ap, row0, n_rows, int(wl.bf16), ptr,
                                 stream)
    if rc != 0:
        raise RuntimeError(f"synth_dev_z_rows failed ({rc})")


# ----------------------------------------------------------------------------- pair transition
TRANSITION_WORKLOADS = {
    # name: (pair-tensor workload whose z the transition updates, hidden units)
    "trans40_f32": ("adhoc40_f32", 128),
    "trans192_bf16": ("adhoc192_bf16", 512),
    "trans24000_bf16": ("asm24000_bf16", 512),
}


def transition_workload(name: str):
    """(pair-tensor Workload, hidden) of a transition workload."""
    zname, hidden = TRANSITION_WORKLOADS[name]
    if zname == "adhoc40_f32":
        wl = Workload("adhoc40_f32", 40, 32, 32, 1, 32, "f32", 1, ((0, 40),))
    elif zname == "adhoc192_bf16":
        wl = Workload("adhoc192_bf16", 192, 128, 128, 16, 24, "bf16", 1, ((0, 192),))
    else:
        wl = WORKLOADS[zname]
    return wl, hidden


def transition_weights(wl: "Workload", hidden: int, affine: bool = False) -> Dict[str, Optional[np.ndarray]]:
    """W1, W2 [hidden, c_z], W3 [c_z, hidden] ~ N(0, 1/fan_in); gamma, beta when affine."""
    c = wl.c_z
    out: Dict[str, Optional[np.ndarray]] = {}
    for name, tid, rows, fan in (("w1", T_TW1, hidden, c), ("w2", T_TW2, hidden, c), ("w3", T_TW3, c, hidden)):
        out[name] = (normal(key(wl.seed, tid), 0, rows * fan) * np.float32(1.0 / np.sqrt(fan))
                     ).astype(np.float32).reshape(rows, fan)
    if affine:
        out["gamma"] = (np.float32(1.0) + np.float32(0.25) * normal(key(wl.seed, T_TGAMMA), 0, c)).astype(np.float32)
        out["beta"] = normal(key(wl.seed, T_TBETA), 0, c)
    else:
        out["gamma"] = out["beta"] = None
    return out


# ----------------------------------------------------------------------------- atom -> token pooling
SCATTER_WORKLOADS = {
    # name: (tokens, channels, feature dtype)
    "pool300_f32": (300, 64, "f32"),
    "pool24000_bf16": (24000, 128, "bf16"),
}


def token_index(n_tokens: int, seed: int = 0) -> np.ndarray:
    """Token of each atom, atoms ordered by token: token t has 4 + word(t) % 11
    atoms (4 .. 14, the heavy-atom counts of residues; mean 9)."""
    counts = (4 + word_np(key(seed, T_ATOMS_PER_TOK), np.arange(n_tokens, dtype=np.uint64)) % np.uint64(11)
              ).astype(np.int64)
    return np.repeat(np.arange(n_tokens, dtype=np.int32), counts)


def atom_features(n_atoms: int, c: int, bf16: bool, seed: int = 0) -> np.ndarray:
    return normal(key(seed, T_AFEAT), 0, n_atoms * c, bf16=bf16).reshape(n_atoms, c)


# ----------------------------------------------------------------------------- kNN workloads
@dataclasses.dataclass(frozen=True)
class KnnWorkload:
    """k nearest neighbours of the query atoms [q_row0, q_row0 + n_q) among all
    L atoms of a synthetic assembly (chains of residues of atoms)."""
    name: str
    n_atoms: int
    k: int
    q_row0: int
    n_q: int
    n_col_blocks: int       # candidate blocks visited in ring order
    per_res: int = 8
    per_chain: int = 1600
    seed: int = 0
    note: str = ""

    @property
    def n_chains(self) -> int:
        return (self.n_atoms + self.per_chain - 1) // self.per_chain


KNN_WORKLOADS: Dict[str, KnnWorkload] = {
    w.name: w
    for w in [
        KnnWorkload("knn300", 300, 128, 0, 300, 1, per_chain=50,
                    note="6 chains of 50 atoms: every query sees every atom"),
        KnnWorkload("knn5000", 5000, 128, 0, 5000, 3, per_chain=1000, note="RFD3's 5000-atom crop, 5 chains"),
        KnnWorkload("knn96k", 96000, 128, 24000, 24000, 4,
                    note="60 chains x 1600 atoms; a 24000-atom query stripe against 4 candidate blocks of 24000"),
    ]
}


def coords(wl: KnnWorkload) -> np.ndarray:
    """Atom coordinates [L, 3] fp32 of the workload's assembly."""
    out = np.empty((wl.n_atoms, 3), dtype=np.float32)
    _host().synth_coords(key(wl.seed, T_XYZ), wl.n_atoms, wl.per_res, wl.per_chain, out.ctypes.data)
    return out


def chain_ids(wl: KnnWorkload) -> np.ndarray:
    return (np.arange(wl.n_atoms) // wl.per_chain).astype(np.int32)


# ----------------------------------------------------------------------------- device twin
_dev_lib = None


def _dev() -> ctypes.CDLL:
    global _dev_lib
    if _dev_lib is None:
        path = os.path.join(_HERE, "libsynth_dev.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        u64, i64, i32, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.synth_dev_z_rows.argtypes = [u64, u64, i64, i64, i32, i64, i64, i32, vp, vp]
        lib.synth_dev_normal.argtypes = [u64, u64, i64, i32, vp, vp]
        lib.synth_dev_copy.argtypes = [vp, vp, i64, vp]
        lib.synth_dev_read.argtypes = [vp, i64, vp, vp]
        lib.synth_dev_read_pattern.argtypes = [vp, i64, i64, i32, vp, vp]
        lib.synth_dev_gather_pattern.argtypes = [vp, vp, i64, vp, i64, i32, vp, vp]
        for f in (lib.synth_dev_z_rows, lib.synth_dev_normal, lib.synth_dev_copy, lib.synth_dev_read,
                  lib.synth_dev_read_pattern, lib.synth_dev_gather_pattern):
            f.restype = ctypes.c_int
        _dev_lib = lib
    return _dev_lib


def z_fill_device(wl: Workload, ptr: int, row0: int, n_rows: int, stream: int) -> None:
    """Write rows [row0, row0+n_rows) of z into device memory at ``ptr``."""
    kz, kb = z_keys(wl)
    rc = _dev().synth_dev_z_rows(kz, kb, wl.z_period, wl.n_tok, wl.c_z, row0, n_rows, int(wl.bf16), ptr, stream)
    if rc != 0:
        raise RuntimeError(f"synth_dev_z_rows failed ({rc})")


def normal_fill_device(k: int, start: int, count: int, bf16: bool, ptr: int, stream: int) -> None:
    rc = _dev().synth_dev_normal(k, start, count, int(bf16), ptr, stream)
    if rc != 0:
        raise RuntimeError(f"synth_dev_normal failed ({rc})")


def device_copy(src: int, dst: int, nbytes: int, stream: int) -> None:
    if _dev().synth_dev_copy(src, dst, nbytes, stream) != 0:
        raise RuntimeError("synth_dev_copy failed")


def device_read_pattern(z: int, n_tok: int, n_rows: int, n_parts: int, sink: int, stream: int) -> None:
    """Reads the 256-B pair vectors of z rows [0, n_rows) in the fused attention
    kernel's order, with no arithmetic (the access pattern's bandwidth ceiling)."""
    if _dev().synth_dev_read_pattern(z, n_tok, n_rows, n_parts, sink, stream) != 0:
        raise RuntimeError("synth_dev_read_pattern failed")


def device_gather_pattern(k: int, v: int, n_atoms: int, nbr: int, n_q: int, n_slots: int, sink: int,
                          stream: int) -> None:
    """Gathers the 256-byte K and V rows of every listed neighbour in the sparse
    attention's pattern, with no arithmetic (that pattern's ceiling)."""
    if _dev().synth_dev_gather_pattern(k, v, n_atoms, nbr, n_q, n_slots, sink, stream) != 0:
        raise RuntimeError("synth_dev_gather_pattern failed")


def device_read(src: int, nbytes: int, sink: int, stream: int) -> None:
    if _dev().synth_dev_read(src, nbytes, sink, stream) != 0:
        raise RuntimeError("synth_dev_read failed")
