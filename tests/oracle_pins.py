"""Pins that tie the fp64 oracle to things other than itself.

Each ``pin_*`` function raises AssertionError when the oracle (whatever
library ``oracle._lib`` currently holds) disagrees with:

* the paper's chunk rule, worked out by hand (tests/golden/chunk_distribution.txt);
* library routines that compute a special case: torch's ``layer_norm`` and
  ``linear`` for the pair bias, torch's ``scaled_dot_product_attention`` for
  the softmax attention with an additive float mask, all in fp64 on the CPU;
* closed forms (uniform attention, a single token, one dominant key, all keys
  masked);
* invariants the definition implies (blocked equals unblocked, per-row bias
  constants and LayerNorm shifts do not matter, token permutation
  equivariance, a masked key equals a deleted one);
* brute force at 40 significant digits on tiny inputs (mpmath).

The k-nearest-neighbour search is pinned to a hand-worked golden file (atoms
on a line), numpy brute force in fp32 with lexicographic (d2, index) order,
integer-lattice ties, the blocked ring merge, merge properties, group modes,
short lists and relabelling.

The pair transition is pinned to its torch composition (layer_norm, linear,
silu), zero-branch and scaling closed forms, the LayerNorm shift, and brute
force at 40 digits.

The atom-to-token mean is pinned to torch's index_reduce("mean") and a numpy
bincount mean, plus closed forms (copies, constants, dropped indices, order).

The sparse (kNN) atom attention has its own pins: torch's SDPA over each
query's gathered keys, the dense pipeline when every atom is a neighbour,
closed forms (one neighbour atom in every slot, all slots empty), slot
permutation, empty slots equal deleted ones, blocked equals unblocked, and
brute force at 40 digits.

``tests/test_oracle_mutants.py`` plants plausible mistakes in copies of the
oracle's C source and checks that every one of them fails at least one pin.
"""
from __future__ import annotations

import os

import mpmath
import numpy as np
import torch
import torch.nn.functional as F

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _case(seed=0, n=9, c_s=6, c_z=8, h=3, d=4, affine=True, mask_frac=0.3, dtype="f32"):
    """Small random case: s, z (all rows), weights, mask."""
    r = _rng(seed)
    s = r.standard_normal((n, c_s)).astype(np.float32)
    z = r.standard_normal((n, n, c_z)).astype(np.float32)
    if dtype == "bf16":
        s = synth.bf16_round(s)
        z = synth.bf16_round(z)
    w = {
        "w_q": (r.standard_normal((h * d, c_s)) / np.sqrt(c_s)).astype(np.float32),
        "w_k": (r.standard_normal((h * d, c_s)) / np.sqrt(c_s)).astype(np.float32),
        "w_v": (r.standard_normal((h * d, c_s)) / np.sqrt(c_s)).astype(np.float32),
        "w_g": (r.standard_normal((h * d, c_s)) / np.sqrt(c_s)).astype(np.float32),
        "w_b": (r.standard_normal((h, c_z)) / np.sqrt(c_z)).astype(np.float32),
        "ln_gamma": (1 + 0.3 * r.standard_normal(c_z)).astype(np.float32) if affine else None,
        "ln_beta": (0.5 * r.standard_normal(c_z)).astype(np.float32) if affine else None,
        "b_b": r.standard_normal(h).astype(np.float32) if affine else None,
    }
    mask = (r.random(n) >= mask_frac).astype(np.uint8)
    mask[r.integers(n)] = 1  # at least one valid key
    return s, z, w, mask


def _torch_pipeline(s, z, w, mask, h, d, eps=1e-5):
    """The definition composed from torch library routines (fp64, CPU)."""
    t = lambda a: None if a is None else torch.from_numpy(oracle.decode(np.asarray(a)) if np.asarray(a).dtype == np.uint16 else np.asarray(a, dtype=np.float64))
    S, Z = t(s), t(z)
    n = S.shape[0]
    c_z = Z.shape[-1]
    q = F.linear(S, t(w["w_q"])).view(n, h, d).transpose(0, 1)
    k = F.linear(S, t(w["w_k"])).view(n, h, d).transpose(0, 1)
    v = F.linear(S, t(w["w_v"])).view(n, h, d).transpose(0, 1)
    g = torch.sigmoid(F.linear(S, t(w["w_g"])))
    ln = F.layer_norm(Z, (c_z,), t(w.get("ln_gamma")), t(w.get("ln_beta")), eps)
    b = F.linear(ln, t(w["w_b"]), t(w.get("b_b")))  # [n, n, h]
    bias = b.permute(2, 0, 1).contiguous()  # [h, i, j]
    if mask is not None:
        bias = bias.masked_fill(torch.from_numpy(mask == 0)[None, None, :], float("-inf"))
    o = F.scaled_dot_product_attention(q.contiguous(), k.contiguous(), v.contiguous(), attn_mask=bias)
    return (g * o.transpose(0, 1).reshape(n, h * d)).numpy()


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ----------------------------------------------------------------------------- chunk rule
def pin_chunk_golden():
    with open(os.path.join(GOLDEN, "chunk_distribution.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            left, right = line.split("|")
            nums = [int(x) for x in left.split()]
            total, parts, sizes = nums[0], nums[1], nums[2:]
            starts = [int(x) for x in right.split()]
            got = [oracle.chunk(total, parts, p) for p in range(parts)]
            assert [g[0] for g in got] == sizes, (total, parts, got)
            assert [g[1] for g in got] == starts, (total, parts, got)


def pin_chunk_properties():
    for total in (1, 2, 7, 100, 4800, 24000, 12347):
        for parts in range(1, min(total, 17) + 1):
            got = [oracle.chunk(total, parts, p) for p in range(parts)]
            sizes = [g[0] for g in got]
            assert sum(sizes) == total
            assert max(sizes) - min(sizes) <= 1
            assert got[0][1] == 0
            for p in range(parts - 1):
                assert got[p + 1][1] == got[p][1] + got[p][0]
            assert sizes == sorted(sizes, reverse=True)


# ----------------------------------------------------------------------------- library pins
def pin_layer_norm_torch():
    """With W_b = I (H = c_z) the bias is LayerNorm(z) itself."""
    r = _rng(1)
    c_z = 12
    z = (3.0 + 2.0 * r.standard_normal((4, 5, c_z))).astype(np.float32)
    gamma = (1 + 0.5 * r.standard_normal(c_z)).astype(np.float32)
    beta = r.standard_normal(c_z).astype(np.float32)
    for eps in (1e-5, 0.3):
        got = oracle.bias(z, np.eye(c_z, dtype=np.float32), None, gamma, beta, eps)
        ref = F.layer_norm(torch.from_numpy(z.astype(np.float64)), (c_z,),
                           torch.from_numpy(gamma.astype(np.float64)), torch.from_numpy(beta.astype(np.float64)),
                           eps).numpy()
        assert _rel(got, ref) <= 1e-12, _rel(got, ref)


def pin_bias_torch():
    for dtype in ("f32", "bf16"):
        s, z, w, _ = _case(2, n=6, c_z=16, h=5, dtype=dtype)
        got = oracle.bias(z, w["w_b"], w["b_b"], w["ln_gamma"], w["ln_beta"], 1e-5)
        Z = torch.from_numpy(oracle.decode(z))
        ref = F.linear(F.layer_norm(Z, (16,), torch.from_numpy(w["ln_gamma"].astype(np.float64)),
                                    torch.from_numpy(w["ln_beta"].astype(np.float64)), 1e-5),
                       torch.from_numpy(w["w_b"].astype(np.float64)),
                       torch.from_numpy(w["b_b"].astype(np.float64))).numpy()
        assert _rel(got, ref) <= 1e-12, _rel(got, ref)


def pin_attend_sdpa():
    """Softmax attention with an explicit bias equals torch SDPA with a float mask."""
    r = _rng(3)
    n_rows, n, h, d = 5, 11, 3, 4
    q = r.standard_normal((n_rows, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    gp = r.standard_normal((n_rows, h * d))
    b = 2.0 * r.standard_normal((n_rows, n, h))
    mask = (r.random(n) > 0.3).astype(np.uint8)
    mask[0] = 1
    got = oracle.attend(q, k, v, gp, b, mask, h, d)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    am = T(b).permute(2, 0, 1).masked_fill(T(mask == 0)[None, None, :], float("-inf"))
    o = F.scaled_dot_product_attention(T(q).view(n_rows, h, d).transpose(0, 1).contiguous(),
                                       T(k).view(n, h, d).transpose(0, 1).contiguous(),
                                       T(v).view(n, h, d).transpose(0, 1).contiguous(), attn_mask=am)
    ref = (torch.sigmoid(T(gp)) * o.transpose(0, 1).reshape(n_rows, h * d)).numpy()
    assert _rel(got, ref) <= 1e-12, _rel(got, ref)


def pin_pipeline_torch():
    """The whole definition equals its composition from torch library routines."""
    for seed, dtype, affine in ((4, "f32", True), (5, "bf16", True), (6, "f32", False)):
        s, z, w, mask = _case(seed, n=10, c_s=7, c_z=8, h=3, d=4, affine=affine, dtype=dtype)
        rows = np.arange(10)
        got = oracle.attention(s, z, rows, mask, w, 3, 4)
        ref = _torch_pipeline(s, z, w, mask, 3, 4)
        assert _rel(got, ref) <= 1e-12, (seed, _rel(got, ref))
    # a row stripe: rows 3..6 of the same tensors
    s, z, w, mask = _case(7, n=10, c_s=7, c_z=8, h=3, d=4)
    rows = np.arange(3, 7)
    got = oracle.attention(s, z[rows], rows, mask, w, 3, 4)
    ref = _torch_pipeline(s, z, w, mask, 3, 4)[rows]
    assert _rel(got, ref) <= 1e-12


# ----------------------------------------------------------------------------- closed forms
def pin_uniform_attention():
    """W_b = 0 and W_q = 0: every valid key gets the same weight."""
    s, z, w, mask = _case(8, n=12, h=2, d=3)
    w = dict(w)
    w["w_b"] = np.zeros_like(w["w_b"])
    w["w_q"] = np.zeros_like(w["w_q"])
    rows = np.arange(12)
    got = oracle.attention(s, z, rows, mask, w, 2, 3)
    S = s.astype(np.float64)
    v = S @ w["w_v"].astype(np.float64).T
    g = 1.0 / (1.0 + np.exp(-(S @ w["w_g"].astype(np.float64).T)))
    ref = g * v[mask == 1].mean(axis=0)[None, :]
    assert _rel(got, ref) <= 1e-13, _rel(got, ref)


def pin_single_token():
    s, z, w, _ = _case(9, n=1, h=2, d=3)
    got = oracle.attention(s, z, [0], None, w, 2, 3)
    S = s.astype(np.float64)
    ref = (1.0 / (1.0 + np.exp(-(S @ w["w_g"].astype(np.float64).T)))) * (S @ w["w_v"].astype(np.float64).T)
    assert _rel(got, ref) <= 1e-14, _rel(got, ref)


def pin_dominant_key():
    r = _rng(10)
    n, h, d = 20, 2, 3
    q = r.standard_normal((1, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    gp = r.standard_normal((1, h * d))
    b = np.zeros((1, n, h))
    b[0, 7, :] = 50.0
    got = oracle.attend(q, k, v, gp, b, None, h, d)
    ref = (1.0 / (1.0 + np.exp(-gp))) * v[7][None, :]
    # every other key's weight is below exp(-50 + spread of q.k/sqrt(d)) < exp(-40)
    tol = (n * np.exp(-40.0) + 1e-15) * np.max(np.abs(v))
    assert np.max(np.abs(got - ref)) <= tol


def pin_all_masked_is_zero():
    s, z, w, _ = _case(11, n=6, h=2, d=3)
    got = oracle.attention(s, z, np.arange(6), np.zeros(6, np.uint8), w, 2, 3)
    assert np.all(got == 0.0)
    got4 = oracle.attention(s, z, np.arange(6), np.zeros(6, np.uint8), w, 2, 3, n_blocks=3)
    assert np.all(got4 == 0.0)


# ----------------------------------------------------------------------------- invariants
def pin_blocked_equals_unblocked():
    s, z, w, mask = _case(12, n=17, h=3, d=4, mask_frac=0.2)
    mask[:6] = 0  # first blocks entirely masked for several partitions
    rows = np.arange(17)
    ref = oracle.attention(s, z, rows, mask, w, 3, 4)
    for nb in (2, 3, 5, 17):
        got, (pm, pl, pa) = oracle.attention(s, z, rows, mask, w, 3, 4, n_blocks=nb, return_parts=True)
        assert _rel(got, ref) <= 1e-12, (nb, _rel(got, ref))
        # each partial's maximum is the block's largest logit (torch logits)
        assert pm.shape == (nb, 3, 17)
        assert np.all(pl[np.isneginf(pm)] == 0.0)


def pin_partial_state_torch():
    """Per-block (m, l, acc) against the torch logits of the same block."""
    s, z, w, mask = _case(13, n=8, h=2, d=3, mask_frac=0.25)
    rows = np.arange(8)
    nb = 3
    _, (pm, pl, pa) = oracle.attention(s, z, rows, mask, w, 2, 3, n_blocks=nb, return_parts=True)
    S, Z = torch.from_numpy(s.astype(np.float64)), torch.from_numpy(z.astype(np.float64))
    q = F.linear(S, torch.from_numpy(w["w_q"].astype(np.float64))).view(8, 2, 3)
    k = F.linear(S, torch.from_numpy(w["w_k"].astype(np.float64))).view(8, 2, 3)
    v = F.linear(S, torch.from_numpy(w["w_v"].astype(np.float64))).view(8, 2, 3)
    ln = F.layer_norm(Z, (8,), torch.from_numpy(w["ln_gamma"].astype(np.float64)),
                      torch.from_numpy(w["ln_beta"].astype(np.float64)), 1e-5)
    b = F.linear(ln, torch.from_numpy(w["w_b"].astype(np.float64)), torch.from_numpy(w["b_b"].astype(np.float64)))
    logits = torch.einsum("ihe,jhe->hij", q, k) / np.sqrt(3.0) + b.permute(2, 0, 1)
    logits = logits.masked_fill(torch.from_numpy(mask == 0)[None, None, :], float("-inf")).numpy()
    vv = v.numpy()
    for p in range(nb):
        size, start = oracle.chunk(8, nb, p)
        blk = logits[:, :, start:start + size]
        m = blk.max(axis=2)
        for h in range(2):
            for i in range(8):
                if np.isneginf(m[h, i]):
                    assert np.isneginf(pm[p, h, i]) and pl[p, h, i] == 0.0
                    continue
                wts = np.exp(blk[h, i] - m[h, i])
                assert abs(pm[p, h, i] - m[h, i]) <= 1e-12 * max(1.0, abs(m[h, i]))
                assert abs(pl[p, h, i] - wts.sum()) <= 1e-12 * wts.sum()
                acc = (wts[:, None] * vv[start:start + size, h, :]).sum(axis=0)
                assert np.max(np.abs(pa[p, i, h] - acc)) <= 1e-12 * max(1.0, np.max(np.abs(acc)))


def pin_merge_identity_and_split():
    r = _rng(14)
    n_rows, h, d = 4, 2, 3
    m = r.standard_normal((3, h, n_rows)) * 3
    l = r.random((3, h, n_rows)) + 0.5
    acc = r.standard_normal((3, n_rows, h, d))
    gate = r.random((n_rows, h * d))
    m_ref, l_ref, a_ref, o_ref = oracle.merge(m, l, acc, gate)
    # an empty partial (-inf, 0, 0) anywhere is the identity
    m2 = np.concatenate([m[:1], np.full((1, h, n_rows), -np.inf), m[1:]])
    l2 = np.concatenate([l[:1], np.zeros((1, h, n_rows)), l[1:]])
    a2 = np.concatenate([acc[:1], np.zeros((1, n_rows, h, d)), acc[1:]])
    _, _, _, o2 = oracle.merge(m2, l2, a2, gate)
    assert _rel(o2, o_ref) <= 1e-15
    # closed form of the merge: weights exp(m_p - max m)
    M = m.max(axis=0)
    wts = np.exp(m - M[None])
    L = (wts * l).sum(axis=0)
    A = (wts.transpose(0, 2, 1)[..., None] * acc).sum(axis=0)
    assert _rel(l_ref, L) <= 1e-14 and np.array_equal(m_ref, M)
    assert _rel(a_ref, A) <= 1e-14
    O = gate * (A / L.T[:, :, None]).reshape(n_rows, h * d)
    assert _rel(o_ref, O) <= 1e-14
    # all-empty merge gives zeros
    _, l0, _, o0 = oracle.merge(np.full((2, h, n_rows), -np.inf), np.zeros((2, h, n_rows)),
                                np.zeros((2, n_rows, h, d)), gate)
    assert np.all(o0 == 0.0) and np.all(l0 == 0.0)


def pin_bias_row_constant():
    """Adding c[i, h] to every key's bias leaves the output unchanged."""
    r = _rng(15)
    n_rows, n, h, d = 4, 9, 3, 2
    q, k, v = r.standard_normal((n_rows, h * d)), r.standard_normal((n, h * d)), r.standard_normal((n, h * d))
    gp, b = r.standard_normal((n_rows, h * d)), r.standard_normal((n_rows, n, h))
    c = 5.0 * r.standard_normal((n_rows, 1, h))
    mask = np.ones(n, np.uint8)
    mask[3] = 0
    a = oracle.attend(q, k, v, gp, b, mask, h, d)
    b2 = oracle.attend(q, k, v, gp, b + c, mask, h, d)
    assert _rel(b2, a) <= 1e-13


def pin_affine_constants_irrelevant():
    """beta and b_b add per-head constants to the bias, so the output ignores them."""
    s, z, w, mask = _case(16, n=8, h=2, d=3)
    w0 = dict(w, ln_beta=None, b_b=None)
    a = oracle.attention(s, z, np.arange(8), mask, w, 2, 3)
    b = oracle.attention(s, z, np.arange(8), mask, w0, 2, 3)
    assert _rel(a, b) <= 1e-13
    # ... but they do change the bias itself
    assert np.max(np.abs(oracle.bias(z, w["w_b"], w["b_b"], w["ln_gamma"], w["ln_beta"])
                         - oracle.bias(z, w["w_b"], None, w["ln_gamma"], None))) > 1e-3


def pin_layer_norm_shift_scale():
    r = _rng(17)
    # values on a 1/64 grid so that the shifted and scaled inputs stay exact in fp32
    zz = (np.round(r.standard_normal((3, 4, 8)) * 64) / 64).astype(np.float32)
    wb = r.standard_normal((2, 8))
    b0 = oracle.bias(zz, wb)
    b_shift = oracle.bias((zz + np.float32(7.25)).astype(np.float32), wb)  # LN(z + c) = LN(z)
    assert _rel(b_shift, b0) <= 1e-13
    b_scale = oracle.bias((zz * np.float32(4.0)).astype(np.float32), wb, eps=1e-5 * 16)
    assert _rel(b_scale, oracle.bias(zz, wb, eps=1e-5)) <= 1e-13


def pin_permutation_equivariance():
    s, z, w, mask = _case(18, n=10, h=2, d=3)
    perm = _rng(19).permutation(10)
    a = oracle.attention(s, z, np.arange(10), mask, w, 2, 3)
    zp = np.ascontiguousarray(z[perm][:, perm])
    b = oracle.attention(np.ascontiguousarray(s[perm]), zp, np.arange(10), mask[perm], w, 2, 3)
    assert _rel(b, a[perm]) <= 1e-13


def pin_masked_equals_deleted():
    s, z, w, mask = _case(20, n=9, h=2, d=3, mask_frac=0.0)
    mask = np.ones(9, np.uint8)
    mask[[2, 5]] = 0
    keep = np.flatnonzero(mask)
    a = oracle.attention(s, z, np.arange(9), mask, w, 2, 3)
    sub = oracle.attention(np.ascontiguousarray(s[keep]), np.ascontiguousarray(z[keep][:, keep]),
                           np.arange(len(keep)), None, w, 2, 3)
    assert _rel(a[keep], sub) <= 1e-13
    z2 = z.copy()
    z2[:, [2, 5], :] = 1e3 * _rng(21).standard_normal((9, 2, z.shape[2])).astype(np.float32)
    b = oracle.attention(s, z2, np.arange(9), mask, w, 2, 3)
    assert np.array_equal(a, b)


# ----------------------------------------------------------------------------- brute force
def pin_bruteforce_mpmath():
    """The definition at 40 digits on tiny inputs."""
    mpmath.mp.dps = 40
    for seed, n, c_s, c_z, h, d in ((22, 4, 3, 5, 2, 3), (23, 5, 2, 6, 1, 4), (24, 3, 4, 3, 2, 2)):
        s, z, w, mask = _case(seed, n=n, c_s=c_s, c_z=c_z, h=h, d=d, mask_frac=0.2)
        got = oracle.attention(s, z, np.arange(n), mask, w, h, d)
        M = lambda a: [[mpmath.mpf(float(x)) for x in row] for row in np.atleast_2d(a)]
        S, Wq, Wk, Wv, Wg, Wb = (M(a) for a in (s, w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"]))
        gam = [mpmath.mpf(float(x)) for x in w["ln_gamma"]]
        bet = [mpmath.mpf(float(x)) for x in w["ln_beta"]]
        bb = [mpmath.mpf(float(x)) for x in w["b_b"]]
        eps = mpmath.mpf(1e-5)
        lin = lambda W, x: [mpmath.fsum(W[o][c] * x[c] for c in range(len(x))) for o in range(len(W))]
        for i in range(n):
            qi, gi = lin(Wq, S[i]), [1 / (1 + mpmath.exp(-t)) for t in lin(Wg, S[i])]
            for hh in range(h):
                logits = []
                for j in range(n):
                    if not mask[j]:
                        continue
                    zz = [mpmath.mpf(float(x)) for x in z[i, j]]
                    mu = mpmath.fsum(zz) / c_z
                    var = mpmath.fsum((x - mu) ** 2 for x in zz) / c_z
                    lnv = [gam[c] * (zz[c] - mu) / mpmath.sqrt(var + eps) + bet[c] for c in range(c_z)]
                    b = mpmath.fsum(Wb[hh][c] * lnv[c] for c in range(c_z)) + bb[hh]
                    kj = lin(Wk, S[j])
                    dot = mpmath.fsum(qi[hh * d + e] * kj[hh * d + e] for e in range(d))
                    logits.append((j, dot / mpmath.sqrt(d) + b))
                mx = max(x for _, x in logits)
                wts = [(j, mpmath.exp(x - mx)) for j, x in logits]
                den = mpmath.fsum(x for _, x in wts)
                for e in range(d):
                    num = mpmath.fsum(x * lin(Wv, S[j])[hh * d + e] for j, x in wts)
                    ref = gi[hh * d + e] * num / den
                    assert abs(float(ref) - got[i, hh * d + e]) <= 1e-13 * max(1.0, abs(float(ref))), (seed, i, hh, e)


# ----------------------------------------------------------------------------- sparse kNN attention
def _sparse_case(seed=0, L=11, c_atom=6, c_ap=5, h=2, d=3, k=7, n_rows=5, empty_frac=0.25, affine=True):
    """Small random sparse case: A, gathered P slices, neighbour lists (repeats
    allowed), query rows, weights."""
    r = _rng(seed)
    a = r.standard_normal((L, c_atom)).astype(np.float32)
    rows = r.choice(L, n_rows, replace=False)
    nbr = r.integers(0, L, (n_rows, k)).astype(np.int32)
    nbr[r.random((n_rows, k)) < empty_frac] = -1
    nbr[:, 0] = r.integers(0, L, n_rows)  # every query keeps a neighbour
    p = r.standard_normal((n_rows, k, c_ap)).astype(np.float32)
    w = {
        "w_q": (r.standard_normal((h * d, c_atom)) / np.sqrt(c_atom)).astype(np.float32),
        "w_k": (r.standard_normal((h * d, c_atom)) / np.sqrt(c_atom)).astype(np.float32),
        "w_v": (r.standard_normal((h * d, c_atom)) / np.sqrt(c_atom)).astype(np.float32),
        "w_g": (r.standard_normal((h * d, c_atom)) / np.sqrt(c_atom)).astype(np.float32),
        "w_b": (r.standard_normal((h, c_ap)) / np.sqrt(c_ap)).astype(np.float32),
        "ln_gamma": (1 + 0.3 * r.standard_normal(c_ap)).astype(np.float32) if affine else None,
        "ln_beta": (0.5 * r.standard_normal(c_ap)).astype(np.float32) if affine else None,
        "b_b": r.standard_normal(h).astype(np.float32) if affine else None,
    }
    return a, p, nbr, rows, w


def _torch_sparse(a, p, nbr, rows, w, h, d, eps=1e-5):
    """Per query: gather K, V at the neighbour indices, bias from torch's
    layer_norm + linear on the gathered P slices, then torch's SDPA with -inf at
    empty slots, then the gate (fp64, CPU)."""
    t = lambda x: None if x is None else torch.from_numpy(np.asarray(x, dtype=np.float64))
    A = t(a)
    L = A.shape[0]
    K = F.linear(A, t(w["w_k"])).view(L, h, d)
    V = F.linear(A, t(w["w_v"])).view(L, h, d)
    out = []
    for r, i in enumerate(rows):
        q = F.linear(A[i], t(w["w_q"])).view(h, 1, d)
        g = torch.sigmoid(F.linear(A[i], t(w["w_g"])))
        j = torch.from_numpy(np.asarray(nbr[r], dtype=np.int64))
        valid = (j >= 0) & (j < L)
        jj = torch.where(valid, j, torch.zeros_like(j))
        P = t(p[r])
        b = F.linear(F.layer_norm(P, (P.shape[-1],), t(w.get("ln_gamma")), t(w.get("ln_beta")), eps),
                     t(w["w_b"]), t(w.get("b_b")))  # [k, h]
        bias = b.t().masked_fill(~valid[None, :], float("-inf"))[:, None, :]  # [h, 1, k]
        o = F.scaled_dot_product_attention(q, K[jj].transpose(0, 1).contiguous(), V[jj].transpose(0, 1).contiguous(),
                                           attn_mask=bias)
        out.append((g * o.reshape(h * d)).numpy())
    return np.stack(out)


def pin_sparse_sdpa_torch():
    for seed, kw in ((40, {}), (41, dict(L=20, k=13, n_rows=8, h=3, d=2)), (42, dict(affine=False, empty_frac=0.6))):
        a, p, nbr, rows, w = _sparse_case(seed, **kw)
        h, d = w["w_b"].shape[0], w["w_q"].shape[0] // w["w_b"].shape[0]
        got = oracle.sparse_attention(a, p, nbr, rows, w, h, d)
        ref = _torch_sparse(a, p, nbr, rows, w, h, d)
        assert _rel(got, ref) <= 1e-12, (seed, _rel(got, ref))


def pin_sparse_full_neighbourhood_is_dense():
    """Every atom a neighbour, slot t = atom t, P slices = rows of a pair
    tensor: the token path's definition, composed from torch routines, with
    masked keys as empty slots."""
    s, z, w, mask = _case(43, n=10, c_s=5, c_z=6, h=2, d=3)
    rows = np.array([0, 3, 9, 4])
    nbr = np.tile(np.where(mask == 1, np.arange(10), -1).astype(np.int32), (len(rows), 1))
    got = oracle.sparse_attention(s, z[rows], nbr, rows, w, 2, 3)
    ref = _torch_pipeline(s, z, w, mask, 2, 3)[rows]
    assert _rel(got, ref) <= 1e-12, _rel(got, ref)


def pin_sparse_one_neighbour_atom():
    """All slots on one atom j (different pair slices): out = g * v_j."""
    a, p, nbr, rows, w = _sparse_case(44, affine=True, empty_frac=0.0)
    jstar = np.array([3, 7, 0, 10, 5], dtype=np.int32)
    nbr[:] = jstar[:, None]
    nbr[1, 2:4] = -1
    got = oracle.sparse_attention(a, p, nbr, rows, w, 2, 3)
    A = a.astype(np.float64)
    v = A[jstar] @ w["w_v"].astype(np.float64).T
    g = 1.0 / (1.0 + np.exp(-(A[rows] @ w["w_g"].astype(np.float64).T)))
    assert _rel(got, g * v) <= 1e-13, _rel(got, g * v)


def pin_sparse_all_empty_is_zero():
    a, p, nbr, rows, w = _sparse_case(45)
    nbr[2, :] = -1
    nbr[4, :] = 11  # == L: not an atom
    got = oracle.sparse_attention(a, p, nbr, rows, w, 2, 3)
    assert np.all(got[2] == 0.0) and np.all(got[4] == 0.0)
    assert np.all(np.abs(got[0]) > 0.0)


def pin_sparse_slot_permutation():
    a, p, nbr, rows, w = _sparse_case(46, k=9)
    base = oracle.sparse_attention(a, p, nbr, rows, w, 2, 3)
    perm = _rng(47).permutation(9)
    got = oracle.sparse_attention(a, p[:, perm], nbr[:, perm], rows, w, 2, 3)
    assert _rel(got, base) <= 1e-13


def pin_sparse_empty_equals_deleted():
    a, p, nbr, rows, w = _sparse_case(48, k=8, empty_frac=0.0)
    nb = nbr.copy()
    nb[:, 5] = -1
    nb[1, 2] = 1000  # out of range counts as empty too
    got = oracle.sparse_attention(a, p, nb, rows, w, 2, 3)
    keep = [t for t in range(8) if t != 5]
    ref = np.empty_like(got)
    for r in range(len(rows)):
        kk = [t for t in keep if not (r == 1 and t == 2)]
        ref[r] = oracle.sparse_attention(a, p[r:r + 1, kk], nbr[r:r + 1, kk], rows[r:r + 1], w, 2, 3)[0]
    assert np.array_equal(got, ref) or _rel(got, ref) <= 1e-14


def pin_sparse_blocked_equals_unblocked():
    a, p, nbr, rows, w = _sparse_case(49, L=23, k=15, n_rows=9)
    base = oracle.sparse_attention(a, p, nbr, rows, w, 2, 3)
    for nb in (2, 3, 7, 23):
        got = oracle.sparse_attention(a, p, nbr, rows, w, 2, 3, n_blocks=nb)
        assert _rel(got, base) <= 1e-12, nb


def pin_sparse_affine_constants_irrelevant():
    a, p, nbr, rows, w = _sparse_case(50)
    w0 = dict(w, ln_beta=None, b_b=None)
    assert _rel(oracle.sparse_attention(a, p, nbr, rows, w, 2, 3),
                oracle.sparse_attention(a, p, nbr, rows, w0, 2, 3)) <= 1e-13


def pin_sparse_bruteforce_mpmath():
    """The sparse definition at 40 digits on tiny inputs."""
    mpmath.mp.dps = 40
    for seed, kw in ((51, dict(L=6, c_atom=3, c_ap=4, h=2, d=2, k=4, n_rows=3)),
                     (52, dict(L=5, c_atom=4, c_ap=3, h=1, d=3, k=5, n_rows=2))):
        a, p, nbr, rows, w = _sparse_case(seed, **kw)
        h, d = kw["h"], kw["d"]
        got = oracle.sparse_attention(a, p, nbr, rows, w, h, d)
        M = lambda x: [[mpmath.mpf(float(v)) for v in row] for row in np.atleast_2d(x)]
        A, Wq, Wk, Wv, Wg, Wb = (M(x) for x in (a, w["w_q"], w["w_k"], w["w_v"], w["w_g"], w["w_b"]))
        gam = [mpmath.mpf(float(x)) for x in w["ln_gamma"]]
        bet = [mpmath.mpf(float(x)) for x in w["ln_beta"]]
        bb = [mpmath.mpf(float(x)) for x in w["b_b"]]
        eps = mpmath.mpf(1e-5)
        c_ap = kw["c_ap"]
        lin = lambda W, x: [mpmath.fsum(W[o][c] * x[c] for c in range(len(x))) for o in range(len(W))]
        for r, i in enumerate(rows):
            qi, gi = lin(Wq, A[i]), [1 / (1 + mpmath.exp(-t)) for t in lin(Wg, A[i])]
            for hh in range(h):
                logits = []
                for t in range(kw["k"]):
                    j = int(nbr[r, t])
                    if j < 0:
                        continue
                    pp = [mpmath.mpf(float(x)) for x in p[r, t]]
                    mu = mpmath.fsum(pp) / c_ap
                    var = mpmath.fsum((x - mu) ** 2 for x in pp) / c_ap
                    lnv = [gam[c] * (pp[c] - mu) / mpmath.sqrt(var + eps) + bet[c] for c in range(c_ap)]
                    b = mpmath.fsum(Wb[hh][c] * lnv[c] for c in range(c_ap)) + bb[hh]
                    kj = lin(Wk, A[j])
                    dot = mpmath.fsum(qi[hh * d + e] * kj[hh * d + e] for e in range(d))
                    logits.append((j, dot / mpmath.sqrt(d) + b))
                mx = max(x for _, x in logits)
                wts = [(j, mpmath.exp(x - mx)) for j, x in logits]
                den = mpmath.fsum(x for _, x in wts)
                for e in range(d):
                    num = mpmath.fsum(x * lin(Wv, A[j])[hh * d + e] for j, x in wts)
                    ref = gi[hh * d + e] * num / den
                    assert abs(float(ref) - got[r, hh * d + e]) <= 1e-13 * max(1.0, abs(float(ref))), (seed, r, hh, e)


# ----------------------------------------------------------------------------- k nearest neighbours
def _knn_numpy(x_q, x_c, k, keep=None):
    """Brute force: squared distances in fp32 numpy arithmetic (each operation
    rounded), candidates sorted by (d2, index)."""
    out_i = np.full((len(x_q), k), -1, dtype=np.int32)
    out_d = np.full((len(x_q), k), np.inf, dtype=np.float32)
    for r, q in enumerate(np.asarray(x_q, dtype=np.float32)):
        d = np.asarray(x_c, dtype=np.float32) - q[None, :]
        d2 = (d[:, 0] * d[:, 0] + d[:, 1] * d[:, 1]) + d[:, 2] * d[:, 2]
        j = np.arange(len(x_c))
        if keep is not None:
            m = keep(r)
            d2, j = d2[m], j[m]
        order = np.lexsort((j, d2))[:k]
        out_i[r, :len(order)] = j[order]
        out_d[r, :len(order)] = d2[order]
    return out_i, out_d


def _coords(seed, n, scale=10.0):
    return (_rng(seed).standard_normal((n, 3)) * scale).astype(np.float32)


def pin_knn_golden_line():
    with open(os.path.join(GOLDEN, "knn_line.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            pos, q, k, want = (part.split() for part in line.split("|"))
            x = np.zeros((len(pos), 3), dtype=np.float32)
            x[:, 0] = [float(p) for p in pos]
            q, k = int(q[0]), int(k[0])
            idx, d2 = oracle.knn(x[q:q + 1], x, k)
            assert idx[0].tolist() == [int(w) for w in want], (line, idx[0])
            for t, w in enumerate(int(w) for w in want):
                assert d2[0, t] == ((x[w, 0] - x[q, 0]) ** 2 if w >= 0 else np.inf)


def pin_knn_numpy_bruteforce():
    for seed, n, k in ((60, 300, 16), (61, 1000, 128), (62, 40, 64)):
        x = _coords(seed, n)
        q = np.arange(0, n, 7)
        idx, d2 = oracle.knn(x[q], x, k)
        ri, rd = _knn_numpy(x[q], x, k)
        assert np.array_equal(idx, ri) and np.array_equal(d2, rd), seed


def pin_knn_ties_by_index():
    """Many equal distances (integer lattice): ties go to the smaller index."""
    g = np.stack(np.meshgrid(np.arange(4), np.arange(4), np.arange(4), indexing="ij"), -1).reshape(-1, 3)
    x = g.astype(np.float32)
    perm = _rng(63).permutation(len(x))
    x = x[perm]
    idx, d2 = oracle.knn(x, x, 20)
    ri, rd = _knn_numpy(x, x, 20)
    assert np.array_equal(idx, ri) and np.array_equal(d2, rd)


def pin_knn_blocked_ring_merge():
    x = _coords(64, 500)
    q = np.arange(3, 500, 11)
    base = oracle.knn(x[q], x, 32)
    for nb in (2, 3, 7, 64):
        got = oracle.knn(x[q], x, 32, n_blocks=nb)
        assert np.array_equal(got[0], base[0]) and np.array_equal(got[1], base[1]), nb


def pin_knn_merge_properties():
    x = _coords(65, 200)
    q = x[:9]
    a = oracle.knn(q, x[:80], 24, c_index0=0)
    b = oracle.knn(q, x[80:], 24, c_index0=80)
    m = oracle.topk_merge(*a, *b)
    full = _knn_numpy(q, x, 24)
    assert np.array_equal(m[0], full[0]) and np.array_equal(m[1], full[1])
    m2 = oracle.topk_merge(*b, *a)
    assert np.array_equal(m2[0], m[0])
    empty = (np.full_like(a[0], -1), np.full_like(a[1], np.inf))
    e = oracle.topk_merge(*a, *empty)
    assert np.array_equal(e[0], a[0]) and np.array_equal(e[1], a[1])


def pin_knn_groups():
    x = _coords(66, 400)
    grp = (np.arange(400) // 50).astype(np.int32)
    q = np.arange(5, 400, 13)
    for mode, keep in ((1, lambda r: grp == grp[q[r]]), (2, lambda r: grp != grp[q[r]])):
        idx, d2 = oracle.knn(x[q], x, 30, group_q=grp[q], group_c=grp, group_mode=mode)
        ri, rd = _knn_numpy(x[q], x, 30, keep=keep)
        assert np.array_equal(idx, ri) and np.array_equal(d2, rd), mode


def pin_knn_short_lists_and_permutation():
    x = _coords(67, 12)
    idx, d2 = oracle.knn(x, x, 20)
    assert (idx[:, 12:] == -1).all() and np.isinf(d2[:, 12:]).all()
    assert sorted(idx[0, :12].tolist()) == list(range(12)) and idx[0, 0] == 0
    # relabelling the candidates relabels the answer (no ties in random data)
    y = _coords(68, 300)
    perm = _rng(69).permutation(300)
    a = oracle.knn(y[:10], y, 25)[0]
    b = oracle.knn(y[:10], y[perm], 25)[0]
    assert np.array_equal(perm[b], a)


# ----------------------------------------------------------------------------- pair transition
def _transition_case(seed=0, n=7, c_z=6, hidden=10, affine=True):
    r = _rng(seed)
    z = (0.5 + r.standard_normal((n, c_z))).astype(np.float32)
    w = {
        "w1": (r.standard_normal((hidden, c_z)) / np.sqrt(c_z)).astype(np.float32),
        "w2": (r.standard_normal((hidden, c_z)) / np.sqrt(c_z)).astype(np.float32),
        "w3": (r.standard_normal((c_z, hidden)) / np.sqrt(hidden)).astype(np.float32),
        "gamma": (1 + 0.3 * r.standard_normal(c_z)).astype(np.float32) if affine else None,
        "beta": (0.4 * r.standard_normal(c_z)).astype(np.float32) if affine else None,
    }
    return z, w


def pin_transition_torch():
    """The update composed from torch's layer_norm, linear and silu (fp64)."""
    for seed, kw in ((70, {}), (71, dict(n=20, c_z=16, hidden=64)), (72, dict(affine=False))):
        z, w = _transition_case(seed, **kw)
        got = oracle.transition(z, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
        t = lambda a: None if a is None else torch.from_numpy(np.asarray(a, dtype=np.float64))
        Z = t(z)
        N = F.layer_norm(Z, (Z.shape[-1],), t(w["gamma"]), t(w["beta"]), 1e-5)
        ref = (Z + F.linear(F.silu(F.linear(N, t(w["w1"]))) * F.linear(N, t(w["w2"])), t(w["w3"]))).numpy()
        assert _rel(got, ref) <= 1e-13, seed


def pin_transition_zero_branches():
    """W1 = 0 (SiLU(0) = 0), W2 = 0 or W3 = 0: the update is the identity."""
    z, w = _transition_case(73)
    for name in ("w1", "w2", "w3"):
        ww = dict(w)
        ww[name] = np.zeros_like(w[name])
        got = oracle.transition(z, ww["w1"], ww["w2"], ww["w3"], ww["gamma"], ww["beta"])
        assert np.array_equal(got, z.astype(np.float64)), name


def pin_transition_silu_branch_and_scaling():
    """SiLU sits on the W1 branch (swapping W1 and W2 changes the result), and
    T is linear in W3 and in W2 (scaling either by 2 doubles T)."""
    z, w = _transition_case(74)
    base = oracle.transition(z, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"]) - z
    swapped = oracle.transition(z, w["w2"], w["w1"], w["w3"], w["gamma"], w["beta"]) - z
    assert _rel(swapped, base) > 1e-3
    for name in ("w2", "w3"):
        ww = dict(w)
        ww[name] = 2 * w[name]
        got = oracle.transition(z, ww["w1"], ww["w2"], ww["w3"], ww["gamma"], ww["beta"]) - z
        assert _rel(got, 2 * base) <= 1e-13, name


def pin_transition_layernorm_shift():
    """LN(z + c) = LN(z): adding a constant to every channel of a pair adds
    exactly that constant to the output."""
    z, w = _transition_case(75, affine=True)
    z = (np.round(z * 64) / 64).astype(np.float32)  # on a grid where z + 3 is exact in fp32
    a = oracle.transition(z, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
    b = oracle.transition(z + np.float32(3.0), w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
    assert np.max(np.abs((b - 3.0) - a)) <= 1e-9


def pin_transition_bruteforce_mpmath():
    mpmath.mp.dps = 40
    z, w = _transition_case(76, n=3, c_z=4, hidden=5)
    got = oracle.transition(z, w["w1"], w["w2"], w["w3"], w["gamma"], w["beta"])
    M = lambda a: [[mpmath.mpf(float(x)) for x in row] for row in np.atleast_2d(a)]
    W1, W2, W3 = M(w["w1"]), M(w["w2"]), M(w["w3"])
    gam = [mpmath.mpf(float(x)) for x in w["gamma"]]
    bet = [mpmath.mpf(float(x)) for x in w["beta"]]
    eps = mpmath.mpf(1e-5)
    for p in range(3):
        x = [mpmath.mpf(float(v)) for v in z[p]]
        mu = mpmath.fsum(x) / 4
        var = mpmath.fsum((v - mu) ** 2 for v in x) / 4
        nn = [gam[c] * (x[c] - mu) / mpmath.sqrt(var + eps) + bet[c] for c in range(4)]
        h = []
        for u in range(5):
            a = mpmath.fsum(W1[u][c] * nn[c] for c in range(4))
            b = mpmath.fsum(W2[u][c] * nn[c] for c in range(4))
            h.append(a / (1 + mpmath.exp(-a)) * b)
        for c in range(4):
            ref = x[c] + mpmath.fsum(W3[c][u] * h[u] for u in range(5))
            assert abs(float(ref) - got[p, c]) <= 1e-13 * max(1.0, abs(float(ref))), (p, c)


# ----------------------------------------------------------------------------- atom -> token mean
def pin_scatter_mean_torch_and_numpy():
    """torch's index_reduce("mean", include_self=False) and a numpy bincount
    mean (fp64); tokens without atoms are 0."""
    r = _rng(80)
    for n_atoms, n_tok, c in ((50, 9, 3), (400, 37, 16), (7, 12, 5)):
        a = r.standard_normal((n_atoms, c)).astype(np.float32)
        idx = r.integers(0, n_tok, n_atoms).astype(np.int32)
        got = oracle.scatter_mean(a, idx, n_tok)
        out = torch.zeros((n_tok, c), dtype=torch.float64)
        out.index_reduce_(0, torch.from_numpy(idx.astype(np.int64)), torch.from_numpy(a.astype(np.float64)), "mean",
                          include_self=False)
        assert _rel(got, out.numpy()) <= 1e-13
        cnt = np.bincount(idx, minlength=n_tok)
        sums = np.stack([np.bincount(idx, weights=a[:, k].astype(np.float64), minlength=n_tok) for k in range(c)], 1)
        ref = np.where(cnt[:, None] > 0, sums / np.maximum(cnt, 1)[:, None], 0.0)
        assert _rel(got, ref) <= 1e-13
        assert np.all(got[cnt == 0] == 0.0)


def pin_scatter_mean_closed_forms():
    """One atom per token copies it; constant features average to the
    constant; out-of-range indices belong to no token; atom order is
    irrelevant up to rounding."""
    r = _rng(81)
    a = r.standard_normal((20, 4)).astype(np.float32)
    perm = r.permutation(20).astype(np.int32)
    got = oracle.scatter_mean(a, perm, 20)
    assert np.array_equal(got[perm], a.astype(np.float64))
    b = np.full((30, 3), 2.5, dtype=np.float32)
    assert np.all(oracle.scatter_mean(b, r.integers(0, 4, 30).astype(np.int32), 4)[:, 0] <= 2.5)
    idx = r.integers(0, 4, 30).astype(np.int32)
    m = oracle.scatter_mean(b, idx, 4)
    assert np.array_equal(m[np.bincount(idx, minlength=4) > 0], np.full((int((np.bincount(idx, minlength=4) > 0).sum()), 3), 2.5))
    feats = np.vstack([a, a[:10]])  # 30 atoms
    idx2 = idx.copy()
    idx2[:5] = [-1, 4, 100, -7, 4]
    keep = (idx2 >= 0) & (idx2 < 4)
    assert np.array_equal(oracle.scatter_mean(feats, idx2, 4), oracle.scatter_mean(feats[keep], idx2[keep], 4))
    q = r.permutation(30)
    c = r.standard_normal((30, 6)).astype(np.float32)
    assert _rel(oracle.scatter_mean(c[q], idx[q], 4), oracle.scatter_mean(c, idx, 4)) <= 1e-14


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
