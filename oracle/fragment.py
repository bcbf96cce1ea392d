"""Literal fragmentation, defragmentation, stuffing and trimming -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg use this module;
the GPU library never imports it.

Everything here follows the paper's definitions in the paper's 1-based notation,
translated to 0-based numpy indices only at the array boundary:

* vectorisation vec_{a x b} and its inverse (Definition "vectorization", Sect. 4.1):
  vec stacks the columns of an a x b matrix on top of each other;
* fragmentation Frag_k: M^{kq x s} -> M^{q x ks}, defined as
  ( vec^{-1}_{ks x q}( vec_{s x kq}( xi^T ) ) )^T  (Definition "fragmentation");
* defragmentation Defrag_k: M^{q x ks} -> M^{kq x s}, defined as
  ( vec^{-1}_{s x kq}( vec_{ks x q}( xi^T ) ) )^T  (Definition after it);
* the closed-form index maps of Lemma "frag-ops" and Lemma "defrag-ops"
  (Sect. 4.1) and the simplified defragmentation map of the appendix lemma, each
  written out separately so that the tests can compare them with the literal
  definitions;
* Stuff_r appends r copies of a dummy sample, Trim_r removes the final r samples
  (Definition "stuff-trim", Sect. 4.3).

A fragmented signal is a matrix whose rows are samples and whose columns are
fragments.  Multi-channel 2-D tensors are fragmented per spatial axis; the two
fragment indices are linearised row-major, (row-fragment, col-fragment), which is
the reading this project takes of the collapse into one image-index dimension in
Sect. 6.1.
"""
from __future__ import annotations

import numpy as np


# ----------------------------------------------------------------------------- 1-D operators

def vec(xi):
    """vec_{a x b}: entry j (1-based) is xi[rem(j-1, a)+1, div(j-1, a)+1]."""
    a, b = xi.shape
    out = np.empty(a * b, dtype=xi.dtype)
    for j in range(1, a * b + 1):
        out[j - 1] = xi[(j - 1) % a, (j - 1) // a]
    return out


def vec_inv(v, a, b):
    """vec^{-1}_{a x b}: entry (i, j) (1-based) is v[(j-1)*a + i]."""
    assert v.shape == (a * b,)
    out = np.empty((a, b), dtype=v.dtype)
    for i in range(1, a + 1):
        for j in range(1, b + 1):
            out[i - 1, j - 1] = v[(j - 1) * a + i - 1]
    return out


def frag(xi, k):
    """Frag_k on a (kq x s) matrix, straight from the definition."""
    kq, s = xi.shape
    assert kq % k == 0, "Frag_k needs a row count divisible by k"
    q = kq // k
    return vec_inv(vec(xi.T), k * s, q).T


def defrag(xi, k):
    """Defrag_k on a (q x ks) matrix, straight from the definition."""
    q, ks = xi.shape
    assert ks % k == 0, "Defrag_k needs a column count divisible by k"
    s = ks // k
    return vec_inv(vec(xi.T), s, k * q).T


def frag_closed(xi, k):
    """Lemma frag-ops: Frag_k(xi)[mu, nu] = xi[div((mu-1)ks+nu-1, s)+1, rem((mu-1)ks+nu-1, s)+1]."""
    kq, s = xi.shape
    q = kq // k
    out = np.empty((q, k * s), dtype=xi.dtype)
    for mu in range(1, q + 1):
        for nu in range(1, k * s + 1):
            t = (mu - 1) * k * s + nu - 1
            out[mu - 1, nu - 1] = xi[t // s, t % s]
    return out


def defrag_closed(xi, k):
    """Lemma defrag-ops: Defrag_k(xi)[mu, nu] = xi[div((mu-1)s+nu-1, ks)+1, rem((mu-1)s+nu-1, ks)+1]."""
    q, ks = xi.shape
    s = ks // k
    out = np.empty((k * q, s), dtype=xi.dtype)
    for mu in range(1, k * q + 1):
        for nu in range(1, s + 1):
            t = (mu - 1) * s + nu - 1
            out[mu - 1, nu - 1] = xi[t // ks, t % ks]
    return out


def defrag_simplified(xi, k):
    """Appendix lemma: Defrag_k(xi)[mu, nu] = xi[div(mu-1, k)+1, rem(mu-1, k)*s + nu]."""
    q, ks = xi.shape
    s = ks // k
    out = np.empty((k * q, s), dtype=xi.dtype)
    for mu in range(1, k * q + 1):
        for nu in range(1, s + 1):
            out[mu - 1, nu - 1] = xi[(mu - 1) // k, ((mu - 1) % k) * s + nu - 1]
    return out


def stuff(xi, r, zeta):
    """Stuff_r: append r copies of the dummy sample zeta (along axis 0)."""
    pad = np.full((r,) + xi.shape[1:], zeta, dtype=xi.dtype)
    return np.concatenate([xi, pad], axis=0)


def trim(xi, r):
    """Trim_r: remove the final r samples (along axis 0)."""
    assert xi.shape[0] >= r + 1
    return xi[: xi.shape[0] - r]


# ----------------------------------------------------------------------------- tensors

def _perm(op, rows, cols, k):
    """The permutation that a 1-D operator applies to a rows x cols matrix,
    obtained by running the literal operator on a matrix of flat indices."""
    idx = np.arange(rows * cols, dtype=np.int64).reshape(rows, cols)
    return op(idx, k)


def _apply_axis(x, op, k, frag_axis, sample_axis):
    """Apply a 1-D operator to every (samples x fragments) matrix of a tensor."""
    xm = np.moveaxis(x, (sample_axis, frag_axis), (-2, -1))
    rows, cols = xm.shape[-2:]
    p = _perm(op, rows, cols, k)
    flat = xm.reshape(xm.shape[:-2] + (rows * cols,))
    res = flat[..., p.reshape(-1)].reshape(xm.shape[:-2] + p.shape)
    return np.moveaxis(res, (-2, -1), (sample_axis, frag_axis))


def frag_tensor(x, kh, kw, Sh, Sw):
    """Frag on a tensor in the library's planar fragment layout.

    x: [Sh*Sw][C][H][W] (Sh row-fragments x Sw col-fragments, linearised row-major)
    returns [(kh*Sh)*(kw*Sw)][C][H/kh][W/kw]: Frag_kh along rows, then Frag_kw along
    columns, each applied literally to every (samples x fragments) matrix."""
    S, C, H, W = x.shape
    assert S == Sh * Sw
    t = x.reshape(Sh, Sw, C, H, W)
    t = _apply_axis(t, frag, kh, frag_axis=0, sample_axis=3)
    t = _apply_axis(t, frag, kw, frag_axis=1, sample_axis=4)
    return np.ascontiguousarray(t.reshape(kh * Sh * kw * Sw, C, H // kh, W // kw))


def defrag_tensor(x, kh, kw, Sh, Sw):
    """Inverse of frag_tensor: [(kh*Sh)*(kw*Sw)][C][H][W] -> [Sh*Sw][C][H*kh][W*kw]."""
    F, C, H, W = x.shape
    assert F == kh * Sh * kw * Sw
    t = x.reshape(kh * Sh, kw * Sw, C, H, W)
    t = _apply_axis(t, defrag, kh, frag_axis=0, sample_axis=3)
    t = _apply_axis(t, defrag, kw, frag_axis=1, sample_axis=4)
    return np.ascontiguousarray(t.reshape(Sh * Sw, C, H * kh, W * kw))
