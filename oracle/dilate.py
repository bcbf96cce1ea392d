"""Dilated evaluation of a processing chain -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg use this module;
the GPU library never imports it.  Everything is double precision numpy,
written from the appendix on functions applied in a dilated fashion:

* `dilated_subsignal(xi, d, k, i)`: Definition "dilatedsubsignal" -- d samples
  of xi starting at sample i (1-based) and k samples apart;
* `dilate(f, xi, c, k)`: Definition "dilate" -- f applied to every feasible
  dilated subsignal of c samples with stride k, results stored contiguously
  (dim(xi) - k(c - 1) of them);
* `eval_dilate(layers, x, upto)`: Definition "evaldilate" -- layer j applies its
  convolution f_j and its pooling kernel g_j both in a dilated fashion with the
  stride k*_{j-1} of the previous layer, per axis on 2-D signals (Sect. 6.1).
  No stuffing, fragmentation or trimming is involved; by Lemma "evaldilate" (b)
  with u_L = 1 the last layer holds exactly the N - B + 1 dense outputs per axis.

Convolutions follow the paper's flipped-filter formula (Sect. 3.3) on weights in
cross-correlation order, like the rest of the oracle.
"""
from __future__ import annotations

import numpy as np

from . import _paper_orientation
from .mixed import _ACT, chain_of, stride_products


def dilated_subsignal(xi, d, k, i):
    """DilatedSubsignal_{(d, k)}(xi, i) along axis 0, i 1-based."""
    D = xi.shape[0]
    assert D >= k * (d - 1) + 1 and 1 <= i <= D - k * (d - 1)
    return np.stack([xi[i - 1 + k * (nu - 1)] for nu in range(1, d + 1)], axis=0)


def dilate(f, xi, c, k):
    """Dilate_{(f, k)}(xi) along axis 0: f(DilatedSubsignal_{(c, k)}(xi, i)) for
    i = 1 .. dim(xi) - k(c - 1)."""
    n = xi.shape[0] - k * (c - 1)
    assert n >= 1
    return np.stack([f(dilated_subsignal(xi, c, k, i)) for i in range(1, n + 1)], axis=0)


def dilate_conv(x, layer, k):
    """Dilate_{(f, k)} per axis, k = (k_h, k_w), for f = one output sample of a
    multi-channel convolution + bias + activation:
    x [C][H][W] -> [Cout][H - k_h(fh-1)][W - k_w(fw-1)], output (y, x) =
    b + sum_{i, m_h, m_w} w~[m_h][m_w] x[y + k_h(fh-1-m_h)][x + k_w(fw-1-m_w)]."""
    w = _paper_orientation(np.asarray(layer["weight"], dtype=np.float64))
    fh, fw = layer["fh"], layer["fw"]
    C, H, W = x.shape
    Eh, Ew = H - k[0] * (fh - 1), W - k[1] * (fw - 1)
    out = np.zeros((layer["cout"], Eh, Ew), dtype=np.float64)
    for mh in range(fh):
        for mw in range(fw):
            oy, ox = k[0] * (fh - 1 - mh), k[1] * (fw - 1 - mw)
            out += np.einsum("oi,iyx->oyx", w[:, :, mh, mw], x[:, oy:oy + Eh, ox:ox + Ew])
    b = layer.get("bias")
    if b is not None:
        out += np.asarray(b, dtype=np.float64)[:, None, None]
    return _ACT[layer["act"]](out)


def dilate_max(x, kh, kw, k):
    """Dilate_{(g, k)} per axis, k = (k_h, k_w), for g = the maximum of a kh x kw block."""
    H, W = x.shape[-2:]
    Ph, Pw = H - k[0] * (kh - 1), W - k[1] * (kw - 1)
    out = x[..., 0:Ph, 0:Pw].copy()
    for a in range(kh):
        for b in range(kw):
            out = np.maximum(out, x[..., k[0] * a:k[0] * a + Ph, k[1] * b:k[1] * b + Pw])
    return out


def eval_dilate(layers, x, upto=None):
    """EvalDilate_j(x) for j = upto (default L): x [C][H][W] -> [C_j][V_j,h][V_j,w]."""
    ch = chain_of(layers)
    ks = stride_products(ch)
    t = np.asarray(x, dtype=np.float64)
    for j in range(1, (len(ch) if upto is None else upto) + 1):
        e = ch[j - 1]
        if e["conv"] is not None:
            t = dilate_conv(t, e["conv"], ks[j - 1])
        t = dilate_max(t, e["k"][0], e["k"][1], ks[j - 1])
    return t
