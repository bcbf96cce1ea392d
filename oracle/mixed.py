"""Relaxed and mixed evaluation of a processing chain -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg use this module;
the GPU library never imports it.  Everything is double precision numpy.

Two independent routes to the same result:

* `dense_downsampled` is the plain definition of what the relaxed and mixed
  evaluations compute: conventional dense scanning (the strided network on every
  window, `eval_stride`) followed by the downsampling operator Down_k of the
  appendix (Definition "downsampling"), per axis, with k = k*_l.  Theorem
  "evalrelax" (l = L) and Theorem "evalrelaxslide" (0 < l < L) state this
  equality; for l = 0 it is Theorem "processing chain" (Sect. 4.3).

* `eval_relax_slide` takes the steps of the mixed algorithm of Theorem
  "evalrelaxslide" in the paper's order, on the whole signal:
    1. per axis r = rem(N - B + k*_l, k*_L); if r < k*_l trim r samples
       (trimming mode), else stuff k*_L - r dummy samples (stuffing mode);
    2. layers 1..l in a relaxed fashion, Stride_g(Slide_f(.)) (Definition
       "evalrelax"): the convolution on the whole signal, then the maximum over
       non-overlapping k_j blocks;
    3. layers l+1..L in a sliding fashion, Frag_k(Slide_g(Slide_f(.)))
       (Definition "evalrelaxslide"), on every fragment;
    4. Defrag_{k*_L / k*_l};
    5. in the stuffing mode, trim the s superfluous samples with
       s = (k*_L - r + s~ - 1) / k*_l, s~ = k*_l if k*_l divides N - B + 1 and
       rem(N - B + 1, k*_l) otherwise.
  `upto=j` stops after layer j and returns the fragment tensor, whose samples
  Lemma "evalrelax" (b) and Lemma "evalrelaxslide" (c), (d) relate to EvalStride.

Convolutions follow the paper's flipped-filter formula (Sect. 3.3) on weights
given in cross-correlation order, like the C oracle; the activation follows the
bias.  The dummy sample of the stuffing is +0.
"""
from __future__ import annotations

import math

import numpy as np

from . import _paper_orientation, eval_stride, fragment

_ACT = {"none": lambda v: v, "relu": lambda v: np.maximum(v, 0.0), "tanh": np.tanh}


# ----------------------------------------------------------------------------- operators

def downsample(xi, k):
    """Down_k along axis 0 (Definition "downsampling"): samples k(nu-1)+1 for
    nu = 1..ceil(D/k) in 1-based indices."""
    D = xi.shape[0]
    n = -(-D // k)
    return np.stack([xi[k * (nu - 1)] for nu in range(1, n + 1)], axis=0)


def slide_conv(x, layer):
    """Slide_f of a multi-channel convolution + bias + activation on every
    fragment of x ([F][Cin][H][W] -> [F][Cout][H-fh+1][W-fw+1]).  Output sample
    (y, x) is b + sum over input channels and paper taps (m_h, m_w) of
    w~[m_h][m_w] * x[y + fh-1 - m_h][x + fw-1 - m_w] (Sect. 3.3, per axis)."""
    w = _paper_orientation(np.asarray(layer["weight"], dtype=np.float64))
    fh, fw = layer["fh"], layer["fw"]
    F, C, H, W = x.shape
    Eh, Ew = H - fh + 1, W - fw + 1
    out = np.zeros((F, layer["cout"], Eh, Ew), dtype=np.float64)
    for mh in range(fh):
        for mw in range(fw):
            oy, ox = fh - 1 - mh, fw - 1 - mw
            out += np.einsum("oi,fiyx->foyx", w[:, :, mh, mw], x[:, :, oy:oy + Eh, ox:ox + Ew])
    b = layer.get("bias")
    if b is not None:
        out += np.asarray(b, dtype=np.float64)[None, :, None, None]
    return _ACT[layer["act"]](out)


def slide_max(x, kh, kw):
    """Slide_g with g the maximum of a kh x kw block: stride 1 (Sect. 4)."""
    H, W = x.shape[-2:]
    Ph, Pw = H - kh + 1, W - kw + 1
    out = x[..., 0:Ph, 0:Pw].copy()
    for a in range(kh):
        for b in range(kw):
            out = np.maximum(out, x[..., a:a + Ph, b:b + Pw])
    return out


def stride_max(x, kh, kw):
    """Stride_g with g the maximum of a kh x kw block: non-overlapping blocks
    starting at the first sample (Definition "strided function", Sect. 4)."""
    H, W = x.shape[-2:]
    assert H % kh == 0 and W % kw == 0, "Stride_g needs extents divisible by the block size"
    out = x[..., 0::kh, 0::kw].copy()
    for a in range(kh):
        for b in range(kw):
            out = np.maximum(out, x[..., a::kh, b::kw])
    return out


# ----------------------------------------------------------------------------- chain

def chain_of(layers):
    """Processing-chain layers from a layer list: a convolution and the max-pool
    that directly follows it form one layer; a convolution alone has k = 1, a
    pool alone has the identity transformation (end of Sect. 4.2)."""
    ch, t = [], 0
    while t < len(layers):
        l = layers[t]
        if l["kind"] == "conv":
            entry = {"conv": l, "c": (l["fh"], l["fw"]), "k": (1, 1)}
            t += 1
            if t < len(layers) and layers[t]["kind"] == "maxpool":
                entry["k"] = (layers[t]["kh"], layers[t]["kw"])
                t += 1
        else:
            entry = {"conv": None, "c": (1, 1), "k": (l["kh"], l["kw"])}
            t += 1
        ch.append(entry)
    return ch


def stride_products(ch):
    """k*_0..k*_L per axis: k*_j = k_1 ... k_j."""
    ks = [(1, 1)]
    for e in ch:
        ks.append((ks[-1][0] * e["k"][0], ks[-1][1] * e["k"][1]))
    return ks


def strided_extents(ch):
    """u_0..u_L per axis from u_L = 1 and u_{j-1} = k_j u_j + c_j - 1
    (Lemma "processing chain" (a)); B = u_0."""
    u = [(1, 1)]
    for e in reversed(ch):
        u.append((e["k"][0] * u[-1][0] + e["c"][0] - 1, e["k"][1] * u[-1][1] + e["c"][1] - 1))
    return list(reversed(u))


def operating_mode(N, B, K, k):
    """Per axis: (mode, r, samples trimmed first, samples stuffed, s) of Theorem
    "evalrelaxslide" for a signal of N samples, receptive field B, final stride
    product K = k*_L and intermediate stride product k = k*_l."""
    r = (N - B + k) % K
    if r < k:
        return "trim", r, r, 0, 0
    s_tilde = k if (N - B + 1) % k == 0 else (N - B + 1) % k
    num = K - r + s_tilde - 1
    assert num % k == 0, "the superfluous-sample count must be a whole number"
    return "stuff", r, 0, K - r, num // k


def _along(x, axis, fn):
    return np.moveaxis(fn(np.moveaxis(x, axis, 0)), 0, axis)


# ----------------------------------------------------------------------------- the two routes

def dense_downsampled(layers, x, step, threads=0):
    """Down_{step_h} x Down_{step_w} of Slide_{EvalStride_L}(x) by its definition:
    EvalStride on the windows whose top-left sample is (step_h*i, step_w*j).
    x [C][H][W] -> float64 [C_out][ceil((H-B_h+1)/step_h)][ceil((W-B_w+1)/step_w)]."""
    ch = chain_of(layers)
    B = strided_extents(ch)[0]
    C, H, W = np.asarray(x).shape
    Oh, Ow = -(-(H - B[0] + 1) // step[0]), -(-(W - B[1] + 1) // step[1])
    ii, jj = np.meshgrid(step[0] * np.arange(Oh, dtype=np.int64), step[1] * np.arange(Ow, dtype=np.int64),
                         indexing="ij")
    res = eval_stride(layers, x, windows=(ii.reshape(-1), jj.reshape(-1)), patch=B, threads=threads)
    return res.reshape(Oh, Ow, -1).transpose(2, 0, 1).copy()


def eval_relax_slide(layers, x, ell, upto=None, zeta=0.0):
    """The mixed evaluation of Theorem "evalrelaxslide" (0 <= ell <= L).

    x [C][H][W].  Returns float64 [C_out][ceil((H-B_h+1)/k*_l,h)][ceil((W-B_w+1)/k*_l,w)],
    or with upto = j the intermediate EvalRelaxSlide_j of the trimmed/stuffed
    signal as planar fragments [F][C_j][h][w] (F = 1 for j <= ell, else
    (k*_j,h/k*_l,h) * (k*_j,w/k*_l,w), row-major over (row, column) fragment)."""
    ch = chain_of(layers)
    L = len(ch)
    if not 0 <= ell <= L:
        raise ValueError("ell must lie in 0..L")
    ks = stride_products(ch)
    B = strided_extents(ch)[0]
    x = np.asarray(x, dtype=np.float64)
    C, H, W = x.shape
    if H < B[0] or W < B[1]:
        raise ValueError("signal smaller than the receptive field")
    modes = [operating_mode(N, B[a], ks[L][a], ks[ell][a]) for a, N in enumerate((H, W))]
    for axis, (_, _, tr, st, _) in zip((1, 2), modes):
        if tr:
            x = _along(x, axis, lambda v, tr=tr: fragment.trim(v, tr))
        if st:
            x = _along(x, axis, lambda v, st=st: fragment.stuff(v, st, zeta))
    t = x[None]
    last = L if upto is None else upto
    for j in range(1, last + 1):
        e = ch[j - 1]
        if e["conv"] is not None:
            t = slide_conv(t, e["conv"])
        kh, kw = e["k"]
        if j <= ell:
            t = stride_max(t, kh, kw)
        else:
            t = slide_max(t, kh, kw)
            Sh, Sw = ks[j - 1][0] // ks[ell][0], ks[j - 1][1] // ks[ell][1]
            t = fragment.frag_tensor(t, kh, kw, Sh, Sw)
    if upto is not None:
        return t
    Fh, Fw = ks[L][0] // ks[ell][0], ks[L][1] // ks[ell][1]
    y = fragment.defrag_tensor(t, Fh, Fw, 1, 1)[0]
    for axis, (_, _, _, _, s) in zip((1, 2), modes):
        if s:
            y = _along(y, axis, lambda v, s=s: fragment.trim(v, s))
    return y


def output_extent(N, B, k):
    """ceil((N - B + 1) / k): samples of Down_k(Slide_{EvalStride_L}(xi))."""
    return math.ceil((N - B + 1) / k)
