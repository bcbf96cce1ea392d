"""Gradients of the dense evaluation -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg use this module;
the GPU library never imports it.  Double precision numpy.

What is differentiated.  The dense evaluation maps a signal x to
T(x)[c][i][j] = EvalStride_L(window (i, j) of x)[c] (Theorem "processing
chain", Sect. 4.3).  For an upstream gradient G of the same shape as T(x), the
scalar  l = sum_{c,i,j} G[c][i][j] * T(x)[c][i][j]  has the gradients

  dl/dW_j, dl/db_j = sum over windows of the ordinary backpropagation through the
                     strided network on that window, seeded with G at the window;
  dl/dx            = the per-window input gradients added back at the windows'
                     positions.

This is the plain definition the fine-tuning remark of Sect. 6.2 relies on (the
transformed network computes the same function, so its gradients are these).
`dense_backward` computes it window by window (vectorised over windows), with
each layer's derivative written out by elementary calculus:

  conv (cross-correlation order, as the weights are given):
    y[o][p] = b[o] + sum_{i,t} w[o][i][t] x[i][p + t],  a = act(y)
    dy = da * act'(y);  db[o] = sum_p dy[o][p];
    dw[o][i][t] = sum_p dy[o][p] x[i][p + t];  dx[i][p + t] += w[o][i][t] dy[o][p]
  max-pool over non-overlapping k_h x k_w blocks: the gradient of each block's
    output goes to the block's maximal input; among equal maxima to the first in
    row-major order (the rule any implementation must share for integer data;
    with continuous data ties have probability zero).

ReLU'(0) = 0; tanh' = 1 - tanh^2.
"""
from __future__ import annotations

import numpy as np

from .mixed import chain_of, strided_extents


def _conv_forward(x, layer):
    """x [N][C][H][W] -> pre-activation [N][Cout][H-fh+1][W-fw+1] (cross-correlation)."""
    w = np.asarray(layer["weight"], dtype=np.float64)
    fh, fw = layer["fh"], layer["fw"]
    N, C, H, W = x.shape
    Eh, Ew = H - fh + 1, W - fw + 1
    y = np.zeros((N, layer["cout"], Eh, Ew))
    for a in range(fh):
        for c in range(fw):
            y += np.einsum("oi,niyx->noyx", w[:, :, a, c], x[:, :, a:a + Eh, c:c + Ew])
    if layer.get("bias") is not None:
        y += np.asarray(layer["bias"], dtype=np.float64)[None, :, None, None]
    return y


def _act(y, act):
    return {"none": lambda v: v, "relu": lambda v: np.maximum(v, 0.0), "tanh": np.tanh}[act](y)


def _act_grad(y, a, act):
    """act'(y) given pre-activation y and output a."""
    if act == "none":
        return np.ones_like(y)
    if act == "relu":
        return (y > 0).astype(np.float64)
    return 1.0 - a * a


def _pool_forward(x, kh, kw):
    """Non-overlapping block maximum and the first maximal position per block."""
    N, C, H, W = x.shape
    assert H % kh == 0 and W % kw == 0
    blocks = x.reshape(N, C, H // kh, kh, W // kw, kw).transpose(0, 1, 2, 4, 3, 5).reshape(N, C, H // kh, W // kw, kh * kw)
    arg = np.argmax(blocks, axis=-1)            # numpy returns the first maximum
    return np.take_along_axis(blocks, arg[..., None], axis=-1)[..., 0], arg


def _pool_backward(g, arg, kh, kw, shape):
    N, C, H, W = shape
    oh, ow = H // kh, W // kw
    out = np.zeros((N, C, oh, ow, kh * kw))
    np.put_along_axis(out, arg[..., None], g[..., None], axis=-1)
    return out.reshape(N, C, oh, ow, kh, kw).transpose(0, 1, 2, 4, 3, 5).reshape(N, C, H, W)


def strided_backward(layers, patches, g_out):
    """Backpropagation through the strided network on a batch of patches.

    patches [N][C][B_h][B_w], g_out [N][C_out] (each patch ends in one sample).
    Returns (dW list, db list) over the conv descriptors in order, and d_patches."""
    acts, caches = np.asarray(patches, dtype=np.float64), []
    for l in layers:
        if l["kind"] == "conv":
            y = _conv_forward(acts, l)
            a = _act(y, l["act"])
            caches.append(("conv", l, acts, y, a))
            acts = a
        else:
            p, arg = _pool_forward(acts, l["kh"], l["kw"])
            caches.append(("pool", l, acts.shape, arg))
            acts = p
    assert acts.shape[2:] == (1, 1), "the strided network must end in one sample per patch"
    g = np.asarray(g_out, dtype=np.float64)[:, :, None, None]
    dW, db = [], []
    for entry in reversed(caches):
        if entry[0] == "pool":
            _, l, shape, arg = entry
            g = _pool_backward(g, arg, l["kh"], l["kw"], shape)
            continue
        _, l, x, y, a = entry
        dy = g * _act_grad(y, a, l["act"])
        w = np.asarray(l["weight"], dtype=np.float64)
        fh, fw = l["fh"], l["fw"]
        Eh, Ew = dy.shape[2:]
        dw = np.zeros_like(w)
        dx = np.zeros_like(x)
        for r in range(fh):
            for c in range(fw):
                xs = x[:, :, r:r + Eh, c:c + Ew]
                dw[:, :, r, c] = np.einsum("noyx,niyx->oi", dy, xs)
                dx[:, :, r:r + Eh, c:c + Ew] += np.einsum("oi,noyx->niyx", w[:, :, r, c], dy)
        dW.append(dw)
        db.append(dy.sum(axis=(0, 2, 3)))
        g = dx
    return dW[::-1], db[::-1], g


def dense_backward(layers, x, g_dense, batch=4096):
    """Gradients of sum(G * T(x)) for the dense evaluation T, window by window.

    x [C][H][W], g_dense [C_out][H-B_h+1][W-B_w+1].
    Returns (dW list, db list, dx [C][H][W])."""
    x = np.asarray(x, dtype=np.float64)
    C, H, W = x.shape
    Bh, Bw = strided_extents(chain_of(layers))[0]
    Oh, Ow = H - Bh + 1, W - Bw + 1
    g_dense = np.asarray(g_dense, dtype=np.float64)
    assert g_dense.shape[1:] == (Oh, Ow)
    convs = [l for l in layers if l["kind"] == "conv"]
    dW = [np.zeros_like(np.asarray(l["weight"], dtype=np.float64)) for l in convs]
    db = [np.zeros(l["cout"]) for l in convs]
    dx = np.zeros_like(x)
    ii, jj = np.meshgrid(np.arange(Oh), np.arange(Ow), indexing="ij")
    ii, jj = ii.reshape(-1), jj.reshape(-1)
    for s in range(0, len(ii), batch):
        bi, bj = ii[s:s + batch], jj[s:s + batch]
        patches = np.stack([x[:, i:i + Bh, j:j + Bw] for i, j in zip(bi, bj)])
        g = g_dense[:, bi, bj].T
        w_, b_, dp = strided_backward(layers, patches, g)
        for t in range(len(convs)):
            dW[t] += w_[t]
            db[t] += b_[t]
        for n, (i, j) in enumerate(zip(bi, bj)):
            dx[:, i:i + Bh, j:j + Bw] += dp[n]
    return dW, db, dx
