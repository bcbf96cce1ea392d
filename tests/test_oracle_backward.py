"""Pins for the oracle's gradients of the dense evaluation (no GPU): torch's CPU
float64 autograd on the strided network over every window (an independent
implementation), central finite differences of the C oracle's forward pass,
closed forms for the last layer, and the tie rule of the max-pool gradient."""
import numpy as np
import pytest
import torch
import torch.nn.functional as tF

import oracle
from oracle import backward as ob
from paper_1508_06904_amd import workloads as wl
from tests.test_oracle import all_patches

ARCHS = {
    "2d_tanh": ([("conv", 2, 3, 3, 2, "tanh"), ("pool", 2, 2), ("conv", 3, 4, 2, 2, "tanh"), ("pool", 1, 2),
                 ("conv", 4, 2, 2, 1, "none")], 2, 2),
    "2d_relu": ([("conv", 3, 5, 3, 3, "relu"), ("pool", 2, 2), ("conv", 5, 4, 2, 2, "relu"), ("conv", 4, 3, 1, 1, "none")],
                3, 2),
    "2d_pool_first": ([("pool", 2, 2), ("conv", 2, 3, 2, 2, "tanh"), ("pool", 2, 2), ("conv", 3, 1, 1, 1, "none")], 2, 2),
    "1d": ([("conv", 1, 3, 1, 4, "tanh"), ("pool", 1, 3), ("conv", 3, 2, 1, 2, "none")], 1, 1),
}
T_ACT = {"none": lambda t: t, "relu": torch.relu, "tanh": torch.tanh}


def _setup(name, extra=(5, 6), seed=0):
    arch, C, nd = ARCHS[name]
    rng = np.random.default_rng(seed)
    layers = wl.init_layers(arch, rng)
    for l in layers:   # float64 copies, so that finite-difference steps are not rounded away
        if l["kind"] == "conv":
            l["weight"] = np.asarray(l["weight"], dtype=np.float64).copy()
            l["bias"] = np.asarray(l["bias"], dtype=np.float64).copy()
    bh, bw = oracle.receptive_field(layers)
    H = 1 if nd == 1 else bh + extra[0]
    W = bw + extra[1]
    x = rng.standard_normal((C, H, W))
    G = rng.standard_normal((layers[-1]["cout"], H - bh + 1, W - bw + 1))
    return layers, x, G, (bh, bw)


def torch_grads(layers, x, G, B):
    """torch autograd (float64, CPU) through the strided network on every window."""
    p, oh, ow = all_patches(x, *B)
    xp = torch.from_numpy(p).requires_grad_(True)
    params, t = [], xp
    for l in layers:
        if l["kind"] == "conv":
            w = torch.from_numpy(np.asarray(l["weight"], dtype=np.float64)).requires_grad_(True)
            b = torch.from_numpy(np.asarray(l["bias"], dtype=np.float64)).requires_grad_(True)
            params.append((w, b))
            t = T_ACT[l["act"]](tF.conv2d(t, w, b))
        else:
            t = tF.max_pool2d(t, (l["kh"], l["kw"]), stride=(l["kh"], l["kw"]))
    g = torch.from_numpy(G.reshape(G.shape[0], -1).T.copy())[:, :, None, None]
    (t * g).sum().backward()
    dx = np.zeros_like(x)
    dp = xp.grad.numpy()
    for i in range(oh):
        for j in range(ow):
            dx[:, i:i + B[0], j:j + B[1]] += dp[i * ow + j]
    return [w.grad.numpy() for w, _ in params], [b.grad.numpy() for _, b in params], dx


@pytest.mark.parametrize("name", list(ARCHS))
def test_matches_torch_autograd(name):
    layers, x, G, B = _setup(name)
    dW, db, dx = ob.dense_backward(layers, x, G)
    tW, tb, tx = torch_grads(layers, x, G, B)
    for a, b in zip(dW, tW):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-11)
    for a, b in zip(db, tb):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dx, tx, rtol=1e-11, atol=1e-11)


def _loss(layers, x, G):
    return float(np.sum(G * oracle.eval_stride(layers, x)))


@pytest.mark.parametrize("name", ["2d_tanh", "1d", "2d_pool_first"])
def test_matches_finite_differences_of_the_forward_oracle(name):
    """Central differences of sum(G * EvalStride on every window), computed by the
    C oracle, at randomly chosen weights, biases and input samples."""
    layers, x, G, B = _setup(name, seed=3)
    dW, db, dx = ob.dense_backward(layers, x, G)
    rng = np.random.default_rng(4)
    h = 1e-6
    convs = [t for t, l in enumerate(layers) if l["kind"] == "conv"]
    for ci, t in enumerate(convs):
        w = layers[t]["weight"]
        for _ in range(3):
            idx = tuple(rng.integers(0, s) for s in w.shape)
            orig = w[idx]
            w[idx] = orig + h
            up = _loss(layers, x, G)
            w[idx] = orig - h
            dn = _loss(layers, x, G)
            w[idx] = orig
            assert abs((up - dn) / (2 * h) - dW[ci][idx]) <= 1e-6 * max(1.0, abs(dW[ci][idx]))
        b = layers[t]["bias"]
        k = int(rng.integers(0, len(b)))
        orig = b[k]
        b[k] = orig + h
        up = _loss(layers, x, G)
        b[k] = orig - h
        dn = _loss(layers, x, G)
        b[k] = orig
        assert abs((up - dn) / (2 * h) - db[ci][k]) <= 1e-6 * max(1.0, abs(db[ci][k]))
    for _ in range(4):
        idx = tuple(rng.integers(0, s) for s in x.shape)
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (_loss(layers, xp, G) - _loss(layers, xm, G)) / (2 * h)
        assert abs(fd - dx[idx]) <= 1e-6 * max(1.0, abs(dx[idx]))


def test_last_layer_closed_forms():
    """For a final 1x1 conv without activation: db = sum of G over the output
    grid, and dW = sum over windows of G times the last hidden features."""
    layers, x, G, B = _setup("2d_relu", seed=5)
    dW, db, dx = ob.dense_backward(layers, x, G)
    np.testing.assert_allclose(db[-1], G.sum(axis=(1, 2)), rtol=1e-12)
    feats = oracle.eval_stride(layers[:-1], x, patch=B)        # [C_hidden][Oh][Ow]
    ref = np.einsum("oyx,iyx->oi", G, feats)
    np.testing.assert_allclose(dW[-1][:, :, 0, 0], ref, rtol=1e-11, atol=1e-11)


def test_max_pool_tie_goes_to_the_first_maximum():
    """A block [[5, 5], [5, 1]] passes its gradient to its first element."""
    layers = [{"kind": "conv", "cin": 1, "cout": 1, "fh": 1, "fw": 1, "act": "none",
               "weight": np.ones((1, 1, 1, 1)), "bias": np.zeros(1)},
              {"kind": "maxpool", "kh": 2, "kw": 2}]
    x = np.array([[[5.0, 5.0], [5.0, 1.0]]])
    dW, db, dx = ob.dense_backward(layers, x, np.array([[[2.0]]]))
    np.testing.assert_array_equal(dx[0], [[2.0, 0.0], [0.0, 0.0]])
    assert dW[0][0, 0, 0, 0] == 10.0 and db[0][0] == 2.0
