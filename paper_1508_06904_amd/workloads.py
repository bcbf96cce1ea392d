"""Seeded synthetic workloads: input signals, layer lists and random weights.

This module is shared by the GPU path's tests/bench and by the oracle's tests.
It only draws random numbers and lays out layer descriptions; it holds none of
the dense-scanning arithmetic (no receptive field, stuffing, fragmentation or
convolution code lives here).

A layer is a plain dict:
  {"kind": "conv", "cin", "cout", "fh", "fw", "act": "none"|"relu"|"tanh",
   "weight": float32 [cout][cin][fh][fw] (cross-correlation order), "bias": float32 [cout]}
  {"kind": "maxpool", "kh", "kw"}

Weights are He-initialised, N(0, 2/fan_in) with fan_in = cin*fh*fw, biases are
0.01.  Draw order from one numpy PCG64 stream: the input first, then each conv
layer's weights in network order.

The paper measured on random images with random weights (runtime section,
Sect. 6.3); the value distributions below are stand-ins of the same shapes.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

ACTS = ("none", "relu", "tanh")


@dataclass
class Workload:
    name: str
    ndim: int                 # 1 or 2; a 1-D signal is stored with H == 1
    dtype: str                # "f32" or "bf16": storage type of input and activations
    x: np.ndarray             # float32 [C][H][W] (bf16 workloads: already bf16-representable)
    layers: list = field(default_factory=list)
    description: str = ""

    @property
    def shape(self):
        return self.x.shape


# --------------------------------------------------------------------------- arch specs
# An arch is a list of tuples: ("conv", cin, cout, fh, fw, act) | ("pool", kh, kw)

def arch_c1():
    return [("conv", 1, 4, 5, 5, "tanh"), ("pool", 2, 2),
            ("conv", 4, 8, 5, 5, "tanh"), ("pool", 2, 2),
            ("conv", 8, 1, 4, 4, "none")]


def arch_c2(w=(16, 32, 64), cout=2):
    a, b, c = w
    return [("conv", 1, a, 1, 9, "relu"), ("pool", 1, 2),
            ("conv", a, b, 1, 9, "relu"), ("pool", 1, 2),
            ("conv", b, c, 1, 9, "relu"), ("pool", 1, 2),
            ("conv", c, cout, 1, 8, "none")]


def arch_c3(w=(32, 64, 128, 256), cin=3, cout=2):
    a, b, c, d = w
    return [("conv", cin, a, 5, 5, "relu"), ("pool", 2, 2),
            ("conv", a, b, 5, 5, "relu"), ("pool", 2, 2),
            ("conv", b, c, 3, 3, "relu"), ("pool", 2, 2),
            ("conv", c, d, 6, 6, "relu"),
            ("conv", d, cout, 1, 1, "none")]


def arch_c4():
    return arch_c3(w=(64, 128, 256, 512))


def arch_c5(w=(32, 64, 128, 256), head=512, cin=3, cout=4):
    out = []
    prev = cin
    for width in w:
        out += [("conv", prev, width, 3, 3, "relu"), ("conv", width, width, 3, 3, "relu"),
                ("pool", 2, 2)]
        prev = width
    out += [("conv", prev, head, 6, 6, "relu"), ("conv", head, cout, 1, 1, "none")]
    return out


def arch_paper_sweep(L, maps=128):
    """The runtime-experiment family of Sect. 6.1/6.3: L 3x3 conv+ReLU layers with
    `maps` feature maps, a 2x2 max-pool after every third conv unless it would be last."""
    out = []
    prev = 1
    for j in range(1, L + 1):
        out.append(("conv", prev, maps, 3, 3, "relu"))
        prev = maps
        if j % 3 == 0 and j != L:
            out.append(("pool", 2, 2))
    return out


# --------------------------------------------------------------------------- weights

def init_layers(arch, rng, bias=0.01, weight_kind="he"):
    """Materialise an arch spec with random weights drawn from `rng` in order."""
    layers = []
    for spec in arch:
        if spec[0] == "pool":
            layers.append({"kind": "maxpool", "kh": int(spec[1]), "kw": int(spec[2])})
            continue
        _, cin, cout, fh, fw, act = spec
        assert act in ACTS
        if weight_kind == "he":
            std = math.sqrt(2.0 / (cin * fh * fw))
            w = (rng.standard_normal((cout, cin, fh, fw)) * std).astype(np.float32)
            b = np.full((cout,), bias, dtype=np.float32)
        elif weight_kind == "int":
            # small integers: every partial sum stays exactly representable
            w = rng.integers(-1, 2, size=(cout, cin, fh, fw)).astype(np.float32)
            b = rng.integers(-2, 3, size=(cout,)).astype(np.float32)
        else:
            raise ValueError(weight_kind)
        layers.append({"kind": "conv", "cin": int(cin), "cout": int(cout), "fh": int(fh),
                       "fw": int(fw), "act": act, "weight": w, "bias": b})
    return layers


def sparse_integer_layers(layers, nonzeros, rng):
    """The same layer shapes with exactly-representable parameters: every output
    channel of conv t gets nonzeros[t] weights of +-1 at random positions of its
    cin x fh x fw taps (the rest zero) and an integer bias in [-2, 2].  With
    integer inputs bounded by b_0, every value and every partial sum of conv t
    stays within b_t = nonzeros[t] * b_{t-1} + 2, so while
    that is below 2^24 binary32 arithmetic computes the forward pass exactly."""
    nz = iter(nonzeros)
    out = []
    for l in layers:
        if l["kind"] != "conv":
            out.append(l)
            continue
        d = next(nz)
        K = l["cin"] * l["fh"] * l["fw"]
        w = np.zeros((l["cout"], K), dtype=np.float32)
        for o in range(l["cout"]):
            w[o, rng.choice(K, size=d, replace=False)] = rng.choice([-1.0, 1.0], size=d)
        out.append(dict(l, weight=w.reshape(l["cout"], l["cin"], l["fh"], l["fw"]),
                        bias=rng.integers(-2, 3, size=l["cout"]).astype(np.float32)))
    return out


# --------------------------------------------------------------------------- inputs

def uniform_image(rng, C, H, W):
    return rng.random((C, H, W), dtype=np.float32)


def blob_image(rng, C, H, W, n_blobs):
    """Per-channel U[0,1) plus n_blobs Gaussian blobs, sigma ~ U[8,48] px,
    per-channel amplitude U[-0.5,0.5], centres uniform over the frame."""
    img = rng.random((C, H, W), dtype=np.float32).astype(np.float64)
    for _ in range(n_blobs):
        cy = rng.uniform(0, H)
        cx = rng.uniform(0, W)
        sig = rng.uniform(8.0, 48.0)
        amp = rng.uniform(-0.5, 0.5, size=C)
        r = int(math.ceil(3 * sig))
        y0, y1 = max(0, int(cy) - r), min(H, int(cy) + r + 1)
        x0, x1 = max(0, int(cx) - r), min(W, int(cx) + r + 1)
        if y0 >= y1 or x0 >= x1:
            continue
        yy = (np.arange(y0, y1) - cy)[:, None]
        xx = (np.arange(x0, x1) - cx)[None, :]
        g = np.exp(-(yy * yy + xx * xx) / (2 * sig * sig))
        img[:, y0:y1, x0:x1] += amp[:, None, None] * g[None]
    return img.astype(np.float32)


def burst_signal(rng, n, n_bursts=64):
    """N(0,1) noise plus seeded sinusoid bursts with a Hann envelope: start uniform,
    length U[256,16384], amplitude U[1,5], frequency U[0.005,0.45] cycles/sample,
    phase U[0,2pi)."""
    sig = rng.standard_normal(n)
    for _ in range(n_bursts):
        start = int(rng.integers(0, n))
        length = int(rng.integers(256, 16385))
        amp = rng.uniform(1.0, 5.0)
        freq = rng.uniform(0.005, 0.45)
        phase = rng.uniform(0.0, 2 * math.pi)
        end = min(n, start + length)
        t = np.arange(end - start)
        env = 0.5 - 0.5 * np.cos(2 * math.pi * t / max(1, length - 1))
        sig[start:end] += amp * env * np.sin(2 * math.pi * freq * t + phase)
    return sig.astype(np.float32)[None, None, :]


def to_bf16_representable(x):
    """Round float32 values to the nearest bfloat16 (ties to even) using torch's CPU cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def bf16_bits(x):
    """uint16 bit patterns of an array that is already bf16-representable."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "array is not bf16-representable"
    return (u >> 16).astype(np.uint16)


# --------------------------------------------------------------------------- named configs

CONFIG_NAMES = ("c1_64x64", "c2_1d_1m", "c3_512", "c4_hd", "c5_4k")


def make(name, seed=0, H=None, W=None, widths=None, weight_kind="he"):
    """Build a named workload.  H/W/widths override the sizes for parity tests at
    reduced scale; the value distribution and layer pattern stay the same."""
    rng = np.random.default_rng(seed)
    if name == "c1_64x64":
        H = H or 64
        W = W or 64
        x = uniform_image(rng, 1, H, W)
        layers = init_layers(arch_c1(), rng, weight_kind=weight_kind)
        return Workload(name, 2, "f32", x, layers,
                        f"2-D 1x{H}x{W} fp32, U[0,1); conv5x5 1-4 tanh, pool2, conv5x5 4-8 tanh, pool2, conv4x4 8-1")
    if name == "c2_1d_1m":
        W = W or (1 << 20)
        x = burst_signal(rng, W, n_bursts=max(1, round(64 * W / (1 << 20))))
        layers = init_layers(arch_c2(*( [widths] if widths else [])), rng, weight_kind=weight_kind)
        return Workload(name, 1, "f32", x, layers,
                        f"1-D 1x{W} fp32 noise+bursts; conv9 1-16-32-64 relu + pool2 x3, conv8 64-2")
    if name == "c3_512":
        H = H or 512
        W = W or 512
        x = blob_image(rng, 3, H, W, n_blobs=max(1, round(24 * H * W / (512 * 512))))
        layers = init_layers(arch_c3(*([widths] if widths else [])), rng, weight_kind=weight_kind)
        return Workload(name, 2, "f32", x, layers,
                        f"2-D 3x{H}x{W} fp32 blobs; conv5x5/pool2 x2, conv3x3/pool2, conv6x6, conv1x1 -> 2")
    if name == "c4_hd":
        H = H or 1080
        W = W or 1920
        x = blob_image(rng, 3, H, W, n_blobs=max(1, round(190 * H * W / (1080 * 1920))))
        arch = arch_c3(w=widths) if widths else arch_c4()
        layers = init_layers(arch, rng, weight_kind=weight_kind)
        return Workload(name, 2, "f32", x, layers,
                        f"2-D 3x{H}x{W} fp32 blobs; widths 64/128/256/512; conv6x6 256-512, conv1x1 512-2")
    if name == "c5_4k":
        H = H or 2160
        W = W or 3840
        x = blob_image(rng, 3, H, W, n_blobs=max(1, round(760 * H * W / (2160 * 3840))))
        x = to_bf16_representable(x)
        arch = arch_c5(*([widths] if widths else []))
        layers = init_layers(arch, rng, weight_kind=weight_kind)
        return Workload(name, 2, "bf16", x, layers,
                        f"2-D 3x{H}x{W} bf16 blobs; 4x(conv3x3,conv3x3,pool2) 32/64/128/256, conv6x6 256-512, conv1x1 512-4")
    raise KeyError(name)


def custom(arch, C, H, W, seed=0, dtype="f32", ndim=2, weight_kind="he", value_kind="uniform"):
    """A workload from an explicit arch spec; used by the property tests."""
    rng = np.random.default_rng(seed)
    if value_kind == "uniform":
        x = uniform_image(rng, C, H, W)
    elif value_kind == "int":
        x = rng.integers(-8, 9, size=(C, H, W)).astype(np.float32)
    elif value_kind == "normal":
        x = rng.standard_normal((C, H, W)).astype(np.float32)
    else:
        raise ValueError(value_kind)
    if dtype == "bf16":
        x = to_bf16_representable(x)
    layers = init_layers(arch, rng, weight_kind=weight_kind)
    return Workload("custom", ndim, dtype, x, layers, "custom arch")


def sample_windows(out_h, out_w, K_h, K_w, per_phase, seed=0):
    """Seeded sample of dense-output positions (i, j): the 4 corners, the 4 edge
    midpoints, and `per_phase` random positions for every residue pair
    (i mod K_h, j mod K_w) that occurs."""
    rng = np.random.default_rng(seed + 12345)
    pts = {(0, 0), (0, out_w - 1), (out_h - 1, 0), (out_h - 1, out_w - 1),
           (0, out_w // 2), (out_h - 1, out_w // 2), (out_h // 2, 0), (out_h // 2, out_w - 1)}
    for ph in range(min(K_h, out_h)):
        nh = (out_h - 1 - ph) // K_h + 1
        for pw in range(min(K_w, out_w)):
            nw = (out_w - 1 - pw) // K_w + 1
            for _ in range(per_phase):
                i = ph + K_h * int(rng.integers(0, nh))
                j = pw + K_w * int(rng.integers(0, nw))
                pts.add((i, j))
    arr = np.array(sorted(pts), dtype=np.int64)
    return arr[:, 0].copy(), arr[:, 1].copy()
