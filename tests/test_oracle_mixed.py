"""Pins for the relaxed / mixed evaluation in the oracle (no GPU).

`oracle.mixed.eval_relax_slide` follows the mixed algorithm of Theorem
"evalrelaxslide" on the whole signal (numpy); `oracle.mixed.dense_downsampled`
is the plain definition Down_{k*_l}(Slide_{EvalStride_L}) computed patch by
patch in C.  The two share nothing but the layer list, so their agreement for
every l and every signal length pins both; the hand-computed figure example,
the closed forms of Lemma "evalrelax" / Lemma "evalrelaxslide", the index maps
(c), (d) against EvalStride and the independence of the dummy value pin the
details (trimming vs stuffing, the superfluous-sample count s)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import mixed
from paper_1508_06904_amd import workloads as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden")

ARCHS = {
    "1d_three": ([("conv", 1, 3, 1, 3, "relu"), ("pool", 1, 2), ("conv", 3, 4, 1, 2, "tanh"), ("pool", 1, 3),
                  ("conv", 4, 2, 1, 2, "relu"), ("pool", 1, 2), ("conv", 2, 1, 1, 2, "none")], 1, 1),
    "2d_mixed": ([("conv", 3, 4, 3, 2, "relu"), ("pool", 2, 1), ("conv", 4, 5, 2, 3, "tanh"), ("pool", 1, 2),
                  ("conv", 5, 2, 2, 2, "none")], 3, 2),
    "2d_pool_first": ([("pool", 2, 2), ("conv", 2, 3, 2, 2, "relu"), ("pool", 2, 2), ("conv", 3, 2, 1, 1, "none")], 2, 2),
    "2d_c1": (wl.arch_c1(), 1, 2),
    "2d_pool_pool": ([("conv", 1, 2, 2, 2, "relu"), ("pool", 2, 2), ("pool", 3, 3), ("conv", 2, 1, 1, 1, "none")], 1, 2),
}


def _layers(name, seed=3):
    arch, C, nd = ARCHS[name]
    return wl.init_layers(arch, np.random.default_rng(seed)), C, nd


def _descriptors_upto(layers, j):
    """Number of layer descriptors that make up chain layers 1..j."""
    n, t = 0, 0
    while n < j:
        t += 1
        if layers[t - 1]["kind"] == "conv" and t < len(layers) and layers[t]["kind"] == "maxpool":
            t += 1
        n += 1
    return t


def _geometry(layers):
    ch = mixed.chain_of(layers)
    return ch, mixed.stride_products(ch), mixed.strided_extents(ch)


# ----------------------------------------------------------------------------- definitions

def test_downsample_definition():
    v = np.arange(7.0)
    np.testing.assert_array_equal(mixed.downsample(v, 3), [0.0, 3.0, 6.0])
    np.testing.assert_array_equal(mixed.downsample(v, 1), v)
    for D in range(1, 11):
        for k in range(1, 5):
            d = mixed.downsample(np.arange(D), k)
            assert len(d) == math.ceil(D / k)
            assert list(d) == list(range(0, D, k))


def test_relaxed_figure_example():
    with open(os.path.join(GOLD, "relaxed_fig.json")) as f:
        g = json.load(f)
    layers = []
    for l in g["layers"]:
        layers.append(dict(l, weight=np.array(l["weight"]), bias=np.array(l["bias"])) if l["kind"] == "conv" else l)
    x = np.array(g["signal"], dtype=np.float64)[None, None, :]
    ch, ks, us = _geometry(layers)
    assert us[0] == (1, g["B"]) and ks[-1] == (1, g["k_star"])
    assert oracle.receptive_field(layers) == (1, g["B"])
    np.testing.assert_array_equal(oracle.eval_stride(layers, x)[0, 0], g["dense"])
    relaxed = mixed.eval_relax_slide(layers, x, ell=1)
    assert relaxed.shape == (1, 1, g["W_1"])
    np.testing.assert_array_equal(relaxed[0, 0], g["relaxed"])
    np.testing.assert_array_equal(mixed.dense_downsampled(layers, x, (1, 4))[0, 0], g["relaxed"])
    starts = [s - 1 for s in g["subsignal_starts_1based"]]
    per_window = oracle.eval_stride(layers, x, windows=(np.zeros(3, np.int64), np.array(starts)))
    np.testing.assert_array_equal(per_window[:, 0], g["relaxed"])
    # D - B = 8 is divisible by k*_1 = 4: the trimming mode trims nothing
    assert mixed.operating_mode(13, 5, 4, 4) == ("trim", 0, 0, 0, 0)


# ----------------------------------------------------------------------------- operating modes

def test_operating_mode_reduces_to_the_sliding_and_relaxed_theorems():
    for B in range(1, 9):
        for K in (1, 2, 3, 4, 6, 8):
            for N in range(B, B + 3 * K + 2):
                # l = 0 (k*_0 = 1): Theorem "processing chain" stuffs (K - rem(N-B+1, K)) mod K
                mode, r, tr, st, s = mixed.operating_mode(N, B, K, 1)
                r_pc = (K - (N - B + 1) % K) % K
                assert tr == 0 and st == r_pc and s == r_pc
                # l = L (k*_l = K): Theorem "evalrelax" trims rem(N - B, K)
                mode, r, tr, st, s = mixed.operating_mode(N, B, K, K)
                assert mode == "trim" and tr == (N - B) % K and st == 0


def test_superfluous_sample_count_restores_the_downsampled_length():
    """After stuffing, the defragmented output of the mixed chain has
    (D - B)/k*_l + 1 samples; removing s of them must leave exactly
    ceil((N - B + 1)/k*_l), the length of Down_{k*_l}(Slide_{EvalStride_L})."""
    seen = set()
    for B in range(1, 10):
        for k in (1, 2, 3, 4):
            for m in (1, 2, 3, 4):
                K = k * m
                for N in range(B, B + 3 * K + 3):
                    mode, r, tr, st, s = mixed.operating_mode(N, B, K, k)
                    D = N - tr + st
                    assert (D - B + k) % K == 0 and (D - B) % k == 0 and D >= B
                    assert (D - B) // k + 1 - s == math.ceil((N - B + 1) / k)
                    seen.add(mode)
    assert seen == {"trim", "stuff"}


# ----------------------------------------------------------------------------- the main equality

def _sizes(B, K, nd):
    """Signal extents covering every residue modulo K (2-D: paired with a shift)."""
    n = list(range(B, B + K + 2))
    return [(1, w) for w in n] if nd == 1 else [(h, w) for h, w in zip(n, n[3:] + n[:3])]


@pytest.mark.parametrize("name", list(ARCHS))
def test_mixed_evaluation_equals_downsampled_dense_scanning(name):
    """Theorem "evalrelaxslide" (0 < l < L), Theorem "evalrelax" (l = L) and
    Theorem "processing chain" (l = 0) for every l and signal length."""
    layers, C, nd = _layers(name)
    ch, ks, us = _geometry(layers)
    L = len(ch)
    B, K = us[0], ks[L]
    rng = np.random.default_rng(8)
    modes = set()
    for (H, W) in _sizes(B[1] if nd == 1 else max(B), max(K), nd):
        if H < B[0] or W < B[1]:
            continue
        x = rng.standard_normal((C, H, W))
        dense = oracle.eval_stride(layers, x)
        for ell in range(L + 1):
            step = ks[ell]
            got = mixed.eval_relax_slide(layers, x, ell)
            want = mixed.dense_downsampled(layers, x, step)
            assert got.shape == want.shape == (layers[-1]["cout"], mixed.output_extent(H, B[0], step[0]),
                                               mixed.output_extent(W, B[1], step[1]))
            np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
            np.testing.assert_array_equal(want, dense[:, ::step[0], ::step[1]])
            for a, N in enumerate((H, W)):
                modes.add(mixed.operating_mode(N, B[a], K[a], step[a])[0])
    assert modes == {"trim", "stuff"}


def test_dummy_value_never_reaches_the_output():
    layers, C, nd = _layers("2d_mixed")
    ch, ks, us = _geometry(layers)
    B, K = us[0], ks[-1]
    x = np.random.default_rng(1).standard_normal((C, B[0] + 3, B[1] + 1))
    for ell in range(len(ch) + 1):
        modes = [mixed.operating_mode(N, B[a], K[a], ks[ell][a])[0] for a, N in enumerate(x.shape[1:])]
        a = mixed.eval_relax_slide(layers, x, ell, zeta=0.0)
        b = mixed.eval_relax_slide(layers, x, ell, zeta=1.0e6)
        np.testing.assert_array_equal(a, b)
        if "stuff" in modes:
            # the dummy value does reach the untrimmed intermediate representation
            ia = mixed.eval_relax_slide(layers, x, ell, upto=len(ch) - 1, zeta=0.0)
            ib = mixed.eval_relax_slide(layers, x, ell, upto=len(ch) - 1, zeta=1.0e6)
            assert not np.array_equal(ia, ib)


# ----------------------------------------------------------------------------- lemmas

def _prepared(layers, x, ell):
    """The trimmed/stuffed signal the mixed chain runs on, and its extents."""
    ch, ks, us = _geometry(layers)
    B, K = us[0], ks[-1]
    C, H, W = x.shape
    out = x
    D = []
    for a, N in enumerate((H, W)):
        mode, r, tr, st, s = mixed.operating_mode(N, B[a], K[a], ks[ell][a])
        D.append(N - tr + st)
    out = np.zeros((C, D[0], D[1]))
    h, w = min(H, D[0]), min(W, D[1])
    out[:, :h, :w] = x[:, :h, :w]
    return out, D


@pytest.mark.parametrize("name", ["1d_three", "2d_mixed", "2d_pool_first", "2d_c1"])
def test_lemma_extents_and_index_maps(name):
    """Lemma "evalrelax" (b) for the relaxed layers and Lemma "evalrelaxslide"
    (a)-(d): intermediate extents in closed form and every intermediate sample
    against EvalStride_j on the corresponding window."""
    layers, C, nd = _layers(name, seed=5)
    ch, ks, us = _geometry(layers)
    L = len(ch)
    B, K = us[0], ks[L]
    H = 1 if nd == 1 else B[0] + K[0] + 1
    W = B[1] + 2 * K[1] + 1
    x = np.random.default_rng(6).standard_normal((C, H, W))
    for ell in range(L + 1):
        xp, D = _prepared(layers, x, ell)
        t = [(D[a] - B[a] + ks[ell][a]) // K[a] for a in range(2)]
        for a in range(2):
            assert D[a] == B[a] + K[a] * t[a] - ks[ell][a] and t[a] >= 1
        for j in range(1, L + 1):
            rep = mixed.eval_relax_slide(layers, x, ell, upto=j)
            Cj = rep.shape[1]
            n_desc = _descriptors_upto(layers, j)
            if j <= ell:
                # one fragment; Lemma "evalrelax" (b): W_j - u_j = (D - B)/k*_j
                assert rep.shape[0] == 1
                Wj = rep.shape[2:]
                for a in range(2):
                    assert (D[a] - B[a]) % ks[j][a] == 0
                    assert Wj[a] - us[j][a] == (D[a] - B[a]) // ks[j][a]
                if j == ell:
                    for a in range(2):  # Lemma "evalrelaxslide" (a)
                        assert Wj[a] == (D[a] - B[a]) // ks[ell][a] + us[ell][a]
                # (c): EvalStride_j on the window at k*_j (i - 1) is the u_j block at i
                ni, nj = Wj[0] - us[j][0] + 1, Wj[1] - us[j][1] + 1
                ii, jj = np.meshgrid(np.arange(ni), np.arange(nj), indexing="ij")
                ref = oracle.eval_stride(layers, xp, windows=(ks[j][0] * ii.reshape(-1), ks[j][1] * jj.reshape(-1)),
                                         upto=n_desc, patch=tuple(B))
                ref = ref.reshape(ni, nj, Cj, us[j][0], us[j][1])
                for i in range(ni):
                    for k in range(nj):
                        np.testing.assert_allclose(rep[0, :, i:i + us[j][0], k:k + us[j][1]], ref[i, k],
                                                   rtol=1e-12, atol=1e-12)
            else:
                Fh, Fw = ks[j][0] // ks[ell][0], ks[j][1] // ks[ell][1]
                assert rep.shape[0] == Fh * Fw  # (b): U^col = k*_j / k*_l
                for a, Fa in enumerate((Fh, Fw)):
                    assert rep.shape[2 + a] - us[j][a] + 1 == (K[a] // ks[j][a]) * t[a]
                # (d): window k*_l (i - 1) sits at sample div(i-1, F) + mu of fragment rem(i-1, F)
                Wl = [(D[a] - B[a]) // ks[ell][a] + us[ell][a] for a in range(2)]
                ni, nj = Wl[0] - us[ell][0] + 1, Wl[1] - us[ell][1] + 1
                ii, jj = np.meshgrid(np.arange(ni), np.arange(nj), indexing="ij")
                ref = oracle.eval_stride(layers, xp,
                                         windows=(ks[ell][0] * ii.reshape(-1), ks[ell][1] * jj.reshape(-1)),
                                         upto=n_desc, patch=tuple(B))
                ref = ref.reshape(ni, nj, Cj, us[j][0], us[j][1])
                for i in range(ni):
                    for k in range(nj):
                        f = (i % Fh) * Fw + (k % Fw)
                        y, z = i // Fh, k // Fw
                        np.testing.assert_allclose(rep[f, :, y:y + us[j][0], z:z + us[j][1]], ref[i, k],
                                                   rtol=1e-12, atol=1e-12)
