"""Pins for the dilated evaluation in the oracle (no GPU).

`oracle.dilate` follows the appendix on functions applied in a dilated fashion.
It is pinned by the figures' sizes, by Remark "dilated-fragment" (Dilate equals
Defrag after Slide after Frag, checked against the literal vec-based fragment
operators), by the closed forms of Lemma "evaldilate" (a), (b), by its index map
(d) against EvalStride on every window, by Remark "evaldilate" (b) against the
oracle's sliding evaluation, and by the final layer being the dense output."""
import numpy as np
import pytest

import oracle
from oracle import dilate, fragment, mixed
from paper_1508_06904_amd import workloads as wl
from tests.test_oracle_mixed import ARCHS, _descriptors_upto


def test_dilated_subsignal_figure_sizes():
    """Figure of the dilated subsignal: D = 8, d = 3, k = 2 gives indices
    1..D - k(d - 1) = 4, the i-th one holding samples i, i+2, i+4."""
    xi = np.arange(1.0, 9.0)
    assert 8 - 2 * (3 - 1) == 4
    for i in range(1, 5):
        np.testing.assert_array_equal(dilate.dilated_subsignal(xi, 3, 2, i), [i, i + 2, i + 4])
    with pytest.raises(AssertionError):
        dilate.dilated_subsignal(xi, 3, 2, 5)
    # k = 1 is ordinary subsignal extraction
    np.testing.assert_array_equal(dilate.dilated_subsignal(xi, 3, 1, 6), [6, 7, 8])


def test_dilate_figure_sizes_and_remark():
    """Figure of Dilate: max with c = 2, stride k = 2 on D = 6 samples gives
    D - k(c - 1) = 4 outputs, equal to Defrag_2(Slide_max(Frag_2(xi)))
    (Remark "dilated-fragment")."""
    xi = np.array([3.0, 9.0, 1.0, 4.0, 7.0, 2.0])
    got = dilate.dilate(np.max, xi, 2, 2)
    np.testing.assert_array_equal(got, [3.0, 9.0, 7.0, 4.0])
    fr = fragment.frag(xi[:, None], 2)                       # 3 x 2
    sl = np.maximum(fr[:-1], fr[1:])                          # Slide_max, c = 2
    np.testing.assert_array_equal(fragment.defrag(sl, 2)[:, 0], got)


@pytest.mark.parametrize("k,c,q", [(2, 3, 5), (3, 2, 4), (4, 3, 6), (1, 4, 7)])
def test_remark_dilated_fragment_for_conv(k, c, q):
    """Dilate_{(f,k)} = Defrag_k o Slide_f o Frag_k for a random linear f with c taps."""
    rng = np.random.default_rng(k * 10 + c)
    xi = rng.standard_normal(k * q)
    w = rng.standard_normal(c)
    f = lambda v: float(np.dot(w, v))
    got = dilate.dilate(f, xi, c, k)
    fr = fragment.frag(xi[:, None], k)                       # q x k
    sl = np.stack([[f(fr[i:i + c, s]) for s in range(k)] for i in range(q - c + 1)])
    np.testing.assert_allclose(fragment.defrag(sl, k)[:, 0], got, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("name", list(ARCHS))
def test_final_layer_is_the_dense_output(name):
    arch, C, nd = ARCHS[name]
    layers = wl.init_layers(arch, np.random.default_rng(3))
    B = mixed.strided_extents(mixed.chain_of(layers))[0]
    rng = np.random.default_rng(4)
    for extra in (0, 1, 3, 7):
        H = 1 if nd == 1 else B[0] + extra
        W = B[1] + 2 * extra + 1
        x = rng.standard_normal((C, H, W))
        got = dilate.eval_dilate(layers, x)
        np.testing.assert_allclose(got, oracle.eval_stride(layers, x), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("name", ["1d_three", "2d_mixed", "2d_pool_first", "2d_c1"])
def test_lemma_evaldilate(name):
    """(a) V_j = D - sum_{mu<=j} k*_{mu-1}(c_mu + k_mu - 2); (b) V_j - k*_j(u_j - 1)
    = D - B + 1; (d) EvalStride_j on window i = DilatedSubsignal_{(u_j, k*_j)}(EvalDilate_j, i)."""
    arch, C, nd = ARCHS[name]
    layers = wl.init_layers(arch, np.random.default_rng(5))
    ch = mixed.chain_of(layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    B = us[0]
    H = 1 if nd == 1 else B[0] + 5
    W = B[1] + 6
    x = np.random.default_rng(6).standard_normal((C, H, W))
    ni, nj = H - B[0] + 1, W - B[1] + 1
    ii, jj = np.meshgrid(np.arange(ni), np.arange(nj), indexing="ij")
    for j in range(len(ch) + 1):
        rep = dilate.eval_dilate(layers, x, upto=j)
        for a, D in enumerate((H, W)):
            V = D - sum(ks[mu - 1][a] * (ch[mu - 1]["c"][a] + ch[mu - 1]["k"][a] - 2) for mu in range(1, j + 1))
            assert rep.shape[1 + a] == V
            assert V - ks[j][a] * (us[j][a] - 1) == D - B[a] + 1
        if j == 0:
            np.testing.assert_array_equal(rep, x)
            continue
        ref = oracle.eval_stride(layers, x, windows=(ii.reshape(-1), jj.reshape(-1)),
                                 upto=_descriptors_upto(layers, j), patch=tuple(B))
        ref = ref.reshape(ni, nj, rep.shape[0], us[j][0], us[j][1])
        for i in range(ni):
            for k in range(nj):
                got = rep[:, i:i + ks[j][0] * (us[j][0] - 1) + 1:ks[j][0], k:k + ks[j][1] * (us[j][1] - 1) + 1:ks[j][1]]
                np.testing.assert_allclose(got, ref[i, k], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("name", ["2d_mixed", "2d_pool_first", "2d_c1", "2d_pool_pool"])
def test_remark_evaldilate_b(name):
    """EvalDilate_j = Defrag_{k*_j}(EvalSlide_j) on a signal that needs no stuffing."""
    arch, C, nd = ARCHS[name]
    layers = wl.init_layers(arch, np.random.default_rng(7))
    ch = mixed.chain_of(layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    B, K = us[0], ks[-1]
    H, W = B[0] - 1 + 2 * K[0], B[1] - 1 + 3 * K[1]
    x = np.random.default_rng(8).standard_normal((C, H, W))
    for a, N in enumerate((H, W)):
        assert mixed.operating_mode(N, B[a], K[a], 1) == ("trim", 0, 0, 0, 0)
    for j in range(1, len(ch) + 1):
        slide = mixed.eval_relax_slide(layers, x, 0, upto=j)
        d = fragment.defrag_tensor(slide, ks[j][0], ks[j][1], 1, 1)[0]
        np.testing.assert_allclose(dilate.eval_dilate(layers, x, upto=j), d, rtol=1e-12, atol=1e-12)
