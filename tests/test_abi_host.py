"""Host-side checks of the C-ABI library (no GPU): it loads, exports every
function the header declares, and its host-only geometry agrees with the
oracle's brute-force receptive field and with the paper's closed forms."""
import os
import re

import numpy as np
import pytest

import oracle
from paper_1508_06904_amd import dss, workloads as wl
from tests.test_oracle import chain_layers, lemma_a_u

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "dss.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dss_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    L = dss.lib()
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(dss.EXPORTS)
    assert L.dss_version().decode().count(".") == 2


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """Without libdss.so the binding raises at its first call: there is no
    fallback path that could compute anything."""
    monkeypatch.setattr(dss, "_lib", None)
    monkeypatch.setattr(dss, "LIB_PATH", str(tmp_path / "libdss.so"))
    with pytest.raises(dss.DssError, match="does not exist"):
        dss.lib()
    with pytest.raises(dss.DssError):
        dss.Plan.from_workload(wl.make("c1_64x64"))


def test_status_strings():
    L = dss.lib()
    for s in range(6):
        assert L.dss_status_string(s)


NAMED = {
    # name: (arch, C, H, W, ndim, B, K, r)
    "c1": (wl.arch_c1(), 1, 64, 64, 2, (28, 28), (4, 4), (3, 3)),
    "c2": (wl.arch_c2(), 1, 1, 1 << 20, 1, (1, 120), (1, 8), (0, 7)),
    "c3": (wl.arch_c3(), 3, 512, 512, 2, (68, 68), (8, 8), (3, 3)),
    "c4": (wl.arch_c4(), 3, 1080, 1920, 2, (68, 68), (8, 8), (3, 3)),
    "c5": (wl.arch_c5(), 3, 2160, 3840, 2, (156, 156), (16, 16), (11, 11)),
}


def theorem_r(N, B, K):
    """Stuffing count of Theorem 'processing chain' (Sect. 4.3)."""
    return 0 if (N - B + 1) % K == 0 else K - (N - B + 1) % K


@pytest.mark.parametrize("name", list(NAMED))
def test_named_geometry(name):
    arch, C, H, W, nd, B, K, r = NAMED[name]
    layers = wl.init_layers(arch, np.random.default_rng(0))
    g = dss.chain_geometry(layers, nd, C, H, W)
    assert (g["B_h"], g["B_w"]) == B == tuple(oracle.receptive_field(layers))
    assert (g["K_h"], g["K_w"]) == K
    assert (g["r_h"], g["r_w"]) == r == (theorem_r(H, B[0], K[0]), theorem_r(W, B[1], K[1]))
    assert (g["out_h"], g["out_w"]) == (H - B[0] + 1, W - B[1] + 1)
    assert (g["D_h"], g["D_w"]) == (H + r[0], W + r[1])
    assert g["out_c"] == [l for l in layers if l["kind"] == "conv"][-1]["cout"]
    # per-layer extents against Lemma 'processing chain' (a)-(c)
    ch = chain_layers(layers)
    D = (g["D_h"], g["D_w"])
    for axis, key in ((0, "h"), (1, "w")):
        u, kstar = lemma_a_u(ch, B[axis], axis)
        for j in range(len(ch) + 1):
            lg = dss.chain_layer_geometry(layers, nd, C, H, W, j)
            assert lg["u_" + key] == u[j]
            assert lg["kstar_" + key] == kstar[j]
            s = sum(kstar[mu - 1] * (ch[mu - 1][0][axis] - 1) for mu in range(1, j + 1))
            assert (D[axis] - kstar[j] + 1 - s) % kstar[j] == 0
            assert lg["U_" + key] == (D[axis] - kstar[j] + 1 - s) // kstar[j]          # Lemma (b)
            assert lg["U_" + key] - u[j] + 1 == (D[axis] - B[axis] + 1) // kstar[j]    # Lemma (c)
    last = dss.chain_layer_geometry(layers, nd, C, H, W, len(ch))
    assert last["F"] == K[0] * K[1] and last["u_h"] == last["u_w"] == 1


def direct_conv_flops(layers, nd, C, H, W):
    """Convolution flops of the sliding evaluation, counted per layer from the
    evaluation counts of Sect. 5.1: U^col_{j-1} (U^row_{j-1} - c_j + 1) evaluations
    of f_j per axis, each Cin * c_h * c_w multiply-adds per output channel."""
    ch = chain_layers(layers)
    convs = [l for l in layers if l["kind"] == "conv"]
    total, ci = 0.0, 0
    for j, (c, k) in enumerate(ch, start=1):
        prev = dss.chain_layer_geometry(layers, nd, C, H, W, j - 1)
        has_conv = dss.chain_layer_geometry(layers, nd, C, H, W, j)["has_conv"]
        if not has_conv:
            continue
        l = convs[ci]
        ci += 1
        n_eval = prev["F"] * (prev["U_h"] - c[0] + 1) * (prev["U_w"] - c[1] + 1)
        total += 2.0 * n_eval * l["cout"] * l["cin"] * c[0] * c[1]
    return total


@pytest.mark.parametrize("name", list(NAMED))
def test_conv_flop_accounting(name):
    arch, C, H, W, nd, *_ = NAMED[name]
    layers = wl.init_layers(arch, np.random.default_rng(0))
    g = dss.chain_geometry(layers, nd, C, H, W)
    assert g["conv_flops"] == pytest.approx(direct_conv_flops(layers, nd, C, H, W), rel=1e-12)


def test_hd_frame_flops_and_speedup_shape():
    """The HD configuration: about 19.8 TFLOP of convolution per frame for the
    sliding evaluation, against EvalStride's (N-B+1)^2 * per-window cost."""
    layers = wl.init_layers(wl.arch_c4(), np.random.default_rng(0))
    g = dss.chain_geometry(layers, 2, 3, 1080, 1920)
    assert 19.7e12 < g["conv_flops"] < 20.0e12
    assert g["workspace_bytes"] > 0 and g["workspace_bytes"] % 256 == 0


def test_every_stuffing_amount():
    """Signal extents B .. B+K cover every stuffing amount r in [0, K-1]."""
    layers = wl.init_layers([("conv", 1, 2, 3, 3, "relu"), ("pool", 2, 2), ("conv", 2, 2, 2, 2, "relu"),
                             ("pool", 3, 3), ("conv", 2, 1, 2, 2, "none")], np.random.default_rng(0))
    B = oracle.receptive_field(layers)
    seen = set()
    for n in range(B[0], B[0] + 7):
        g = dss.chain_geometry(layers, 2, 1, n, n + 1)
        assert g["r_h"] == theorem_r(n, B[0], 6)
        assert (g["D_h"] - g["B_h"] + 1) % g["K_h"] == 0
        seen.add(g["r_h"])
    assert seen == set(range(6))


def test_paper_sweep_fragment_count():
    for L in (3, 4, 12, 15):
        layers = wl.init_layers(wl.arch_paper_sweep(L, maps=4), np.random.default_rng(0))
        B = oracle.receptive_field(layers)
        g = dss.chain_geometry(layers, 2, 1, 240, 320)
        assert (g["B_h"], g["B_w"]) == B
        if L == 12:
            assert g["K_h"] * g["K_w"] == 64


@pytest.mark.parametrize("bad", ["cin_mismatch", "zero_filter", "empty", "ndim", "1d_fh", "small_signal", "act"])
def test_validation_errors(bad):
    layers = wl.init_layers(wl.arch_c1(), np.random.default_rng(0))
    nd, C, H, W = 2, 1, 64, 64
    want = 1
    if bad == "cin_mismatch":
        layers[2]["cin"] = 5
        layers[2]["weight"] = np.zeros((8, 5, 5, 5), np.float32)
    elif bad == "zero_filter":
        layers[0]["fh"] = 0
        layers[0]["weight"] = np.zeros((4, 1, 0, 5), np.float32)
    elif bad == "empty":
        layers = []
    elif bad == "ndim":
        nd, want = 3, 3
    elif bad == "1d_fh":
        nd = 1
    elif bad == "small_signal":
        H, want = 27, 2
    elif bad == "act":
        layers[0]["act"] = "none"
        dss_layers = layers
    with pytest.raises(dss.DssError) as e:
        if bad == "act":
            la = dss._LayerArray(layers)
            la.arr[0].act = 7
            g = dss.Geometry()
            dss._check(dss.lib().dss_chain_geometry(la.arr, la.n, nd, C, 0, H, W, 0, dss.ctypes.byref(g)), "geom")
        else:
            dss.chain_geometry(layers, nd, C, H, W)
    assert e.value.status == want
    assert dss.lib().dss_last_error().decode() != ""


# ----------------------------------------------------------------------------- mixed evaluation geometry

from oracle import mixed  # noqa: E402
from tests.test_oracle_mixed import ARCHS as MIXED_ARCHS  # noqa: E402


@pytest.mark.parametrize("name", list(MIXED_ARCHS))
def test_mixed_geometry_matches_the_oracle_algorithm(name):
    """Per mixed level and signal length: trimming/stuffing amounts, output
    extents, per-layer fragment counts and extents and the convolution flop count
    agree with the oracle's literal mixed algorithm (its tensor shapes)."""
    arch, C, nd = MIXED_ARCHS[name]
    layers = wl.init_layers(arch, np.random.default_rng(0))
    ch = mixed.chain_of(layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    L, B, K = len(ch), us[0], ks[-1]
    rng = np.random.default_rng(2)
    sizes = [(1, w) for w in range(B[1], B[1] + K[1] + 2)] if nd == 1 else \
        [(B[0] + a, B[1] + b) for a in range(K[0] + 1) for b in (0, K[1] - 1, K[1] + 2)]
    for (H, W) in sizes:
        x = rng.standard_normal((C, H, W))
        for ell in range(L + 1):
            g = dss.chain_geometry(layers, nd, C, H, W, ell=ell)
            assert g["ell"] == ell and (g["step_h"], g["step_w"]) == ks[ell]
            for a, N, key in ((0, H, "h"), (1, W, "w")):
                mode, r, tr, st, s = mixed.operating_mode(N, B[a], K[a], ks[ell][a])
                assert (g["trim_" + key], g["r_" + key]) == (tr, st)
                assert g["D_" + key] == N - tr + st
                assert g["out_" + key] == mixed.output_extent(N, B[a], ks[ell][a])
            flops = 0.0
            prev = (1, C, g["D_h"], g["D_w"])
            for j in range(1, L + 1):
                lg = dss.chain_layer_geometry(layers, nd, C, H, W, j, ell=ell)
                rep = mixed.eval_relax_slide(layers, x, ell, upto=j)
                assert (lg["F"], lg["channels"], lg["U_h"], lg["U_w"]) == rep.shape
                assert lg["relaxed"] == (1 if j <= ell else 0)
                conv = ch[j - 1]["conv"]
                if conv is not None:
                    Eh, Ew = prev[2] - conv["fh"] + 1, prev[3] - conv["fw"] + 1
                    flops += 2.0 * prev[0] * Eh * Ew * conv["cout"] * conv["cin"] * conv["fh"] * conv["fw"]
                prev = rep.shape
            assert g["conv_flops"] == flops
            lg0 = dss.chain_layer_geometry(layers, nd, C, H, W, 0, ell=ell)
            assert (lg0["F"], lg0["U_h"], lg0["U_w"]) == (1, g["D_h"], g["D_w"])


def test_mixed_level_zero_is_the_dense_geometry():
    layers = wl.init_layers(wl.arch_c4(), np.random.default_rng(0))
    a = dss.chain_geometry(layers, 2, 3, 1080, 1920)
    b = dss.chain_geometry(layers, 2, 3, 1080, 1920, ell=0)
    assert a == b and a["trim_h"] == a["trim_w"] == 0 and a["step_h"] == a["step_w"] == 1


def test_mixed_hd_frame_work_shrinks_with_the_level():
    """The relaxed layers evaluate one fragment: the convolution work falls by
    about k*_l^2 in the relaxed part (Sect. 5 counts for the relaxed fashion)."""
    layers = wl.init_layers(wl.arch_c4(), np.random.default_rng(0))
    # five chain layers; the last two have no pool, so k*_3 = k*_4 = k*_5 = 8 and
    # relaxing them changes nothing
    f = [dss.chain_geometry(layers, 2, 3, 1080, 1920, ell=l)["conv_flops"] for l in range(6)]
    assert f[0] > f[1] > f[2] > f[3] == f[4] == f[5]
    g5 = dss.chain_geometry(layers, 2, 3, 1080, 1920, ell=5)
    assert (g5["out_h"], g5["out_w"]) == (-(-(1080 - 67) // 8), -(-(1920 - 67) // 8))


@pytest.mark.parametrize("ell", [-1, 6])
def test_mixed_level_out_of_range(ell):
    layers = wl.init_layers(wl.arch_c4(), np.random.default_rng(0))
    with pytest.raises(dss.DssError) as e:
        dss.chain_geometry(layers, 2, 3, 512, 512, ell=ell)
    assert e.value.status == 1
    with pytest.raises(dss.DssError) as e:
        dss.chain_layer_geometry(layers, 2, 3, 512, 512, 1, ell=ell)
    assert e.value.status == 1


# ----------------------------------------------------------------------------- strided baseline geometry


@pytest.mark.parametrize("L", [1, 4, 7, 12, 15])
def test_stride_geometry_flops(L):
    """Conv flops of the patch-by-patch baseline: per window sum_j 2 E_j,h E_j,w Cout Cin c_h c_w
    with E_j = k_j u_j = u_{j-1} - c_j + 1 (Lemma (a)), times the batch size; the
    workspace grows linearly with the batch."""
    layers = wl.init_layers(wl.arch_paper_sweep(L, maps=16), np.random.default_rng(0))
    ch = mixed.chain_of(layers)
    us = mixed.strided_extents(ch)
    per = 0.0
    for j, e in enumerate(ch, start=1):
        if e["conv"] is not None:
            Eh, Ew = e["k"][0] * us[j][0], e["k"][1] * us[j][1]
            assert (Eh, Ew) == (us[j - 1][0] - e["c"][0] + 1, us[j - 1][1] - e["c"][1] + 1)
            c = e["conv"]
            per += 2.0 * Eh * Ew * c["cout"] * c["cin"] * c["fh"] * c["fw"]
    for count in (1, 7, 1000):
        ws, fl = dss.chain_stride_geometry(layers, 2, 1, count)
        assert fl == pytest.approx(count * per, rel=1e-12)
        assert ws >= 2 * count * us[0][0] * us[0][1] * 4
    # per window, the baseline does at least the dense evaluation's work per output
    g = dss.chain_geometry(layers, 2, 1, 240, 320)
    assert per >= g["conv_flops"] / (g["out_h"] * g["out_w"]) * (0.99 if L == 1 else 1.0)


@pytest.mark.parametrize("count", [0, -3])
def test_stride_geometry_rejects_empty_batch(count):
    layers = wl.init_layers(wl.arch_c1(), np.random.default_rng(0))
    with pytest.raises(dss.DssError) as e:
        dss.chain_stride_geometry(layers, 2, 1, count)
    assert e.value.status == 1


# ----------------------------------------------------------------------------- dilated fashion geometry

from oracle import dilate as odilate  # noqa: E402


@pytest.mark.parametrize("name", list(MIXED_ARCHS))
def test_dilate_geometry_matches_oracle(name):
    """V_j of every layer equals the oracle's EvalDilate_j extents; the last one is
    the dense output; with no stuffing needed, the convolution work equals the
    sliding evaluation's (the appendix's complexity remark: equal evaluation counts)."""
    arch, C, nd = MIXED_ARCHS[name]
    layers = wl.init_layers(arch, np.random.default_rng(0))
    ch = mixed.chain_of(layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    B, K = us[0], ks[-1]
    H = 1 if nd == 1 else B[0] - 1 + 2 * K[0]
    W = B[1] - 1 + 3 * K[1]
    x = np.random.default_rng(1).standard_normal((C, H, W))
    for j in range(len(ch) + 1):
        vh, vw, ws, fl = dss.chain_dilate_geometry(layers, nd, C, H, W, j)
        assert (vh, vw) == odilate.eval_dilate(layers, x, upto=j).shape[1:]
    g = dss.chain_geometry(layers, nd, C, H, W)
    assert (g["r_h"], g["r_w"]) == (0, 0)
    assert (vh, vw) == (g["out_h"], g["out_w"])
    assert fl == g["conv_flops"]


def test_dilate_geometry_errors():
    layers = wl.init_layers(wl.arch_c1(), np.random.default_rng(0))
    with pytest.raises(dss.DssError) as e:
        dss.chain_dilate_geometry(layers, 2, 1, 27, 64, 3)
    assert e.value.status == 2
    with pytest.raises(dss.DssError) as e:
        dss.chain_dilate_geometry(layers, 2, 1, 64, 64, 4)
    assert e.value.status == 1


# ----------------------------------------------------------------------------- backward geometry


@pytest.mark.parametrize("name", ["c1", "c3", "c4"])
def test_backward_geometry(name):
    """Gradient buffer sizes are the weight and bias counts; the work is the
    forward convolutions plus a weight gradient and an input gradient of the same
    size each (the first layer's input gradient only when the signal's is wanted)."""
    arch, C, H, W, nd, B, K, r = NAMED[name]
    layers = wl.init_layers(arch, np.random.default_rng(0))
    g = dss.chain_geometry(layers, nd, C, H, W)
    convs = [l for l in layers if l["kind"] == "conv"]
    ws1, wf, bf, fl1 = dss.chain_backward_geometry(layers, nd, C, H, W, True)
    ws0, wf0, bf0, fl0 = dss.chain_backward_geometry(layers, nd, C, H, W, False)
    assert wf == wf0 == sum(l["cout"] * l["cin"] * l["fh"] * l["fw"] for l in convs)
    assert bf == bf0 == sum(l["cout"] for l in convs)
    assert fl1 == pytest.approx(3 * g["conv_flops"], rel=1e-12)
    ch = mixed.chain_of(layers)
    first = ch[0]["conv"]
    D = (g["D_h"], g["D_w"])
    first_flops = 2.0 * (D[0] - first["fh"] + 1) * (D[1] - first["fw"] + 1) * first["cout"] * first["cin"] * \
        first["fh"] * first["fw"]
    assert fl0 == pytest.approx(3 * g["conv_flops"] - first_flops, rel=1e-12)
    assert ws1 >= ws0 >= 2 * g["workspace_bytes"] // 2
