"""GPU parity of the relaxed / mixed evaluation (dss_eval_mixed, dss_eval_slide
with a mixed level) against the oracle's definition Down_{k*_l}(Slide_{EvalStride_L})
and against its literal mixed algorithm for the intermediate layers.
binary32 within 1e-4 * max|oracle|, bfloat16 within 2e-2 * max|oracle|,
integer-valued data bit-exact."""
import numpy as np
import pytest

import oracle
from oracle import mixed
from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import assert_close, log, oracle_layers, sampled_windows, to_device
from tests.test_gpu_parity import CHAINS, EXACT_ARCH

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dss.lib()
    yield
    torch.cuda.synchronize()


def gpu_mixed(plan, x, ell, dtype="f32"):
    import torch
    out = plan.eval_mixed(to_device(x, dtype), ell)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def gpu_dense(plan, x, dtype="f32"):
    import torch
    out = plan.eval_dense(to_device(x, dtype))
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def levels(layers):
    return len(mixed.chain_of(layers))


def _sizes(B, K, nd):
    """Extents that exercise both operating modes on both axes."""
    if nd == 1:
        return [(1, B[1] + 40 * K[1] + d) for d in (0, K[1] // 2, K[1] - 1)]
    return [(B[0] + 2 * K[0] + a, B[1] + 3 * K[1] + b) for a, b in ((0, K[1] - 1), (K[0] - 1, 1), (K[0] // 2, 0))]


@pytest.mark.parametrize("name", list(CHAINS))
def test_mixed_matches_downsampled_dense_definition(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    ch = mixed.chain_of(w0.layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    plan = dss.Plan(w0.layers, nd, C)
    modes = set()
    for (H, W) in _sizes(us[0], ks[-1], nd):
        w = wl.custom(arch, C, H, W, seed=H + W, value_kind="normal")
        w.layers = w0.layers  # the plan's weights; only the signal changes per size
        dense = gpu_dense(plan, w.x)
        for ell in range(len(ch) + 1):
            log("chain %s %dx%d ell=%d" % (name, H, W, ell))
            g = plan.geometry(H, W, ell)
            modes.add(("trim" if g["trim_h"] else "stuff" if g["r_h"] else "none",
                       "trim" if g["trim_w"] else "stuff" if g["r_w"] else "none"))
            out = gpu_mixed(plan, w.x, ell)
            ref = mixed.dense_downsampled(w.layers, w.x, ks[ell])
            assert_close(out, ref, F32_TOL, "%s ell=%d" % (name, ell))
            # the same kernels see the same samples in the same order: bit-identical
            # to the dense evaluation downsampled
            np.testing.assert_array_equal(out, dense[:, ::ks[ell][0], ::ks[ell][1]])
    flat = {m for pair in modes for m in pair}
    assert "trim" in flat and "stuff" in flat


@pytest.mark.parametrize("kernel", ["mfma", "direct"])
def test_mixed_exact_integer_chain(kernel, monkeypatch):
    if kernel == "direct":
        monkeypatch.setenv("DSS_CONV_KERNEL", "direct")
    w = wl.custom(EXACT_ARCH, 16, 45, 50, seed=3, weight_kind="int", value_kind="int")
    plan = dss.Plan(w.layers, 2, 16)
    ks = mixed.stride_products(mixed.chain_of(w.layers))
    for ell in range(levels(w.layers) + 1):
        log("exact chain %s ell=%d" % (kernel, ell))
        out = gpu_mixed(plan, w.x, ell)
        ref = mixed.dense_downsampled(w.layers, w.x, ks[ell])
        assert np.abs(ref).max() < 2 ** 23
        np.testing.assert_array_equal(out, ref)


@pytest.mark.parametrize("name", ["2d_mfma_mixed", "2d_pool_pool"])
def test_mixed_bf16(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    ch = mixed.chain_of(w0.layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    B, K = us[0], ks[-1]
    w = wl.custom(arch, C, B[0] + 2 * K[0] + 3, B[1] + 3 * K[1] + 1, seed=4, dtype="bf16")
    plan = dss.Plan(w.layers, nd, C, "bf16")
    for ell in range(len(ch) + 1):
        log("bf16 chain %s ell=%d" % (name, ell))
        out = gpu_mixed(plan, w.x, ell, "bf16")
        ref = mixed.dense_downsampled(oracle_layers(w.layers, "bf16"), w.x, ks[ell])
        assert_close(out, ref, BF16_TOL, "%s ell=%d" % (name, ell))


def test_relaxed_figure_example_gpu():
    """The relaxed-fashion figure of the appendix (two-sample transformation,
    max-pool stride 4, D = 13): relaxed output [4, 4, 3]."""
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "relaxed_fig.json")) as f:
        g = json.load(f)
    layers = [dict(l, weight=np.array(l["weight"]), bias=np.array(l["bias"])) if l["kind"] == "conv" else l
              for l in g["layers"]]
    plan = dss.Plan(layers, 1, 1)
    x = np.array(g["signal"], dtype=np.float32)[None, None, :]
    np.testing.assert_array_equal(gpu_mixed(plan, x, 1)[0, 0], g["relaxed"])
    np.testing.assert_array_equal(gpu_mixed(plan, x, 0)[0, 0], g["dense"])


@pytest.mark.parametrize("name", ["2d_mfma_mixed", "2d_pool_first", "1d_c2_like"])
def test_mixed_intermediate_layers(name):
    """dss_eval_slide at a mixed level against the oracle's literal mixed
    algorithm after every layer (relaxed layers: one fragment, Lemma
    "evalrelaxslide" (c); sliding layers: k*_j/k*_l fragments, (d))."""
    import torch
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    ch = mixed.chain_of(w0.layers)
    ks, us = mixed.stride_products(ch), mixed.strided_extents(ch)
    B, K = us[0], ks[-1]
    H = 1 if nd == 1 else B[0] + K[0] + 3
    W = B[1] + 2 * K[1] + 5
    w = wl.custom(arch, C, H, W, seed=6, value_kind="normal")
    plan = dss.Plan(w.layers, nd, C)
    xd = to_device(w.x, "f32")
    for ell in range(len(ch) + 1):
        for j in range(len(ch) + 1):
            log("intermediate %s ell=%d j=%d" % (name, ell, j))
            got = plan.eval_slide(xd, j, ell=ell)
            torch.cuda.synchronize()
            got = got.cpu().numpy().astype(np.float64)
            if j == 0:
                g = plan.geometry(H, W, ell)
                ref = np.zeros((1, C, g["D_h"], g["D_w"]))
                h, ww = min(H, g["D_h"]), min(W, g["D_w"])
                ref[0, :, :h, :ww] = w.x[:, :h, :ww]
                np.testing.assert_array_equal(got, ref)
                continue
            ref = mixed.eval_relax_slide(w.layers, w.x, ell, upto=j)
            assert_close(got, ref, F32_TOL, "%s ell=%d j=%d" % (name, ell, j))


@pytest.mark.parametrize("name,ells,max_phases", [("c2_1d_1m", (1, 2, 3), None), ("c4_hd", (1, 2, 3), None),
                                                  ("c5_4k", (2, 4), 32)])
def test_named_full_size_mixed_sampled(name, ells, max_phases):
    """Full-size workloads at several mixed levels; the oracle checks a seeded
    sample of output positions (corners, edges and every fragment phase of the
    remaining sliding part)."""
    w = wl.make(name)
    plan = dss.Plan.from_workload(w)
    H, W = w.x.shape[1:]
    for ell in ells:
        g = plan.geometry(H, W, ell)
        log("%s full size ell=%d step=%dx%d out=%dx%d" % (name, ell, g["step_h"], g["step_w"], g["out_h"], g["out_w"]))
        out = gpu_mixed(plan, w.x, ell, w.dtype)
        assert out.shape == (g["out_c"], g["out_h"], g["out_w"])
        assert np.all(np.isfinite(out))
        Gh, Gw = g["K_h"] // g["step_h"], g["K_w"] // g["step_w"]
        i, j = sampled_windows(g["out_h"], g["out_w"], Gh, Gw, per_phase=1, max_phases=max_phases, seed=ell)
        log("  checking %d output positions" % len(i))
        ref = oracle.eval_stride(oracle_layers(w.layers, w.dtype), w.x, windows=(g["step_h"] * i, g["step_w"] * j))
        assert_close(out[:, i, j].T, ref, BF16_TOL if w.dtype == "bf16" else F32_TOL, "%s ell=%d" % (name, ell))


def test_mixed_level_zero_is_dense_bit_exact():
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    w = wl.custom(arch, C, 66, 71, seed=21)
    plan = dss.Plan(w.layers, nd, C)
    np.testing.assert_array_equal(gpu_mixed(plan, w.x, 0), gpu_dense(plan, w.x))


def test_mixed_errors_leave_output_untouched():
    import torch
    w = wl.make("c1_64x64")
    plan = dss.Plan.from_workload(w)
    out = torch.full((1, 10, 10), 7.0, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    xd = to_device(w.x, "f32")
    stream = dss._stream(None)
    for bad in (-1, 4):
        st = dss.lib().dss_eval_mixed(plan.handle, dss._ptr(xd), 64, 64, bad, dss._ptr(out), dss._ptr(ws), ws.numel(),
                                      stream)
        assert st == 1 and "mixed level" in dss.lib().dss_last_error().decode()
    # a workspace too small for the level is rejected before anything runs
    st = dss.lib().dss_eval_mixed(plan.handle, dss._ptr(xd), 64, 64, 1, dss._ptr(out), dss._ptr(ws), 1024, stream)
    assert st == 2
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)


def test_mixed_timing_records():
    w = wl.make("c3_512", H=120, W=130, widths=(16, 32, 64, 128))
    plan = dss.Plan.from_workload(w)
    for ell in (1, 2, 3):
        plan.set_timing(True)
        gpu_mixed(plan, w.x, ell)
        recs = plan.timings()
        names = [r["kernel"] for r in recs]
        # the final 1x1 projection is folded into the conv6x6 epilogue
        assert names[0] == "stuff_pack" and names[-1] == "defrag_sum" and names[-2].endswith("_proj")
        assert names.count("pool_stride") == ell and names.count("pool_frag") == 3 - ell
        g = plan.geometry(120, 130, ell)
        assert sum(r["flops"] for r in recs) == pytest.approx(g["conv_flops"], rel=1e-9)
