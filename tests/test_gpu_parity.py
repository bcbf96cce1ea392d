"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Bit-exact for permutations and integer-valued data;
binary32 within 1e-4 * max|oracle|, bfloat16 within 2e-2 * max|oracle|."""
import os

import numpy as np
import pytest

import oracle
from oracle import fragment as fr
from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import (assert_close, check_bf16_storage_model, gpu_dense, kstar, log, oracle_layers,
                               oracle_windows, to_device)
from tests.test_oracle import HAND, _layers_from_json, chain_layers

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2
BF16_STORAGE_TOL = 1e-2   # against the bfloat16 storage model (see test_gpu_tiles)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dss.lib()
    yield
    torch.cuda.synchronize()


@pytest.fixture
def direct_conv(monkeypatch):
    """Plans created inside the test use the VALU convolution for every layer."""
    monkeypatch.setenv("DSS_CONV_KERNEL", "direct")


def chain_ends(layers):
    """Number of layer descriptors consumed after each processing-chain layer."""
    ends, t = [], 0
    while t < len(layers):
        t += 1
        if layers[t - 1]["kind"] == "conv" and t < len(layers) and layers[t]["kind"] == "maxpool":
            t += 1
        ends.append(t)
    return ends


# ----------------------------------------------------------------------------- Frag / Defrag


@pytest.mark.parametrize("kh,kw,Sh,Sw,C,H,W", [(2, 2, 1, 1, 3, 8, 10), (2, 3, 2, 1, 5, 6, 9), (1, 2, 1, 4, 1, 1, 16),
                                               (3, 2, 2, 2, 2, 9, 4), (4, 4, 2, 2, 7, 12, 20), (2, 2, 4, 4, 64, 34, 66)])
@pytest.mark.parametrize("elem", [4, 2])
def test_frag_defrag_bit_exact(kh, kw, Sh, Sw, C, H, W, elem):
    import torch
    log("frag/defrag k=%dx%d S=%dx%d C=%d H=%d W=%d elem=%d" % (kh, kw, Sh, Sw, C, H, W, elem))
    rng = np.random.default_rng(kh * 7 + kw + Sh + C)
    npdt, tdt = (np.int32, torch.int32) if elem == 4 else (np.int16, torch.int16)
    info = np.iinfo(npdt)
    x = rng.integers(info.min, info.max, size=(Sh * Sw, C, H, W), dtype=npdt)
    xd = torch.from_numpy(x).cuda()
    y = dss.frag(xd, kh, kw, Sh, Sw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), fr.frag_tensor(x, kh, kw, Sh, Sw))
    z = dss.defrag(y, kh, kw, Sh, Sw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(z.cpu().numpy(), x)
    np.testing.assert_array_equal(z.cpu().numpy(), fr.defrag_tensor(fr.frag_tensor(x, kh, kw, Sh, Sw), kh, kw, Sh, Sw))


def test_frag_rejects_bad_shape():
    import torch
    x = torch.zeros((1, 1, 5, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(dss.DssError) as e:
        dss.frag(x, 2, 2, 1, 1)
    assert e.value.status == 2


# ----------------------------------------------------------------------------- hand-derived cases


@pytest.mark.parametrize("case", HAND, ids=[c["name"] for c in HAND])
def test_hand_chain_gpu(case):
    layers = _layers_from_json(case["layers"])
    x = np.array(case["x"], dtype=np.float32)
    nd = 1 if x.shape[1] == 1 and all(l.get("fh", 1) == 1 and l.get("kh", 1) == 1 for l in layers) else 2
    out, plan = gpu_dense(layers, x, nd)
    g = plan.geometry(x.shape[1], x.shape[2])
    assert [g["B_h"], g["B_w"]] == case["B"] and [g["K_h"], g["K_w"]] == case["K"]
    assert [g["r_h"], g["r_w"]] == case["r"]
    np.testing.assert_array_equal(out, np.array(case["expected"], dtype=np.float64))


# ----------------------------------------------------------------------------- exact integer arithmetic

EXACT_ARCH = [("conv", 16, 32, 3, 3, "relu"), ("pool", 2, 2), ("conv", 32, 48, 3, 2, "relu"), ("pool", 2, 2),
              ("conv", 48, 136, 2, 3, "relu"), ("conv", 136, 3, 1, 1, "none")]


@pytest.mark.parametrize("kernel", ["mfma", "direct"])
def test_exact_integer_chain_bit_identical(kernel, monkeypatch):
    """Integer inputs, weights in {-1,0,1}, integer biases: every partial sum is an
    exactly representable integer, so any summation order must reproduce the
    oracle bit for bit.  Pins Stuff, Frag, Defrag, Trim and the output placement."""
    if kernel == "direct":
        monkeypatch.setenv("DSS_CONV_KERNEL", "direct")
    w = wl.custom(EXACT_ARCH, 16, 41, 47, seed=3, weight_kind="int", value_kind="int")
    log("exact chain %s on %s" % (kernel, w.x.shape))
    out, plan = gpu_dense(w.layers, w.x, 2)
    ref = oracle.eval_stride(w.layers, w.x)
    assert np.abs(ref).max() < 2 ** 23
    np.testing.assert_array_equal(out, ref)


def test_exact_integer_bf16_conv_bit_identical():
    """bfloat16 MFMA path on integer data: one conv layer whose binary32 output is exact."""
    arch = [("conv", 32, 48, 3, 3, "none")]
    w = wl.custom(arch, 32, 19, 70, seed=5, weight_kind="int", value_kind="int", dtype="bf16")
    out, _ = gpu_dense(w.layers, w.x, 2, "bf16")
    ref = oracle.eval_stride(w.layers, w.x)
    np.testing.assert_array_equal(out, ref)


# ----------------------------------------------------------------------------- random chains

CHAINS = {
    "2d_small_direct": ([("conv", 3, 5, 3, 2, "relu"), ("pool", 2, 1), ("conv", 5, 6, 2, 3, "tanh"), ("pool", 1, 2),
                         ("conv", 6, 2, 2, 2, "none")], 3, 2),
    "2d_mfma_mixed": ([("conv", 3, 16, 5, 5, "relu"), ("pool", 2, 2), ("conv", 16, 40, 3, 3, "relu"), ("pool", 2, 2),
                       ("conv", 40, 72, 3, 3, "tanh"), ("pool", 2, 2), ("conv", 72, 130, 4, 4, "relu"),
                       ("conv", 130, 2, 1, 1, "none")], 3, 2),
    "2d_pool_first": ([("pool", 2, 2), ("conv", 2, 20, 2, 2, "relu"), ("pool", 3, 3), ("conv", 20, 32, 2, 2, "relu"),
                       ("conv", 32, 1, 1, 1, "none")], 2, 2),
    "2d_pool_pool": ([("conv", 4, 24, 3, 3, "relu"), ("pool", 2, 2), ("pool", 2, 2), ("conv", 24, 20, 3, 3, "relu"),
                      ("conv", 20, 4, 1, 1, "none")], 4, 2),
    "1d_c2_like": ([("conv", 1, 16, 1, 9, "relu"), ("pool", 1, 2), ("conv", 16, 32, 1, 9, "relu"), ("pool", 1, 2),
                    ("conv", 32, 64, 1, 9, "relu"), ("pool", 1, 2), ("conv", 64, 2, 1, 8, "none")], 1, 1),
    "2d_ragged_cin": ([("conv", 20, 36, 3, 3, "relu"), ("pool", 2, 2), ("conv", 36, 20, 2, 2, "none")], 20, 2),
    # last layer on the lane-sum kernel (64 input channels, 3 outputs in two launch
    # columns, a 3 x 2 filter): taps k*_2 = 4 apart in the dilated fashion
    "2d_lanesum_last": ([("conv", 3, 16, 3, 3, "relu"), ("pool", 2, 2), ("conv", 16, 64, 2, 2, "relu"), ("pool", 2, 2),
                         ("conv", 64, 3, 3, 2, "none")], 3, 2),
}


@pytest.mark.parametrize("name", list(CHAINS))
def test_random_chain_f32(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    K = kstar(arch)
    H = 1 if nd == 1 else B[0] + 3 * K[0] + 1
    W = B[1] + 5 * K[1] + 3 if nd == 1 else B[1] + 4 * K[1] + 2
    if nd == 1:
        W = B[1] + 300
    w = wl.custom(arch, C, H, W, seed=2, value_kind="normal")
    log("chain %s on %s, B=%s" % (name, w.x.shape, B))
    out, _ = gpu_dense(w.layers, w.x, nd)
    ref = oracle.eval_stride(w.layers, w.x)
    assert_close(out, ref, F32_TOL, name)


@pytest.mark.parametrize("name", ["2d_mfma_mixed", "2d_pool_pool", "2d_ragged_cin"])
def test_random_chain_bf16(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    K = kstar(arch)
    w = wl.custom(arch, C, B[0] + 2 * K[0] + 1, B[1] + 3 * K[1] + 2, seed=4, dtype="bf16")
    log("bf16 chain %s on %s" % (name, w.x.shape))
    plan = dss.Plan(w.layers, nd, w.x.shape[0], "bf16")
    plan.set_timing(True)
    out, _ = gpu_dense(w.layers, w.x, nd, "bf16", plan=plan)
    L = oracle_layers(w.layers, "bf16")
    ref = oracle.eval_stride(L, w.x)
    assert_close(out, ref, BF16_TOL, name)
    check_bf16_storage_model(out, L, w.x, plan.timings(), BF16_STORAGE_TOL, name)


# The MFMA kernel runs its steps (input-channel chunk x filter tap) in threes
# over rotating weight-operand registers, with a chunk change inside the
# rotation: step counts of every residue mod 3, one to three chunks (16 binary32
# or 32 bfloat16 channels each), the single-buffered halo of a 7x7 filter, and
# small pooled fragments (flat tiles).
STEP_CASES = [(cin, f, pool) for cin in (1, 2, 3) for f in (1, 2, 5, 7) for pool in (False,)] + \
             [(2, 6, False), (2, 3, True), (3, 5, True), (1, 1, True)]


@pytest.mark.parametrize("chunks,f,pool", STEP_CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mfma_step_rotation(dtype, chunks, f, pool):
    # input channels in `chunks` chunks, the last one ragged where the MFMA kernel's
    # 16-byte staging allows it (at least 16 channels, multiples of 4 / 8)
    cin = {"f32": {1: 16, 2: 28, 3: 44}, "bf16": {1: 24, 2: 56, 3: 88}}[dtype][chunks]
    arch = ([("pool", 2, 2)] if pool else []) + [("conv", cin, 136, f, f, "relu")]
    H, W = (2 * f + 23, 2 * f + 37) if pool else (f + 29, f + 70)
    w = wl.custom(arch, cin, H, W, seed=cin + f, dtype=dtype)
    log("%s conv %dx%d cin=%d pool=%s on %s" % (dtype, f, f, cin, pool, w.x.shape))
    out, _ = gpu_dense(w.layers, w.x, 2, dtype)
    ref = oracle.eval_stride(oracle_layers(w.layers, dtype), w.x)
    assert_close(out, ref, BF16_TOL if dtype == "bf16" else F32_TOL, "%s %dx%d cin=%d" % (dtype, f, f, cin))


def test_direct_and_mfma_agree(direct_conv):
    """Both convolution kernels on the same chain agree to rounding."""
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    w = wl.custom(arch, C, 60, 57, seed=7)
    d, _ = gpu_dense(w.layers, w.x, nd)
    os.environ.pop("DSS_CONV_KERNEL")
    m, _ = gpu_dense(w.layers, w.x, nd)
    assert_close(m, d, 1e-5, "mfma vs direct")


# ----------------------------------------------------------------------------- geometry edge cases


def test_every_stuffing_amount_gpu():
    arch = [("conv", 2, 16, 3, 3, "relu"), ("pool", 2, 2), ("conv", 16, 16, 2, 2, "relu"), ("pool", 3, 3),
            ("conv", 16, 2, 2, 2, "none")]
    w0 = wl.custom(arch, 2, 1, 1, seed=0)
    B = oracle.receptive_field(w0.layers)
    plan = dss.Plan(w0.layers, 2, 2)
    seen = set()
    for n in range(B[0], B[0] + 7):
        w = wl.custom(arch, 2, n, B[1] + 6 - (n - B[0]), seed=n)
        w.layers = w0.layers
        out, _ = gpu_dense(w.layers, w.x, 2, plan=plan)
        ref = oracle.eval_stride(w.layers, w.x)
        assert_close(out, ref, F32_TOL, "n=%d" % n)
        seen.add(plan.geometry(n, w.x.shape[2])["r_h"])
    assert seen == set(range(6))


def test_signal_equal_to_receptive_field():
    w = wl.make("c1_64x64", H=28, W=28)
    out, _ = gpu_dense(w.layers, w.x, 2)
    assert out.shape == (1, 1, 1)
    assert_close(out, oracle.eval_stride(w.layers, w.x), F32_TOL)


def test_eval_slide_lemma_d():
    """Per-layer check of Lemma 'processing chain' (d): the strided network's
    layer-j output on window (i, w) sits in fragment (i mod k*_h) k*_w + (w mod k*_w)
    of the sliding evaluation, at offset (i div k*_h, w div k*_w)."""
    import torch
    arch = [("conv", 3, 16, 3, 3, "relu"), ("pool", 2, 2), ("conv", 16, 24, 2, 3, "relu"), ("pool", 2, 3),
            ("conv", 24, 20, 3, 2, "relu"), ("conv", 20, 2, 1, 1, "none")]
    w = wl.custom(arch, 3, 40, 45, seed=9)
    plan = dss.Plan(w.layers, 2, 3)
    B = plan.geometry(40, 45)
    ch = chain_layers(w.layers)
    xd = to_device(w.x, "f32")
    ends = chain_ends(w.layers)
    rng = np.random.default_rng(0)
    for j in range(1, len(ch) + 1):
        lg = plan.layer_geometry(40, 45, j)
        slide = plan.eval_slide(xd, j)
        torch.cuda.synchronize()
        slide = slide.cpu().numpy().astype(np.float64)
        wi = rng.integers(0, B["out_h"], size=12)
        wj = rng.integers(0, B["out_w"], size=12)
        ref = oracle.eval_stride(w.layers, w.x, windows=(wi, wj), upto=ends[j - 1])
        C, uh, uw = lg["channels"], lg["u_h"], lg["u_w"]
        ref = ref.reshape(len(wi), C, uh, uw)
        for q in range(len(wi)):
            f = (wi[q] % lg["kstar_h"]) * lg["kstar_w"] + (wj[q] % lg["kstar_w"])
            y0, x0 = wi[q] // lg["kstar_h"], wj[q] // lg["kstar_w"]
            got = slide[f, :, y0:y0 + uh, x0:x0 + uw]
            assert_close(got, ref[q], F32_TOL, "layer %d window (%d,%d)" % (j, wi[q], wj[q]))


def test_translation_equivariance_gpu():
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    w = wl.custom(arch, C, 90, 85, seed=12)
    full, plan = gpu_dense(w.layers, w.x, 2)
    g = plan.geometry(90, 85)
    a, b, h, ww = 5, 3, g["B_h"] + 9, g["B_w"] + 11
    crop, _ = gpu_dense(w.layers, np.ascontiguousarray(w.x[:, a:a + h, b:b + ww]), 2, plan=plan)
    assert_close(crop, full[:, a:a + h - g["B_h"] + 1, b:b + ww - g["B_w"] + 1], 1e-6, "crop")


# ----------------------------------------------------------------------------- named workloads


def test_c1_full_dense():
    w = wl.make("c1_64x64")
    out, plan = gpu_dense(w.layers, w.x, 2)
    assert out.shape == (1, 37, 37)
    assert_close(out, oracle.eval_stride(w.layers, w.x), F32_TOL, "c1")


@pytest.mark.parametrize("name,H,W,widths", [("c2_1d_1m", 1, 20000, None), ("c3_512", 100, 118, (16, 32, 48, 64)),
                                             ("c4_hd", 90, 97, (16, 32, 64, 128)),
                                             ("c5_4k", 170, 181, (16, 16, 32, 32))])
def test_named_reduced_full_oracle(name, H, W, widths):
    """The named layer patterns at reduced extents and widths, every window checked."""
    w = wl.make(name, H=H, W=W, widths=widths)
    log("%s reduced %s widths=%s" % (name, w.x.shape, widths))
    plan = dss.Plan.from_workload(w)
    plan.set_timing(True)
    out, _ = gpu_dense(w.layers, w.x, w.ndim, w.dtype, plan=plan)
    L = oracle_layers(w.layers, w.dtype)
    ref = oracle.eval_stride(L, w.x)
    assert_close(out, ref, BF16_TOL if w.dtype == "bf16" else F32_TOL, name)
    if w.dtype == "bf16":
        check_bf16_storage_model(out, L, w.x, plan.timings(), BF16_STORAGE_TOL, name)


# Full-size workloads in the benchmark's launch configuration.  The dense
# evaluation of each runs once per session; the oracle then checks every window
# of the 1-D workload, and on the 2-D frames 8 seeded windows of every fragment
# phase pair (i mod K, j mod K) plus the corners and edge midpoints, and on the
# 512x512 and HD frames every window of the last K rows and the last K columns
# (the outputs whose fragments end next to the stuffed samples and in the
# masked edge tiles).  The theorem (Sect. 4.3) makes the equality hold at every
# window and phase.
_FULL = {}


def full_size(name):
    """(workload, geometry, GPU dense output as float64) of a named workload."""
    if name not in _FULL:
        import torch
        w = wl.make(name)
        log("%s full size %s" % (name, w.x.shape))
        plan = dss.Plan.from_workload(w)
        out = plan.eval_dense(to_device(w.x, w.dtype))
        torch.cuda.synchronize()
        g = plan.geometry(w.x.shape[1], w.x.shape[2])
        plan.close()
        got = out.cpu().numpy().astype(np.float64)
        del out
        torch.cuda.empty_cache()
        assert got.shape == (g["out_c"], g["out_h"], g["out_w"])
        assert np.all(np.isfinite(got))
        _FULL[name] = (w, g, got)
    return _FULL[name]


def _check_windows(name, i, j, what):
    w, g, got = full_size(name)
    log("  %s: checking %d windows (%s)" % (name, len(i), what))
    ref = oracle_windows(oracle_layers(w.layers, w.dtype), w.x, i, j)
    assert_close(got[:, i, j].T, ref, BF16_TOL if w.dtype == "bf16" else F32_TOL, "%s %s" % (name, what))


def test_c2_full_frame_every_window():
    w, g, got = full_size("c2_1d_1m")
    log("  c2_1d_1m: oracle on all %d windows" % (g["out_h"] * g["out_w"]))
    ref = oracle.eval_stride(w.layers, w.x)
    assert_close(got, ref, F32_TOL, "c2 every window")


@pytest.mark.parametrize("name", ["c3_512", "c4_hd"])
def test_full_size_every_phase(name):
    _, g, _ = full_size(name)
    i, j = wl.sample_windows(g["out_h"], g["out_w"], g["K_h"], g["K_w"], per_phase=8, seed=0)
    assert len(set(zip((i % g["K_h"]).tolist(), (j % g["K_w"]).tolist()))) == g["K_h"] * g["K_w"]
    _check_windows(name, i, j, "8 per phase")


def _edge_windows(g, part, parts):
    """Every window of the last K_h rows and the last K_w columns, split into
    `parts` column ranges of the rows plus the columns block as the last part."""
    K_h, K_w, oh, ow = g["K_h"], g["K_w"], g["out_h"], g["out_w"]
    if part < parts:
        c0, c1 = ow * part // parts, ow * (part + 1) // parts
        ii, jj = np.meshgrid(np.arange(oh - K_h, oh), np.arange(c0, c1), indexing="ij")
    else:
        ii, jj = np.meshgrid(np.arange(0, oh - K_h), np.arange(ow - K_w, ow), indexing="ij")
    return ii.reshape(-1).astype(np.int64), jj.reshape(-1).astype(np.int64)


@pytest.mark.parametrize("name,part,parts", [("c3_512", 0, 1), ("c3_512", 1, 1), ("c4_hd", 0, 3), ("c4_hd", 1, 3),
                                             ("c4_hd", 2, 3), ("c4_hd", 3, 3)])
def test_full_size_last_rows_and_columns(name, part, parts):
    _, g, _ = full_size(name)
    i, j = _edge_windows(g, part, parts)
    _check_windows(name, i, j, "edge part %d of %d" % (part, parts + 1))


@pytest.mark.parametrize("half", [0, 1])
def test_c5_full_size_every_phase(half):
    """The 4K bfloat16 frame: 8 windows for each of the 256 phase pairs (split
    over two tests by row phase) plus corners and edge midpoints."""
    _, g, _ = full_size("c5_4k")
    i, j = wl.sample_windows(g["out_h"], g["out_w"], g["K_h"], g["K_w"], per_phase=8, seed=0)
    assert len(set(zip((i % g["K_h"]).tolist(), (j % g["K_w"]).tolist()))) == g["K_h"] * g["K_w"]
    keep = (i % g["K_h"]) // (g["K_h"] // 2) == half
    _check_windows("c5_4k", i[keep], j[keep], "8 per phase, row phases %s" % ("0-7", "8-15")[half])


# ----------------------------------------------------------------------------- robustness


def test_errors_leave_output_untouched():
    import torch
    w = wl.make("c1_64x64")
    plan = dss.Plan.from_workload(w)
    out = torch.full((1, 37, 37), 123.0, device="cuda")
    small = to_device(w.x[:, :27, :], "f32")
    with pytest.raises(dss.DssError) as e:
        plan.eval_dense(small, out=torch.empty((1, 1, 1), device="cuda"))
    assert e.value.status == 2
    ws = torch.empty(16 * 1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(dss.DssError) as e:
        plan.eval_dense(to_device(w.x, "f32"), out=out, workspace=ws)
    assert e.value.status == 2
    torch.cuda.synchronize()
    assert torch.all(out == 123.0)


def test_run_twice_bit_identical():
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    w = wl.custom(arch, C, 70, 66, seed=13)
    a, plan = gpu_dense(w.layers, w.x, nd)
    b, _ = gpu_dense(w.layers, w.x, nd, plan=plan)
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_concurrent_evaluations_one_plan(dtype):
    """Two host threads evaluate one plan at the same time, each on its own
    stream with its own workspace (the concurrency the C ABI allows when timing
    is off): every result equals the serial evaluation bit for bit."""
    import threading
    import torch
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    H, W = 90, 84
    sig = [wl.custom(arch, C, H, W, seed=s) for s in (21, 22)]
    plan = dss.Plan(sig[0].layers, nd, C, dtype)
    xs = [to_device(w.x, dtype) for w in sig]
    serial = [plan.eval_dense(x) for x in xs]
    torch.cuda.synchronize()
    serial = [s.cpu() for s in serial]
    need = plan.geometry(H, W)["workspace_bytes"]
    spaces = [torch.empty(need, dtype=torch.uint8, device="cuda") for _ in xs]
    outs = [torch.empty(s.shape, dtype=torch.float32, device="cuda") for s in serial]
    streams = [torch.cuda.Stream() for _ in xs]
    torch.cuda.synchronize()
    errors = []

    def run(i):
        try:
            for _ in range(4):
                plan.eval_dense(xs[i], out=outs[i], workspace=spaces[i], stream=streams[i])
            streams[i].synchronize()
        except Exception as e:   # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=run, args=(i,)) for i in range(len(xs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
    torch.cuda.synchronize()
    for i in range(len(xs)):
        assert torch.equal(outs[i].cpu(), serial[i]), i


@pytest.mark.parametrize("fold", [True, False])
def test_timing_records(fold, monkeypatch):
    if not fold:
        monkeypatch.setenv("DSS_FUSE_PROJECTION", "0")
    w = wl.make("c3_512", H=120, W=130, widths=(16, 32, 64, 128))
    plan = dss.Plan.from_workload(w)
    plan.set_timing(True)
    gpu_dense(w.layers, w.x, 2, plan=plan)
    recs = plan.timings()
    names = [r["kernel"] for r in recs]
    assert names[0] == "stuff_pack"
    assert "conv_mfma_f32_n64" in names and "conv_mfma_f32_n32" in names and "pool_frag" in names
    if fold:
        # the final 1x1 projection folded into the conv6x6 epilogue (the 128-channel
        # layer runs the 64-channel tile here: at this size the 128-channel tile
        # would give too few workgroups to fill the GPU)
        assert names[-2:] == ["conv_mfma_f32_n64_proj", "defrag_sum"]
    else:
        # the final 1x1 projection 128 -> 2 runs the
        # lane-sum form of the direct kernel
        assert names[-2:] == ["conv_lanesum", "defrag_trim"]
    g = plan.geometry(120, 130)
    assert sum(r["flops"] for r in recs) == pytest.approx(g["conv_flops"], rel=1e-9)
    assert all(r["ms"] >= 0 for r in recs)
