"""GPU parity of the convolution kernel's launch variants, every window checked
against the oracle: the 128-channel N tile (taken only by launches of at least
512 workgroups) with ragged channel chunks and masked edge tiles, and a seeded
sweep of small random chains whose sizes straddle the choices between the
64- and 128-channel tiles and between spatial and flat tiles.  The launch
records name the kernel and tile mode each layer actually ran."""
import numpy as np
import pytest

import oracle
import oracle.bf16
from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import assert_close, check_bf16_storage_model, gpu_dense, log, oracle_layers

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2
# against the oracle's bfloat16 storage model: the GPU rounds at the same places,
# so only single rounding-boundary flips (binary32 sums in another order) remain;
# 4.6e-3 at worst over 80 random bfloat16 chains
BF16_STORAGE_TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dss.lib()
    yield
    torch.cuda.synchronize()


def timed_dense(w):
    """Dense evaluation with launch records: (float64 output, records)."""
    plan = dss.Plan.from_workload(w)
    plan.set_timing(True)
    out, _ = gpu_dense(w.layers, w.x, w.ndim, w.dtype, plan=plan)
    recs = plan.timings()
    plan.close()
    return out, recs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_n128_tile_every_window(dtype):
    """Two convolutions with 136 and 130 output channels (two N blocks of 128,
    the second almost all padding) and 44 / 88 input channels (2.75 chunks: the
    last one ragged), on extents that leave partial edge tiles.  Both launches
    have more than 512 workgroups, so both run the 128-channel tile; the second
    also computes the final 1x1 projection in its epilogue."""
    cin = 44 if dtype == "f32" else 88
    arch = [("conv", cin, 136, 3, 3, "relu"), ("pool", 2, 2), ("conv", 136, 130, 2, 2, "relu"),
            ("conv", 130, 3, 1, 1, "none")]
    w = wl.custom(arch, cin, 260, 291, seed=17, dtype=dtype)
    log("n128 %s on %s" % (dtype, w.x.shape))
    out, recs = timed_dense(w)
    names = [r["kernel"] for r in recs if r["flops"] > 0]
    log("  launches: %s" % names)
    # the second carries the folded 1x1 projection
    assert names == ["conv_mfma_%s_n128" % dtype, "conv_mfma_%s_n128_proj" % dtype]
    assert all(r["tile_mode"] == 0 for r in recs if "n128" in r["kernel"])
    ref = oracle.eval_stride(oracle_layers(w.layers, dtype), w.x)
    assert_close(out, ref, BF16_TOL if dtype == "bf16" else F32_TOL, "n128 %s" % dtype)


# Output extents whose least-masked spatial tile is 16 x 16 (48 x 80: 8-wide tiles
# would pad 48 rows to 64, 32-wide ones 80 columns to 96) or 32 x 8 (96 x 40: 16-wide
# tiles would pad 40 columns to 48), and filter widths giving every row distance
# of the interleaved order: halo rows HW = TW + fw - 1 samples long, rows d apart
# with d = 8 >> tz(HW) (8-wide) or 16 >> tz(HW) (16-wide, HW even), else d = 1.
NARROW_TILE_CASES = [(16, 2), (16, 3), (16, 5), (16, 9), (8, 2), (8, 3), (8, 5), (8, 6), (8, 9)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("tw,fw", NARROW_TILE_CASES, ids=["tw%d_fw%d" % c for c in NARROW_TILE_CASES])
def test_narrow_tile_row_order_every_window(tw, fw, dtype):
    """An fw x fw convolution 32 -> 64 on extents that make 8- or 16-wide tiles
    the least-masked shape, whose samples the kernel takes from rows d apart
    (the LDS bank-conflict-free order), then a 1x1 convolution 64 -> 16, checked
    at every output position.  The first launch stores its activations through
    the store epilogue (bfloat16 or binary32), which maps the samples back by
    the same order; a row order that is not a bijection of the tile, or an
    epilogue that maps differently, shows up as wrong or missing outputs."""
    hout, wout = (48, 80) if tw == 16 else (96, 40)
    arch = [("conv", 32, 64, fw, fw, "relu"), ("conv", 64, 16, 1, 1, "none")]
    w = wl.custom(arch, 32, hout + fw - 1, wout + fw - 1, seed=100 + 10 * tw + fw, dtype=dtype)
    log("narrow tile %s tw=%d fw=%d on %s" % (dtype, tw, fw, w.x.shape))
    out, recs = timed_dense(w)
    names = [r["kernel"] for r in recs if r["flops"] > 0]
    log("  launches: %s" % names)
    assert names[0] == "conv_mfma_%s_n64" % dtype, names
    assert all(r["tile_mode"] == 0 for r in recs if r["kernel"].startswith("conv_mfma"))
    layers = oracle_layers(w.layers, dtype)
    ref = oracle.eval_stride(layers, w.x)
    assert out.shape == ref.shape == (16, hout, wout)
    if dtype == "bf16":
        check_bf16_storage_model(out, layers, w.x, recs, BF16_STORAGE_TOL, "narrow tile tw=%d fw=%d" % (tw, fw))
    assert_close(out, ref, BF16_TOL if dtype == "bf16" else F32_TOL, "narrow tile %s tw=%d fw=%d" % (dtype, tw, fw))


def _random_chain(seed):
    """A small random chain and signal size.  Even seeds: one wide layer (132 to
    256 binary32 / 512 bfloat16 output channels) on signals of 150-330 samples
    per axis, so that its launch lands on both sides of the 512-workgroup line
    of the 128-channel tile.  Odd seeds: two or three conv + pool layers on
    30-110 samples, whose pooled fragments take flat or spatial tiles."""
    rng = np.random.default_rng(5000 + seed)
    dtype = "bf16" if seed % 3 == 2 else "f32"
    q = 8 if dtype == "bf16" else 4
    if seed % 2 == 0:
        C0 = int(rng.choice([16, 24, 32]))
        cout = q * int(rng.integers(33, 65))
        f = int(rng.integers(1, 3))
        k = int(rng.integers(1, 3))
        arch = [("conv", C0, cout, f, f, "relu")] + ([("pool", k, k)] if k > 1 else []) + \
               [("conv", cout, int(rng.choice([2, 3])), 1, 1, "none")]
        side = int(rng.integers(150, 330))
    else:
        C0 = int(rng.choice([3, 16, 24]))
        arch, c = [], C0
        for _ in range(int(rng.integers(2, 4))):
            cout = q * int(rng.integers(4, 17))
            f = int(rng.integers(2, 4))
            arch += [("conv", c, cout, f, f, str(rng.choice(["relu", "tanh"]))), ("pool", 2, 2)]
            c = cout
        arch.append(("conv", c, int(rng.choice([1, 2, 3])), int(rng.integers(1, 4)), int(rng.integers(1, 4)),
                     "none"))
        side = int(rng.integers(30, 110))
    B = oracle.receptive_field(wl.custom(arch, C0, 1, 1, seed=0).layers)
    H = max(side + int(rng.integers(0, 9)), B[0] + int(rng.integers(2, 12)))
    W = max(side + int(rng.integers(0, 9)), B[1] + int(rng.integers(2, 12)))
    return arch, C0, H, W, dtype


SWEEP = list(range(30))


@pytest.fixture(scope="module")
def sweep_log():
    seen = []
    yield seen
    # the sweep as a whole must reach each variant (checked at module teardown
    # only when every sweep case ran)
    if len(seen) == len(SWEEP):
        kinds = {k for case in seen for k in case}
        log("sweep variants: %s" % sorted(kinds))
        for need in ("n64", "n128", "flat", "spatial"):
            assert any(need in k for k in kinds), "no sweep case ran the %s variant" % need


@pytest.mark.parametrize("seed", SWEEP)
def test_random_chain_sweep(seed, sweep_log):
    arch, C0, H, W, dtype = _random_chain(seed)
    w = wl.custom(arch, C0, H, W, seed=seed, dtype=dtype)
    out, recs = timed_dense(w)
    kinds = set()
    for r in recs:
        if r["tile_mode"] >= 0:
            kinds.add([t for t in r["kernel"].split("_") if t in ("n32", "n64", "n128")][0])
            kinds.add(("spatial", "flat", "dilated")[r["tile_mode"]])
    log("sweep %d: %s %s on %dx%d, variants %s" % (seed, dtype, arch, H, W, sorted(kinds)))
    sweep_log.append(kinds)
    L = oracle_layers(w.layers, dtype)
    ref = oracle.eval_stride(L, w.x)
    assert_close(out, ref, BF16_TOL if dtype == "bf16" else F32_TOL, "sweep %d" % seed)
    if dtype == "bf16":
        # tighter: against the exact evaluation with bfloat16-stored activations
        # (kept in binary32 before a folded projection, as the launch records show)
        fold = any(r["kernel"].endswith("_proj") for r in recs)
        emu = oracle.bf16.eval_dilate_bf16_storage(L, w.x, fold=fold)
        assert_close(out, emu, BF16_STORAGE_TOL, "sweep %d vs bfloat16 storage model" % seed)


FOLD_CASES = {
    # (arch, channels, H, W, dtype, value kind)
    "f32_n64": ([("conv", 3, 16, 5, 5, "relu"), ("pool", 2, 2), ("conv", 16, 40, 3, 3, "relu"), ("pool", 2, 2),
                 ("conv", 40, 72, 3, 3, "tanh"), ("pool", 2, 2), ("conv", 72, 130, 4, 4, "relu"),
                 ("conv", 130, 2, 1, 1, "none")], 3, 93, 101, "f32", "uniform"),
    "f32_n32_act": ([("conv", 16, 20, 3, 3, "relu"), ("pool", 2, 2), ("conv", 20, 24, 2, 2, "tanh"),
                     ("conv", 24, 3, 1, 1, "tanh")], 16, 77, 70, "f32", "normal"),
    "bf16_n128": ([("conv", 32, 256, 2, 2, "relu"), ("conv", 256, 4, 1, 1, "none")], 32, 300, 310, "bf16", "uniform"),
    "int_f32": ([("conv", 16, 32, 3, 3, "relu"), ("pool", 2, 2), ("conv", 32, 48, 3, 2, "relu"), ("pool", 2, 2),
                 ("conv", 48, 136, 2, 3, "relu"), ("conv", 136, 3, 1, 1, "none")], 16, 41, 47, "f32", "int"),
    # 32 taps of |x| <= 8 with weights in {-1, 0, 1}: the stored bfloat16 activations stay
    # integers of at most 256, which bfloat16 holds exactly
    "int_bf16_n128": ([("conv", 16, 200, 1, 2, "relu"), ("conv", 200, 2, 1, 1, "relu")], 16, 290, 285, "bf16", "int"),
    # the bfloat16 launch with a folded projection computes transposed blocks; its
    # 64- and 32-channel tiles (NT = 2 and 1), ragged channel groups (96 of 128,
    # 40 of 64) and tanh on both sides of the fold
    "bf16_n64_tanh": ([("conv", 16, 96, 3, 3, "tanh"), ("conv", 96, 3, 1, 1, "tanh")], 16, 83, 95, "bf16", "uniform"),
    "bf16_n32": ([("conv", 24, 40, 2, 3, "relu"), ("conv", 40, 2, 1, 1, "none")], 24, 70, 66, "bf16", "normal"),
    "int_bf16_n64": ([("conv", 16, 100, 2, 1, "relu"), ("conv", 100, 4, 1, 1, "none")], 16, 120, 131, "bf16", "int"),
}


FOLD_KERNEL = {"bf16_n64_tanh": "conv_mfma_bf16_n64_proj", "bf16_n32": "conv_mfma_bf16_n32_proj",
               "int_bf16_n64": "conv_mfma_bf16_n64_proj"}


@pytest.mark.parametrize("case", list(FOLD_CASES))
def test_projection_fold(case, monkeypatch):
    """The final 1x1 projection folded into the previous convolution's epilogue
    (partial dot products per group of 64 channels, or 32 with the 32-channel
    N tile, summed in group order by the final defragmentation) against the
    unfused evaluation and the oracle; integer data bit-exact both ways."""
    arch, C, H, W, dtype, kind = FOLD_CASES[case]
    w = wl.custom(arch, C, H, W, seed=31, dtype=dtype, value_kind=kind,
                  weight_kind="int" if kind == "int" else "he")
    fused, rf = timed_dense(w)
    monkeypatch.setenv("DSS_FUSE_PROJECTION", "0")
    plain, rp = timed_dense(w)
    names_f = [r["kernel"] for r in rf]
    names_p = [r["kernel"] for r in rp]
    log("fold %s: %s / %s" % (case, names_f[-2:], names_p[-2:]))
    assert names_f[-2].endswith("_proj") and names_f[-1] == "defrag_sum"
    if case in FOLD_KERNEL:
        assert names_f[-2] == FOLD_KERNEL[case], names_f
    assert not any(n.endswith("_proj") for n in names_p) and names_p[-1] == "defrag_trim"
    assert sum(r["flops"] for r in rf) == pytest.approx(sum(r["flops"] for r in rp), rel=1e-12)
    ref = oracle.eval_stride(oracle_layers(w.layers, dtype), w.x)
    if kind == "int":
        assert np.abs(ref).max() < 2 ** 23
        np.testing.assert_array_equal(fused, ref)
        np.testing.assert_array_equal(plain, ref)
        return
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    assert_close(fused, ref, tol, "fold %s fused" % case)
    assert_close(plain, ref, tol, "fold %s unfused" % case)
    if dtype == "f32":
        # same products, summed in another order
        assert_close(fused, plain, 1e-6, "fold %s fused vs unfused" % case)


POOL_CASES = {
    # (arch, channels, W, value kind, dtype): 1-D chains whose convolutions carry the pool
    "c2_pattern": ([("conv", 1, 16, 1, 9, "relu"), ("pool", 1, 2), ("conv", 16, 32, 1, 9, "relu"), ("pool", 1, 2),
                    ("conv", 32, 64, 1, 9, "relu"), ("pool", 1, 2), ("conv", 64, 2, 1, 8, "none")], 1, 20011, "normal",
                   "f32"),
    "k3_ragged": ([("conv", 16, 20, 1, 7, "tanh"), ("pool", 1, 3), ("conv", 20, 36, 1, 5, "relu"), ("pool", 1, 2),
                   ("conv", 36, 2, 1, 4, "none")], 16, 6007, "uniform", "f32"),
    "int_exact": ([("conv", 16, 24, 1, 3, "relu"), ("pool", 1, 2), ("conv", 24, 40, 1, 2, "relu"), ("pool", 1, 3),
                   ("conv", 40, 3, 1, 2, "none")], 16, 5003, "int", "f32"),
    # first layers on the direct kernel: 3 channels, tanh, k = 3; bfloat16 (the
    # MFMA convolutions of bfloat16 plans keep the separate pool)
    "direct_k3_tanh": ([("conv", 3, 8, 1, 4, "tanh"), ("pool", 1, 3), ("conv", 8, 2, 1, 3, "none")], 3, 4001, "normal",
                       "f32"),
    "direct_bf16": ([("conv", 1, 16, 1, 9, "relu"), ("pool", 1, 2), ("conv", 16, 32, 1, 5, "relu"), ("pool", 1, 2),
                     ("conv", 32, 2, 1, 4, "none")], 1, 8009, "uniform", "bf16"),
}


@pytest.mark.parametrize("case", list(POOL_CASES))
def test_pool_in_conv_epilogue_1d(case, monkeypatch):
    """One-row fragments: the sliding max-pool and Frag computed in the MFMA
    convolution's epilogue (tiles overlapping by k - 1 samples) or, for layers
    with few input channels, in the direct convolution kernel, against the
    separate pool + Frag kernel (bit-identical: maxima of the same values) and
    the oracle."""
    arch, C, W, kind, dtype = POOL_CASES[case]
    w = wl.custom(arch, C, 1, W, seed=41, ndim=1, dtype=dtype, value_kind=kind,
                  weight_kind="int" if kind == "int" else "he")
    fused, rf = timed_dense(w)
    monkeypatch.setenv("DSS_FUSE_POOL", "0")
    plain, rp = timed_dense(w)
    nf = [r["kernel"] for r in rf]
    npl = [r["kernel"] for r in rp]
    log("pool fusion %s: %s / %s" % (case, nf, npl))
    pairs = [arch[t] for t in range(len(arch) - 1) if arch[t][0] == "conv" and arch[t + 1][0] == "pool"]
    n_fused = sum(1 for c in pairs if c[1] < 16 or dtype == "f32")
    assert sum(n.endswith("_pool") for n in nf) == n_fused >= 1
    assert nf.count("conv_direct_pool") == sum(1 for c in pairs if c[1] < 16)
    assert not any(n.endswith("_pool") for n in npl)
    assert npl.count("pool_frag") - nf.count("pool_frag") == n_fused
    np.testing.assert_array_equal(fused, plain)
    ref = oracle.eval_stride(oracle_layers(w.layers, dtype), w.x)
    if kind == "int":
        np.testing.assert_array_equal(fused, ref)
    else:
        assert_close(fused, ref, BF16_TOL if dtype == "bf16" else F32_TOL, "pool fusion %s" % case)


LANESUM_CASES = {
    # (arch, channels, H, W, ndim, dtype, value kind): last layers with input
    # channels in multiples of 64 and at most 8 output channels per launch column
    "1d_fw8_cout2": ([("conv", 16, 64, 1, 3, "relu"), ("pool", 1, 2), ("conv", 64, 2, 1, 8, "none")], 16, 1, 3001,
                     1, "f32", "normal"),
    "1d_fw5_cout1_c192": ([("conv", 16, 192, 1, 2, "relu"), ("pool", 1, 3), ("conv", 192, 1, 1, 5, "tanh")], 16, 1,
                          2113, 1, "f32", "uniform"),
    "2d_3x3_cout3": ([("conv", 16, 64, 3, 3, "relu"), ("pool", 2, 2), ("conv", 64, 3, 3, 3, "none")], 16, 61, 75, 2,
                     "f32", "uniform"),
    "2d_2x7_cout8": ([("conv", 16, 128, 2, 2, "relu"), ("conv", 128, 8, 2, 7, "relu")], 16, 40, 77, 2, "f32",
                     "normal"),
    "2d_1x1_cout5_bf16": ([("conv", 16, 128, 3, 3, "relu"), ("pool", 2, 2), ("conv", 128, 5, 1, 1, "none")], 16, 57,
                          66, 2, "bf16", "uniform"),
    "2d_4x4_cout2_bf16": ([("conv", 32, 64, 2, 2, "relu"), ("pool", 2, 2), ("conv", 64, 64, 2, 2, "relu"),
                           ("conv", 64, 2, 4, 4, "none")], 32, 70, 53, 2, "bf16", "uniform"),
    # integer data and weights: every sum exact in binary32, so any summation order
    # gives the oracle's value bit for bit
    "int_2d_fw6": ([("conv", 16, 64, 2, 2, "relu"), ("pool", 2, 2), ("conv", 64, 4, 2, 6, "none")], 16, 50, 67, 2,
                   "f32", "int"),
}


@pytest.mark.parametrize("case", list(LANESUM_CASES))
def test_lanesum_last_layer(case, monkeypatch):
    """The lane-sum form of the direct kernel (lanes over input channels, a
    butterfly across the lanes at the end) on every window against the oracle,
    for 1 to 8 output channels per launch column, filters 1 to 8 wide, one and
    two dimensions, binary32 and bfloat16; the launch records name it for the
    last layer.  Binary32 plans take it for such layers by themselves; bfloat16
    plans run those on the MFMA tile, so their cases select the direct kernels
    for every layer."""
    monkeypatch.setenv("DSS_FUSE_PROJECTION", "0")
    arch, C, H, W, ndim, dtype, kind = LANESUM_CASES[case]
    if dtype == "bf16":
        monkeypatch.setenv("DSS_CONV_KERNEL", "direct")
    w = wl.custom(arch, C, H, W, seed=53, dtype=dtype, ndim=ndim, value_kind=kind,
                  weight_kind="int" if kind == "int" else "he")
    out, recs = timed_dense(w)
    names = [r["kernel"] for r in recs]
    log("lanesum %s: %s" % (case, names))
    assert names[-2] == "conv_lanesum"
    ref = oracle.eval_stride(oracle_layers(w.layers, dtype), w.x)
    if kind == "int":
        assert np.abs(ref).max() < 2 ** 23
        np.testing.assert_array_equal(out, ref)
        return
    assert_close(out, ref, BF16_TOL if dtype == "bf16" else F32_TOL, "lanesum %s" % case)
