"""GPU parity of the dilated fashion (dss_eval_dilate): every intermediate
EvalDilate_j against the oracle's literal dilated evaluation, the final layer
against the dense oracle and bit for bit against dss_eval_dense (the same
kernels evaluate the same taps in the same order; only the addressing differs)."""
import numpy as np
import pytest

import oracle
from oracle import dilate as odilate
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


def gpu_dilate(plan, x, j=None, dtype="f32"):
    import torch
    out = plan.eval_dilate(to_device(x, dtype), j)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def gpu_dense(plan, x, dtype="f32"):
    import torch
    out = plan.eval_dense(to_device(x, dtype))
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("name", list(CHAINS))
def test_dilate_every_layer(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    ch = mixed.chain_of(w0.layers)
    B = mixed.strided_extents(ch)[0]
    K = mixed.stride_products(ch)[-1]
    H = 1 if nd == 1 else B[0] + K[0] + 2
    W = B[1] + (200 if nd == 1 else 2 * K[1] + 1)
    w = wl.custom(arch, C, H, W, seed=7, value_kind="normal")
    plan = dss.Plan(w.layers, nd, C)
    for j in range(len(ch) + 1):
        log("dilate %s %dx%d j=%d" % (name, H, W, j))
        got = gpu_dilate(plan, w.x, j)
        ref = odilate.eval_dilate(w.layers, w.x, upto=j)
        if j == 0:
            np.testing.assert_array_equal(got, ref)
        else:
            assert_close(got, ref, F32_TOL, "%s j=%d" % (name, j))
    np.testing.assert_array_equal(got, gpu_dense(plan, w.x))
    assert_close(got, oracle.eval_stride(w.layers, w.x), F32_TOL, name + " vs EvalStride")


@pytest.mark.parametrize("kernel", ["mfma", "direct"])
def test_dilate_exact_integer_chain(kernel, monkeypatch):
    if kernel == "direct":
        monkeypatch.setenv("DSS_CONV_KERNEL", "direct")
    w = wl.custom(EXACT_ARCH, 16, 43, 52, seed=3, weight_kind="int", value_kind="int")
    plan = dss.Plan(w.layers, 2, 16)
    np.testing.assert_array_equal(gpu_dilate(plan, w.x), oracle.eval_stride(w.layers, w.x))


@pytest.mark.parametrize("name", ["2d_mfma_mixed", "2d_pool_pool"])
def test_dilate_bf16(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    w = wl.custom(arch, C, B[0] + 13, B[1] + 21, seed=4, dtype="bf16")
    plan = dss.Plan(w.layers, nd, C, "bf16")
    got = gpu_dilate(plan, w.x, dtype="bf16")
    assert_close(got, oracle.eval_stride(oracle_layers(w.layers, "bf16"), w.x), BF16_TOL, name)
    np.testing.assert_array_equal(got, gpu_dense(plan, w.x, "bf16"))


@pytest.mark.parametrize("name,max_phases", [("c2_1d_1m", None), ("c4_hd", None), ("c5_4k", 32)])
def test_named_full_size_dilate_sampled(name, max_phases):
    """Full-size workloads in the dilated fashion: sampled windows against the
    oracle, and the whole output bit-identical to the dense evaluation."""
    w = wl.make(name)
    plan = dss.Plan.from_workload(w)
    g = plan.geometry(w.x.shape[1], w.x.shape[2])
    log("%s full size dilated" % name)
    got = gpu_dilate(plan, w.x, dtype=w.dtype)
    assert got.shape == (g["out_c"], g["out_h"], g["out_w"])
    np.testing.assert_array_equal(got, gpu_dense(plan, w.x, w.dtype))
    i, j = sampled_windows(g["out_h"], g["out_w"], g["K_h"], g["K_w"], per_phase=1, max_phases=max_phases, seed=3)
    ref = oracle.eval_stride(oracle_layers(w.layers, w.dtype), w.x, windows=(i, j))
    assert_close(got[:, i, j].T, ref, BF16_TOL if w.dtype == "bf16" else F32_TOL, name)


def test_dilate_errors_leave_output_untouched():
    import torch
    w = wl.make("c1_64x64")
    plan = dss.Plan.from_workload(w)
    xd = to_device(w.x, "f32")
    out = torch.full((1, 37, 37), 3.0, device="cuda")
    ws = torch.empty(1 << 22, dtype=torch.uint8, device="cuda")
    stream = dss._stream(None)
    L = dss.lib()
    assert L.dss_eval_dilate(plan.handle, dss._ptr(xd), 64, 64, 4, dss._ptr(out), dss._ptr(ws), ws.numel(),
                             stream) == 1
    assert L.dss_eval_dilate(plan.handle, dss._ptr(xd), 64, 64, 3, dss._ptr(out), dss._ptr(ws), 4096, stream) == 2
    assert L.dss_eval_dilate(plan.handle, dss._ptr(xd), 27, 64, 3, dss._ptr(out), dss._ptr(ws), ws.numel(),
                             stream) == 2
    torch.cuda.synchronize()
    assert torch.all(out == 3.0)


def test_dilate_timing_records():
    w = wl.make("c3_512", H=120, W=130, widths=(16, 32, 64, 128))
    plan = dss.Plan.from_workload(w)
    plan.set_timing(True)
    gpu_dilate(plan, w.x)
    recs = plan.timings()
    names = [r["kernel"] for r in recs]
    # the final 1x1 projection is folded into the dilated conv6x6 epilogue
    assert names[0] == "stuff_pack" and names[-1] == "planar_sum" and names.count("pool_dilate") == 3
    assert names[-2].endswith("_proj")
    assert sum(r["flops"] for r in recs) == pytest.approx(plan.dilate_geometry(120, 130, 5)[3], rel=1e-9)
