"""GPU parity of the patch-by-patch baseline (dss_eval_stride): the strided
network on batches of extracted windows, against the oracle (which is the same
EvalStride definition in fp64) and against the GPU dense evaluation.  The two
GPU paths run the same convolution kernels on the same samples in the same
summation order, so they must agree bit for bit."""
import numpy as np
import pytest

import oracle
from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import assert_close, log, oracle_layers, to_device
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


def gpu_stride_all(plan, x, dtype="f32", batch=37):
    """Every window, in batches of `batch` (the last one ragged)."""
    import torch
    xd = to_device(x, dtype)
    _, H, W = x.shape
    g = plan.geometry(H, W)
    n = g["out_h"] * g["out_w"]
    out = torch.full((g["out_c"], g["out_h"], g["out_w"]), float("nan"), device="cuda")
    ws = torch.empty(max(256, plan.stride_geometry(batch)[0]), dtype=torch.uint8, device="cuda")
    for first in range(0, n, batch):
        plan.eval_stride(xd, first, min(batch, n - first), out=out, workspace=ws)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def gpu_dense(plan, x, dtype="f32"):
    import torch
    out = plan.eval_dense(to_device(x, dtype))
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("name", list(CHAINS))
def test_stride_matches_oracle_and_dense(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    H = 1 if nd == 1 else B[0] + 9
    W = B[1] + (150 if nd == 1 else 11)
    w = wl.custom(arch, C, H, W, seed=5, value_kind="normal")
    plan = dss.Plan(w.layers, nd, C)
    log("stride baseline %s on %s" % (name, w.x.shape))
    got = gpu_stride_all(plan, w.x)
    assert_close(got, oracle.eval_stride(w.layers, w.x), F32_TOL, name)
    np.testing.assert_array_equal(got, gpu_dense(plan, w.x))


def test_stride_exact_integer_chain():
    w = wl.custom(EXACT_ARCH, 16, 30, 33, seed=3, weight_kind="int", value_kind="int")
    plan = dss.Plan(w.layers, 2, 16)
    got = gpu_stride_all(plan, w.x, batch=64)
    np.testing.assert_array_equal(got, oracle.eval_stride(w.layers, w.x))


def test_stride_bf16_matches_dense_bit_exact():
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    w = wl.custom(arch, C, B[0] + 6, B[1] + 9, seed=8, dtype="bf16")
    plan = dss.Plan(w.layers, nd, C, "bf16")
    got = gpu_stride_all(plan, w.x, "bf16", batch=29)
    assert_close(got, oracle.eval_stride(oracle_layers(w.layers, "bf16"), w.x), BF16_TOL, "bf16")
    np.testing.assert_array_equal(got, gpu_dense(plan, w.x, "bf16"))


def test_paper_sweep_family_sample():
    """The runtime-experiment family (3x3 convs, 2x2 pool every third conv) at
    L = 7 on a 240x320 input: a batch in the middle of the grid and the last,
    ragged batch, against the dense evaluation bit for bit."""
    import torch
    layers = wl.init_layers(wl.arch_paper_sweep(7, maps=32), np.random.default_rng(0))
    x = np.random.default_rng(1).random((1, 240, 320), dtype=np.float32)
    plan = dss.Plan(layers, 2, 1)
    g = plan.geometry(240, 320)
    n = g["out_h"] * g["out_w"]
    dense = gpu_dense(plan, x)
    xd = to_device(x, "f32")
    out = torch.full((g["out_c"], g["out_h"], g["out_w"]), float("nan"), device="cuda")
    for first, count in ((n // 3, 1000), (n - 777, 777)):
        plan.eval_stride(xd, first, count, out=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(g["out_c"], -1)
    ref = dense.reshape(g["out_c"], -1)
    for first, count in ((n // 3, 1000), (n - 777, 777)):
        np.testing.assert_array_equal(got[:, first:first + count], ref[:, first:first + count])
    untouched = np.ones(n, bool)
    untouched[n // 3:n // 3 + 1000] = False
    untouched[n - 777:] = False
    assert np.all(np.isnan(got[:, untouched]))


def test_stride_rejects_bad_ranges():
    import torch
    w = wl.make("c1_64x64")
    plan = dss.Plan.from_workload(w)
    xd = to_device(w.x, "f32")
    out = torch.full((1, 37, 37), 5.0, device="cuda")
    ws = torch.empty(1 << 22, dtype=torch.uint8, device="cuda")
    stream = dss._stream(None)
    L = dss.lib()
    for first, count in ((-1, 4), (0, 0), (37 * 37 - 3, 4)):
        st = L.dss_eval_stride(plan.handle, dss._ptr(xd), 64, 64, first, count, dss._ptr(out), dss._ptr(ws),
                               ws.numel(), stream)
        assert st == 1
    st = L.dss_eval_stride(plan.handle, dss._ptr(xd), 64, 64, 0, 100, dss._ptr(out), dss._ptr(ws), 1024, stream)
    assert st == 2
    torch.cuda.synchronize()
    assert torch.all(out == 5.0)
