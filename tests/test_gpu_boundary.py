"""GPU tests of the C ABI's buffer contract: the plan-owned workspace selected by
workspace == NULL, writes confined to the output and workspace (canary bands on
both sides), no reads of unwritten workspace (a NaN-filled workspace changes no
output bit), and the binding's buffer checks."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import assert_close, log, oracle_layers, to_device

pytestmark = pytest.mark.gpu

CANARY = -12345.25


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dss.lib()
    yield
    torch.cuda.synchronize()


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dense_raw(plan, x, out, ws):
    """dss_eval_dense through ctypes; ws None passes NULL (the plan's workspace)."""
    _, H, W = x.shape
    wp = ctypes.c_void_p(None) if ws is None else ctypes.c_void_p(ws.data_ptr())
    wb = 0 if ws is None else ws.numel()
    return dss.lib().dss_eval_dense(plan.handle, ctypes.c_void_p(x.data_ptr()), H, W,
                                    ctypes.c_void_p(out.data_ptr()), wp, wb, _stream())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_null_workspace_plan_owned(dtype):
    """workspace == NULL runs in the plan's own buffer: same bits as a caller
    workspace, including after the buffer grows and for a smaller signal after."""
    import torch
    w0 = wl.make("c3_512", H=80, W=90, widths=(16, 32, 48, 64)) if dtype == "f32" else \
        wl.make("c5_4k", H=170, W=175, widths=(16, 16, 32, 32))
    plan = dss.Plan.from_workload(w0)
    sizes = [(w0.x.shape[1], w0.x.shape[2]), (w0.x.shape[1] + 37, w0.x.shape[2] + 21), (w0.x.shape[1] - 3,
                                                                                       w0.x.shape[2] - 5)]
    for n, (H, W) in enumerate(sizes):
        x = to_device(np.random.default_rng(40 + n).random((w0.x.shape[0], H, W), dtype=np.float32), dtype)
        g = plan.geometry(H, W)
        shape = (g["out_c"], g["out_h"], g["out_w"])
        a = torch.full(shape, CANARY, device="cuda")
        b = torch.full(shape, CANARY, device="cuda")
        ws = torch.empty(g["workspace_bytes"], dtype=torch.uint8, device="cuda")
        assert _dense_raw(plan, x, a, ws) == 0
        status = _dense_raw(plan, x, b, None)
        assert status == 0, dss.lib().dss_last_error().decode()
        torch.cuda.synchronize()
        log("  %s %dx%d NULL workspace vs caller workspace" % (dtype, H, W))
        assert torch.equal(a, b)
        assert not torch.any(b == CANARY)


def test_null_workspace_other_entry_points():
    """Mixed, slide, dilated, strided and backward evaluations also accept NULL."""
    import torch
    w = wl.make("c3_512", H=76, W=81, widths=(16, 32, 48, 64))
    plan = dss.Plan.from_workload(w)
    x = to_device(w.x, "f32")
    H, W = w.x.shape[1:]
    dense = plan.eval_dense(x, workspace=plan.workspace(H, W))
    mixed = plan.eval_mixed(x, 1)
    ref_mixed = plan.eval_mixed(x, 1, workspace=plan.workspace(H, W, ell=1))
    slide = plan.eval_slide(x, 2)
    ref_slide = plan.eval_slide(x, 2, workspace=plan.workspace(H, W))
    dil = plan.eval_dilate(x)
    n = dense.shape[1] * dense.shape[2] - 20       # windows 17 .. the third-last
    strided = plan.eval_stride(x, 17, n)
    gout = torch.randn(dense.shape, generator=torch.Generator(device="cuda").manual_seed(3), device="cuda")
    need = plan.backward_geometry(H, W)[0]
    gw1, gb1, gx1 = plan.backward(x, gout)
    gw2, gb2, gx2 = plan.backward(x, gout, workspace=torch.empty(need, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(mixed, ref_mixed)
    assert torch.equal(slide, ref_slide)
    assert torch.equal(dil, dense)
    flat_d, flat_s = dense.reshape(dense.shape[0], -1), strided.reshape(dense.shape[0], -1)
    assert torch.equal(flat_s[:, 17:17 + n], flat_d[:, 17:17 + n])
    assert torch.equal(gw1, gw2) and torch.equal(gb1, gb2) and torch.equal(gx1, gx2)


@pytest.mark.parametrize("name", ["c3_512", "c5_4k", "c2_1d_1m"])
def test_canary_bands_and_nan_workspace(name):
    """The output sits inside a larger buffer with canary bands on both sides,
    and the workspace inside a larger NaN-filled one (every byte 0xFF: a NaN
    in binary32 and bfloat16).  The evaluation must write only its output, write
    every output sample, touch nothing outside its workspace, and read no
    workspace byte it did not write first (a NaN read would reach an output)."""
    import torch
    sizes = {"c3_512": dict(H=101, W=117, widths=(16, 32, 48, 64)),
             "c5_4k": dict(H=171, W=183, widths=(16, 16, 32, 32)), "c2_1d_1m": dict(W=3001)}
    w = wl.make(name, **sizes[name])
    plan = dss.Plan.from_workload(w)
    H, W = w.x.shape[1:]
    g = plan.geometry(H, W)
    n = g["out_c"] * g["out_h"] * g["out_w"]
    pad = 4099
    buf = torch.full((n + 2 * pad,), CANARY, device="cuda")
    out = buf[pad:pad + n].view(g["out_c"], g["out_h"], g["out_w"])
    wpad = 64 * 1024
    wsbuf = torch.full((g["workspace_bytes"] + 2 * wpad,), 0xFF, dtype=torch.uint8, device="cuda")
    ws = wsbuf[wpad:wpad + g["workspace_bytes"]]
    plan.eval_dense(to_device(w.x, w.dtype), out=out, workspace=ws)
    torch.cuda.synchronize()
    assert torch.all(buf[:pad] == CANARY) and torch.all(buf[pad + n:] == CANARY), "write outside the output"
    assert torch.all(wsbuf[:wpad] == 0xFF) and torch.all(wsbuf[wpad + g["workspace_bytes"]:] == 0xFF), \
        "write outside the workspace"
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got)), "an unwritten (NaN) workspace byte reached the output"
    assert not np.any(got == CANARY)
    ref = oracle.eval_stride(oracle_layers(w.layers, w.dtype), w.x)
    assert_close(got, ref, 2e-2 if w.dtype == "bf16" else 1e-4, name)


def test_binding_rejects_bad_buffers():
    """The binding checks every caller buffer against the plan geometry: the C
    ABI takes no sizes for them."""
    import torch
    w = wl.make("c1_64x64")
    plan = dss.Plan.from_workload(w)
    x = to_device(w.x, "f32")
    bad_outs = [torch.empty((1, 37, 36), device="cuda"), torch.empty((1, 37, 37), dtype=torch.float16, device="cuda"),
                torch.empty((1, 37, 74), device="cuda")[:, :, ::2], torch.empty((1, 37, 37))]
    for out in bad_outs:
        with pytest.raises(ValueError):
            plan.eval_dense(x, out=out)
        with pytest.raises(ValueError):
            plan.eval_mixed(x, 1, out=out)
    with pytest.raises(ValueError):
        plan.eval_slide(x, 1, out=torch.empty(5, device="cuda"))
    with pytest.raises(ValueError):
        plan.eval_dilate(x, out=torch.empty(5, device="cuda"))
    with pytest.raises(ValueError):
        plan.eval_stride(x, 0, 10, out=torch.empty(5, device="cuda"))
    with pytest.raises(ValueError):
        plan.eval_dense(x, workspace=torch.empty(1 << 20, dtype=torch.uint8, device="cuda")[::2])
    gout = torch.zeros((1, 37, 37), device="cuda")
    with pytest.raises(ValueError):
        plan.backward(x, gout[:, :36])
    with pytest.raises(ValueError):
        plan.backward(x, gout, grad_weight=torch.empty(3, device="cuda"))
    t = torch.zeros((4, 3, 8, 8), device="cuda")
    with pytest.raises(ValueError):
        dss.frag(t, 2, 2, 1, 1)                  # 4 fragments given, S_h * S_w = 1
    with pytest.raises(ValueError):
        dss.frag(t, 2, 2, 2, 2, out=torch.empty((16, 3, 4, 3), device="cuda"))
    with pytest.raises(ValueError):
        dss.defrag(t, 2, 2, 2, 2)                # 4 fragments given, (2*2)*(2*2) = 16 expected
    with pytest.raises(ValueError):
        dss.frag(torch.zeros((4, 3, 8, 8), dtype=torch.float64, device="cuda"), 2, 2, 2, 2)
    y = dss.frag(t, 2, 2, 2, 2)
    torch.cuda.synchronize()
    assert y.shape == (16, 3, 4, 4)


@pytest.mark.parametrize("name", ["c3_512", "c5_4k", "c2_1d_1m"])
def test_nan_samples_beyond_the_windows(name):
    """Samples past the last window that a kept output reads play the role of
    the dummy samples of Stuff (Theorem "processing chain": the kept outputs do
    not depend on them).  A signal extended by NaN samples must give finite
    outputs on every window that lies inside the original signal, equal to the
    evaluation of the original signal; a leak through Frag, Defrag, Trim or an
    edge tile would carry a NaN there."""
    import torch
    sizes = {"c3_512": dict(H=97, W=110, widths=(16, 32, 48, 64)),
             "c5_4k": dict(H=170, W=177, widths=(16, 16, 32, 32)), "c2_1d_1m": dict(W=2500)}
    w = wl.make(name, **sizes[name])
    plan = dss.Plan.from_workload(w)
    C, H, W = w.x.shape
    eh = 0 if name == "c2_1d_1m" else 13
    xl = np.full((C, H + eh, W + 21), np.nan, dtype=np.float32)
    xl[:, :H, :W] = w.x
    a = plan.eval_dense(to_device(w.x, w.dtype))
    b = plan.eval_dense(to_device(xl, w.dtype))
    torch.cuda.synchronize()
    a = a.cpu().numpy().astype(np.float64)
    b = b.cpu().numpy().astype(np.float64)[:, :a.shape[1], :a.shape[2]]
    assert np.all(np.isfinite(b)), "a NaN sample reached the output of a window that does not contain it"
    assert_close(b, a, 1e-6, "%s with NaN samples appended" % name)


def test_library_first_then_torch_in_a_fresh_process():
    """A fresh process that creates a plan (the library's HIP runtime) before it
    makes any torch tensor must still get torch's device and a correct result:
    the binding brings torch's runtime up before it loads the library."""
    import os
    import subprocess
    import sys
    code = (
        "import numpy as np\n"
        "from paper_1508_06904_amd import dss, workloads as wl\n"
        "w = wl.make('c1_64x64')\n"
        "plan = dss.Plan.from_workload(w)\n"
        "import torch\n"
        "x = torch.from_numpy(w.x).cuda().contiguous()\n"
        "out = plan.eval_dense(x)\n"
        "torch.cuda.synchronize()\n"
        "o = out.cpu().numpy()\n"
        "print('shape', o.shape, 'finite', bool(np.isfinite(o).all()), flush=True)\n"
        "np.save(sys.argv[1], o)\n")
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "out.npy")
        root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
        r = subprocess.run([sys.executable, "-c", "import sys\n" + code, path], cwd=root, capture_output=True,
                           text=True, timeout=110)
        log(r.stdout.strip() + " " + r.stderr.strip()[-300:])
        assert r.returncode == 0, r.stderr[-2000:]
        got = np.load(path).astype(np.float64)
    w = wl.make("c1_64x64")
    ref = oracle.eval_stride(oracle_layers(w.layers, w.dtype), w.x)
    assert_close(got, ref, 1e-4, "library first, then torch")
