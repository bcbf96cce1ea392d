"""GPU parity of the backward pass (dss_backward_dense) against the oracle's
window-by-window backpropagation.  Integer-valued chains are exact (every
partial sum is an integer below 2^24, so any summation order gives the same
bits, and ties in the max-pool exercise the shared first-maximum rule); random
binary32 chains within 1e-4 * max|oracle| per gradient tensor."""
import numpy as np
import pytest

import oracle
from oracle import backward as ob
from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import log, sampled_windows, to_device
from tests.test_gpu_parity import CHAINS, EXACT_ARCH

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dss.lib()
    yield
    torch.cuda.synchronize()


def gpu_backward(plan, x, G, with_dx=True):
    import torch
    gw, gb, gx = plan.backward(to_device(x, "f32"), to_device(G, "f32"), with_signal_grad=with_dx)
    torch.cuda.synchronize()
    ws, bs = plan.split_grads(gw, gb)
    return ([w.cpu().numpy().astype(np.float64) for w in ws], [b.cpu().numpy().astype(np.float64) for b in bs],
            None if gx is None else gx.cpu().numpy().astype(np.float64))


def close(got, ref, what, tol=TOL):
    scale = float(np.abs(ref).max())
    err = float(np.abs(got - ref).max())
    log("  %s max|err| = %.3e, max|oracle| = %.3e, ratio %.2e" % (what, err, scale, err / max(scale, 1e-300)))
    assert got.shape == ref.shape and np.all(np.isfinite(got))
    assert err <= tol * scale, what


def check_all(got, ref, tag, tol=TOL):
    for t, (a, b) in enumerate(zip(got[0], ref[0])):
        close(a, b, "%s dW%d" % (tag, t), tol)
    for t, (a, b) in enumerate(zip(got[1], ref[1])):
        close(a, b, "%s db%d" % (tag, t), tol)
    if got[2] is not None:
        close(got[2], ref[2], "%s dx" % tag, tol)


@pytest.mark.parametrize("name", ["2d_small_direct", "2d_mfma_mixed", "2d_pool_first", "2d_pool_pool", "1d_c2_like",
                                  "2d_ragged_cin"])
def test_backward_random_chain(name):
    arch, C, nd = CHAINS[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    K = (1, 1)
    for l in w0.layers:
        if l["kind"] == "maxpool":
            K = (K[0] * l["kh"], K[1] * l["kw"])
    H = 1 if nd == 1 else B[0] + K[0] + 3
    W = B[1] + (120 if nd == 1 else 2 * K[1] + 1)
    w = wl.custom(arch, C, H, W, seed=11, value_kind="normal")
    G = np.random.default_rng(12).standard_normal((w.layers[-1]["cout"], H - B[0] + 1, W - B[1] + 1))
    plan = dss.Plan(w.layers, nd, C)
    log("backward %s on %s" % (name, w.x.shape))
    check_all(gpu_backward(plan, w.x, G), ob.dense_backward(w.layers, w.x, G), name)


# Layers with at most 32 input channels take the packed weight-gradient mode
# (several taps share the 64 MFMA columns); these chains give it one channel,
# channel counts that are not powers of two, wide filters split into several tap
# groups, and ragged last groups (filter widths 7, 9, 11, 13 and 5 against group
# capacities of 16, 16, 6, 16 and 6 taps).
NARROW = {
    "2d_narrow": ([("conv", 1, 8, 3, 7, "relu"), ("pool", 2, 2), ("conv", 8, 12, 2, 9, "tanh"),
                   ("conv", 12, 3, 2, 2, "none")], 1, 2),
    "1d_narrow": ([("conv", 5, 24, 1, 13, "relu"), ("pool", 1, 3), ("conv", 24, 32, 1, 11, "relu"),
                   ("conv", 32, 2, 1, 5, "none")], 5, 1),
}


@pytest.mark.parametrize("name", list(NARROW))
def test_backward_narrow_layers(name):
    arch, C, nd = NARROW[name]
    w0 = wl.custom(arch, C, 1, 1, seed=1)
    B = oracle.receptive_field(w0.layers)
    H = 1 if nd == 1 else B[0] + 40
    W = B[1] + (3000 if nd == 1 else 100)
    w = wl.custom(arch, C, H, W, seed=21, value_kind="normal")
    G = np.random.default_rng(22).standard_normal((w.layers[-1]["cout"], H - B[0] + 1, W - B[1] + 1))
    plan = dss.Plan(w.layers, nd, C)
    log("backward %s on %s" % (name, w.x.shape))
    check_all(gpu_backward(plan, w.x, G), ob.dense_backward(w.layers, w.x, G), name)


@pytest.mark.parametrize("kernel", ["mfma", "direct"])
def test_backward_exact_integer_chain(kernel, monkeypatch):
    if kernel == "direct":
        monkeypatch.setenv("DSS_CONV_KERNEL", "direct")
    w = wl.custom(EXACT_ARCH, 16, 27, 31, seed=3, weight_kind="int", value_kind="int")
    B = oracle.receptive_field(w.layers)
    G = np.random.default_rng(5).integers(-2, 3, size=(w.layers[-1]["cout"], 27 - B[0] + 1, 31 - B[1] + 1)).astype(
        np.float64)
    plan = dss.Plan(w.layers, 2, 16)
    got = gpu_backward(plan, w.x, G)
    ref = ob.dense_backward(w.layers, w.x, G)
    for a, b in zip(got[0] + got[1] + [got[2]], ref[0] + ref[1] + [ref[2]]):
        assert np.abs(b).max() < 2 ** 23
        np.testing.assert_array_equal(a, b)


def test_backward_without_signal_gradient():
    arch, C, nd = CHAINS["2d_mfma_mixed"]
    w = wl.custom(arch, C, 60, 61, seed=2, value_kind="normal")
    B = oracle.receptive_field(w.layers)
    G = np.random.default_rng(3).standard_normal((w.layers[-1]["cout"], 60 - B[0] + 1, 61 - B[1] + 1))
    plan = dss.Plan(w.layers, nd, C)
    a = gpu_backward(plan, w.x, G, with_dx=True)
    b = gpu_backward(plan, w.x, G, with_dx=False)
    assert b[2] is None
    for u, v in zip(a[0] + a[1], b[0] + b[1]):
        np.testing.assert_array_equal(u, v)


@pytest.mark.parametrize("name,H,W,widths", [("c3_512", 80, 84, (16, 32, 48, 64)), ("c1_64x64", 64, 64, None)])
def test_backward_named_reduced(name, H, W, widths):
    w = wl.make(name, H=H, W=W, widths=widths)
    g = dss.chain_geometry(w.layers, w.ndim, w.x.shape[0], H, W)
    G = np.random.default_rng(9).standard_normal((g["out_c"], g["out_h"], g["out_w"]))
    plan = dss.Plan.from_workload(w)
    log("backward %s reduced %s" % (name, w.x.shape))
    check_all(gpu_backward(plan, w.x, G), ob.dense_backward(w.layers, w.x, G), name)


def integer_bound(layers, b0):
    """Per conv, a bound on |value| and on every partial sum of an integer
    network with inputs bounded by b0: the largest sum of |w| over one output's
    taps times the input bound, plus |bias| (pooling and ReLU keep the bound)."""
    b, bounds = float(b0), []
    for l in layers:
        if l["kind"] == "conv":
            w = np.abs(np.asarray(l["weight"], dtype=np.float64)).reshape(l["cout"], -1).sum(axis=1)
            b = float(np.max(w * b + np.abs(np.asarray(l["bias"], dtype=np.float64))))
            bounds.append(b)
    return bounds


def _hd_windows(g, seed):
    """16 of the 64 fragment phases plus the corners and edge midpoints."""
    return sampled_windows(g["out_h"], g["out_w"], g["K_h"], g["K_w"], per_phase=1, max_phases=16, seed=seed)


def test_backward_hd_frame_exact_forward():
    """The HD frame at full size in the launch configuration of the benchmark,
    element-wise within 1e-4 * max|oracle| on every weight and bias gradient.

    The gradient depends on discrete decisions of the forward pass (each ReLU
    mask, the position of each pool maximum).  With He-init weights and the
    frame's continuous data, some of an HD window's decisions are closer to a
    tie than binary32 rounding of its sums can resolve (a fp64 forward pass
    counts 40 to 50 of them per window, at 4 sqrt(K) u times the sum of absolute
    products), so binary32 and fp64 take some differently.  Here the network has
    the HD layer shapes but integer parameters (sparse +-1 weights, integer
    biases) and the frame integer samples in [-8, 8], chosen so that every value
    and every partial sum of the forward pass stays far below 2^24: the binary32
    forward pass is exact, its decisions are the oracle's (ties, frequent with
    integers, follow the first-maximum rule on both sides), and what remains is
    the rounding of the gradient sums.  The upstream gradient is nonzero on 24
    sampled windows, so the oracle sums 24 per-window backpropagations."""
    w = wl.make("c4_hd")
    rng = np.random.default_rng(11)
    x = rng.integers(-8, 9, size=w.x.shape).astype(np.float32)
    layers = wl.sparse_integer_layers(w.layers, (8, 8, 8, 16, 64), rng)
    bounds = integer_bound(layers, 8)
    log("HD exact-forward network, value bounds %s" % bounds)
    assert max(bounds) < 2 ** 24
    plan = dss.Plan(layers, 2, 3)
    g = plan.geometry(1080, 1920)
    i, j = _hd_windows(g, seed=4)
    G = np.zeros((g["out_c"], g["out_h"], g["out_w"]))
    G[:, i, j] = np.random.default_rng(6).standard_normal((g["out_c"], len(i)))
    log("HD backward (exact forward) with %d nonzero windows" % len(i))
    got = gpu_backward(plan, x, G, with_dx=False)
    B = (g["B_h"], g["B_w"])
    patches = np.stack([x[:, a:a + B[0], b:b + B[1]] for a, b in zip(i, j)]).astype(np.float64)
    dW, db, _ = ob.strided_backward(layers, patches, G[:, i, j].T)
    for t, (a, b) in enumerate(zip(got[0], dW)):
        close(a, b, "hd exact dW%d" % t)
    for t, (a, b) in enumerate(zip(got[1], db)):
        close(a, b, "hd exact db%d" % t)


def close_l2(got, ref, what, rel_l2=2e-3, rel_max=5e-3):
    """Relative L2 bound plus a loose elementwise one: an extra check of the
    He-init HD frame, whose gradients a few near-tie forward decisions move
    (see test_backward_hd_frame_exact_forward, the element-wise gate)."""
    scale = float(np.abs(ref).max())
    err = np.abs(got - ref)
    l2 = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
    n_out = int(np.sum(err > TOL * scale))
    log("  %s rel L2 %.2e, max|err|/max|oracle| %.2e, elements above 1e-4: %d of %d" % (
        what, l2, float(err.max()) / scale, n_out, err.size))
    assert got.shape == ref.shape and np.all(np.isfinite(got))
    assert l2 <= rel_l2 and float(err.max()) <= rel_max * scale, what


def test_backward_hd_frame_he_init():
    """The HD workload itself (He-init weights, blob frame), upstream gradient
    on 17 sampled windows.  The gradients that no decision touches are held
    element-wise: the last layer is linear, so its bias gradient is sum(G) and
    its weight gradient sum_w G_w * (its input on window w), which a near-tie
    decision moves only by the decision's margin.  The others, whose values a
    flipped decision moves, get the relative L2 check."""
    w = wl.make("c4_hd")
    plan = dss.Plan.from_workload(w)
    g = plan.geometry(1080, 1920)
    i, j = sampled_windows(g["out_h"], g["out_w"], g["K_h"], g["K_w"], per_phase=1, max_phases=8, seed=4)
    G = np.zeros((g["out_c"], g["out_h"], g["out_w"]))
    G[:, i, j] = np.random.default_rng(6).standard_normal((g["out_c"], len(i)))
    log("HD backward with %d nonzero windows" % len(i))
    got = gpu_backward(plan, w.x, G, with_dx=False)
    B = (g["B_h"], g["B_w"])
    patches = np.stack([w.x[:, a:a + B[0], b:b + B[1]] for a, b in zip(i, j)]).astype(np.float64)
    dW, db, _ = ob.strided_backward(w.layers, patches, G[:, i, j].T)
    close(got[0][-1], dW[-1], "hd dW_last")
    close(got[1][-1], db[-1], "hd db_last")
    close(got[1][-1], G.sum(axis=(1, 2)), "hd db_last vs sum(G)", tol=1e-6)
    for t, (a, b) in enumerate(zip(got[0][:-1], dW[:-1])):
        close_l2(a, b, "hd dW%d" % t)
    for t, (a, b) in enumerate(zip(got[1][:-1], db[:-1])):
        close_l2(a, b, "hd db%d" % t)
    # the backward pass is linear in G with the forward decisions fixed: doubling
    # G doubles every intermediate exactly, so every gradient doubles bit for bit
    got2 = gpu_backward(plan, w.x, 2.0 * G, with_dx=False)
    for a, b in zip(got[0] + got[1], got2[0] + got2[1]):
        np.testing.assert_array_equal(2.0 * a, b)


def test_backward_rejects_bf16_and_short_workspace():
    import torch
    w = wl.make("c1_64x64")
    G = to_device(np.ones((1, 37, 37)), "f32")
    plan = dss.Plan(w.layers, 2, 1, "bf16")
    with pytest.raises(dss.DssError) as e:
        plan.backward(to_device(w.x, "bf16"), G)
    assert e.value.status == 3
    plan = dss.Plan.from_workload(w)
    gw = torch.full((plan.backward_geometry(64, 64)[1],), 9.0, device="cuda")
    gb = torch.full((plan.backward_geometry(64, 64)[2],), 9.0, device="cuda")
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    with pytest.raises(dss.DssError) as e:
        plan.backward(to_device(w.x, "f32"), G, grad_weight=gw, grad_bias=gb, workspace=ws)
    assert e.value.status == 2
    torch.cuda.synchronize()
    assert torch.all(gw == 9.0) and torch.all(gb == 9.0)


def test_backward_timing_records():
    w = wl.make("c3_512", H=100, W=104, widths=(16, 32, 64, 128))
    plan = dss.Plan.from_workload(w)
    g = plan.geometry(100, 104)
    G = np.random.default_rng(1).standard_normal((g["out_c"], g["out_h"], g["out_w"]))
    plan.set_timing(True)
    gpu_backward(plan, w.x, G)
    recs = plan.timings()
    names = [r["kernel"] for r in recs]
    assert names.count("wgrad_mfma") == 5 and names.count("pool_frag_backward") == 3
    assert sum(r["flops"] for r in recs) == pytest.approx(plan.backward_geometry(100, 104)[3], rel=1e-9)
