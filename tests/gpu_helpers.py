"""Shared glue of the GPU tests: move seeded inputs to the device, run the
library through its C ABI, run the oracle on the same inputs, compare."""
import sys

import numpy as np

import oracle
from paper_1508_06904_amd import dss, workloads as wl


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(x, dtype):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda")
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.contiguous()


def oracle_layers(layers, dtype):
    """The weights the oracle sees: bfloat16-rounded for bfloat16 plans (the
    plan rounds its own copy independently), biases unchanged."""
    if dtype != "bf16":
        return layers
    out = []
    for l in layers:
        if l["kind"] == "conv":
            out.append(dict(l, weight=wl.to_bf16_representable(l["weight"])))
        else:
            out.append(l)
    return out


def gpu_dense(layers, x, ndim, dtype="f32", plan=None):
    import torch
    if plan is None:
        plan = dss.Plan(layers, ndim, x.shape[0], dtype)
    out = plan.eval_dense(to_device(x, dtype))
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), plan


def assert_close(gpu, ref, rel, what=""):
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), "non-finite GPU output " + what
    scale = float(np.abs(ref).max())
    err = float(np.abs(gpu - ref).max())
    log("  %s max|err| = %.3e, max|oracle| = %.3e, ratio = %.3e (bound %.1e)" % (what, err, scale,
                                                                                    err / max(scale, 1e-300), rel))
    assert err <= rel * scale, "%s: max|err| %.3e > %.1e * max|oracle| %.3e" % (what, err, rel, scale)


def kstar(arch):
    kh = kw = 1
    for s in arch:
        if s[0] == "pool":
            kh *= s[1]
            kw *= s[2]
    return kh, kw


def sampled_windows(out_h, out_w, Kh, Kw, per_phase=1, max_phases=None, seed=0):
    i, j = wl.sample_windows(out_h, out_w, Kh, Kw, per_phase, seed=seed)
    if max_phases is not None and len(i) > max_phases + 8:
        rng = np.random.default_rng(seed + 99)
        keep = np.sort(rng.choice(len(i), size=max_phases, replace=False))
        corners = np.array([k for k in range(len(i)) if (i[k] in (0, out_h - 1) or j[k] in (0, out_w - 1))])
        keep = np.unique(np.concatenate([keep, corners])).astype(np.int64)
        i, j = i[keep], j[keep]
    return i, j


def oracle_windows(layers, x, i, j):
    """Oracle output at listed windows: [nwin][Cout]."""
    return oracle.eval_stride(layers, x, windows=(i, j))


def check_bf16_storage_model(out, layers, x, plan_records, tol, what):
    """A bfloat16 result against the oracle's bfloat16 storage model: the exact
    evaluation with every stored activation rounded to bfloat16, except before a
    final projection folded into the previous convolution (the launch records
    show the fold), which reads binary32 activations."""
    import oracle.bf16
    fold = any(r["kernel"].endswith("_proj") for r in plan_records)
    emu = oracle.bf16.eval_dilate_bf16_storage(layers, x, fold=fold)
    assert_close(out, emu, tol, "%s vs bfloat16 storage model" % what)

