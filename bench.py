"""Benchmark: dense window outputs per second of the exact dense evaluation on one MI355X.

One step = one full dss_eval_dense of a frame that is already resident in HBM:
Stuff, every convolution (MFMA implicit GEMM or direct), every sliding
max-pool + Frag, and the final Defrag + Trim -- the same inclusive accounting
as the paper's runtime experiment (Sect. 6.3).  The default workload is the HD
frame (3x1080x1920 binary32, conv widths 64/128/256/512), the configuration the
MFMA-utilisation target is stated for.

Prints ONE JSON line with the throughput, a roofline object for the dominant
kernel, a per-kernel breakdown, and the oracle's throughput on a bounded window
sample of the same frame (CPU baseline, also used as a parity spot check).  The
K timed steps run twice: plainly, for the throughput, and with the library's
per-launch HIP events on its stream, for the per-kernel durations of the
roofline and the breakdown (an event pair per launch costs about as much as a
launch, which shows on the 64x64 workload).

`--sweep` runs the paper's runtime experiment shape instead (Sect. 6.3: one
240x320 random image, L = 1..15 layers of 3x3 convolutions with 128 maps and a
2x2 max-pool after every third one, random weights): per L, the dense
evaluation against the patch-by-patch baseline (dss_eval_stride, all windows
in memory-sized batches through the same kernels), and prints one JSON line
with both times and the speed-up.

`--fashion dilate` times the dilated fashion instead of the sliding one
(appendix, Definition "evaldilate": the same dense output, computed on one
full-resolution signal with dilated taps instead of fragments), for an A/B of
the two schemes on the same kernels.

`--backward` times one whole-image gradient step instead (dss_backward_dense:
the dense forward pass keeping every layer's output, then the gradients of all
weights and biases for a random upstream gradient of the dense output -- the
fine-tuning step of Sect. 6.2); the metric counts the windows whose gradients a
step accumulates.

`--ell l` (l > 0) times the mixed evaluation instead (appendix, Theorem
"evalrelaxslide"): the first l chain layers pool with stride, and the output is
the dense output downsampled by k*_l per axis; the metric then counts those
window outputs.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}   # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0

WORKLOAD_TEXT = {
    "c1_64x64": "2-D 1x64x64 fp32, conv5x5 1-4 tanh, pool2, conv5x5 4-8 tanh, pool2, conv4x4 8-1 (B=28)",
    "c2_1d_1m": "1-D 1x1048576 fp32, conv9 1-16-32-64 relu + pool2 x3, conv8 64-2 (B=120)",
    "c3_512": "2-D 3x512x512 fp32, conv5x5 3-32, pool2, conv5x5 32-64, pool2, conv3x3 64-128, pool2, conv6x6 128-256, conv1x1 256-2 (B=68)",
    "c4_hd": "2-D 3x1080x1920 fp32 HD frame, conv5x5 3-64, pool2, conv5x5 64-128, pool2, conv3x3 128-256, pool2, conv6x6 256-512, conv1x1 512-2 (B=68)",
    "c5_4k": "2-D 3x2160x3840 bf16 4K frame, 4x(conv3x3, conv3x3, pool2) 32/64/128/256, conv6x6 256-512, conv1x1 512-4 (B=156)",
}


# The workloads measured besides the headline (HD frame) in a default run, the
# fewest timed steps for each (the small ones run well under a millisecond), and
# the oracle's time budget on each (the 64x64 frame is checked in full).
EXTRA_CONFIGS = ("c1_64x64", "c2_1d_1m", "c3_512", "c5_4k")
MIN_STEPS = {"c1_64x64": 500, "c2_1d_1m": 200, "c3_512": 100}
EXTRA_CPU_SECONDS = {"c1_64x64": 6.0, "c2_1d_1m": 16.0, "c3_512": 6.0, "c5_4k": 8.0}


def host_cpu_info():
    """The host the oracle runs on: logical CPUs, the ones this process may use,
    physical cores and the CPU model (from /proc/cpuinfo)."""
    info = {"nproc": os.cpu_count()}
    try:
        info["affinity_cpus"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        pass
    try:
        cores, model, phys = set(), None, None
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k, v = k.strip(), v.strip()
            if k == "model name" and model is None:
                model = v
            elif k == "physical id":
                phys = v
            elif k == "core id":
                cores.add((phys, v))
        info["physical_cores"] = len(cores) or None
        info["cpu_model"] = model
    except OSError:
        pass
    return info


def child_processes():
    """Processes this benchmark left running (there should be none)."""
    try:
        import psutil
        return [{"pid": c.pid, "name": c.name(), "cmdline": " ".join(c.cmdline())[:200]}
                for c in psutil.Process().children(recursive=True)]
    except Exception as e:   # psutil missing or the process table unreadable
        return [{"error": str(e)}]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def profiled_traffic(kernel, config):
    """HBM bytes per launch of `kernel` on `config` from the committed rocprofv3
    counter summaries (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), or None
    when no summary covers it or the kernel source changed since it was taken
    (the hash covers the kernel's own source file and the shared device header)."""
    import glob
    import hashlib
    files = ("backward.hip" if kernel.startswith("wgrad") else "conv_mfma.hip", "dev_common.h")
    src = b"".join(open(os.path.join(ROOT, "paper_1508_06904_amd", "csrc", f), "rb").read() for f in files)
    h = hashlib.sha256(src).hexdigest()[:16]
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for line in open(path):
            if line.startswith("traffic-json:"):
                d = json.loads(line.split(":", 1)[1])
                if d["kernel"] == kernel and d["workload"] == config and d["source_sha256_16"] == h:
                    return d["traffic_bytes_per_launch"]
    return None


def summarize(recs, steps):
    by = {}
    for r in recs:
        d = by.setdefault(r["kernel"], {"ms": 0.0, "flops": 0.0, "bytes": 0.0, "n": 0})
        d["ms"] += r["ms"]
        d["flops"] += r["flops"]
        d["bytes"] += r["bytes"]
        d["n"] += 1
    out = []
    for k, d in sorted(by.items(), key=lambda kv: -kv[1]["ms"]):
        e = {"kernel": k, "launches_per_step": d["n"] / steps, "ms_per_step": d["ms"] / steps,
             "avg_launch_ms": d["ms"] / d["n"]}
        if d["flops"] > 0:
            e["tflops"] = d["flops"] / d["ms"] / 1e9
        if d["bytes"] > 0:
            e["gbs"] = d["bytes"] / d["ms"] / 1e6
            if d["flops"] == 0:                       # HBM-bound data movement: pooling, Frag, Defrag
                e["frac_of_hbm_peak"] = e["gbs"] / PEAK_HBM_GBS
        out.append((e, d))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=None, choices=sorted(WORKLOAD_TEXT),
                    help="headline workload (default c4_hd, plus per-workload entries for the other four)")
    ap.add_argument("--configs", default=None,
                    help="comma-separated workloads measured after the headline into the 'configs' key "
                         "(default: the other four named workloads when --config is not given; '' for none)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ell", type=int, default=0,
                    help="mixed level: chain layers 1..ell run relaxed (0 = dense evaluation)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run plain 1 GiB device-to-device copies (scales the HBM byte counters of a profiler)")
    ap.add_argument("--fashion", default="slide", choices=("slide", "dilate"),
                    help="dense evaluation scheme: fragments (slide) or dilated taps (dilate)")
    ap.add_argument("--backward", action="store_true",
                    help="time dss_backward_dense (forward + weight/bias gradients) instead of the forward pass")
    ap.add_argument("--sweep", action="store_true",
                    help="EvalSlide vs patch-by-patch EvalStride on the paper's 240x320 family, L = 1..15")
    ap.add_argument("--sweep-layers", default="1-15", help="range of L for --sweep, e.g. 1-15 or 12")
    args = ap.parse_args()
    args.config_given = args.config is not None
    args.config = args.config or "c4_hd"
    if args.calibrate_copy:
        return calibrate_copy()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: the dense evaluation of one frame runs on a single GPU in this "
              "build (multi-GPU sharding is a design note only); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    torch.cuda.set_device(0)
    if args.sweep:
        return sweep(args)
    record = measure(args, args.config, args.steps, args.warmup, args.cpu_seconds, args.no_cpu_baseline)
    extra = [c for c in args.configs.split(",") if c] if args.configs is not None else \
        ([] if args.config_given or args.ell or args.backward or args.fashion != "slide"
         else [c for c in EXTRA_CONFIGS if c != args.config])
    if extra:
        record["configs"] = {}
        for c in extra:
            steps = max(args.steps, MIN_STEPS.get(c, 0))
            r = measure(argparse.Namespace(ell=0, fashion="slide", backward=False), c, steps, args.warmup,
                        EXTRA_CPU_SECONDS.get(c, 6.0), args.no_cpu_baseline)
            record["configs"][c] = {k: r[k] for k in ("value", "unit", "ms_per_step", "ms_per_step_median", "steps",
                                                      "dtype", "config", "roofline", "conv_aggregate", "breakdown",
                                                      "cpu_baseline") if k in r}
            if "parity_spot_check" in r:
                record["configs"][c]["parity_spot_check"] = r["parity_spot_check"]
    record["children_at_exit"] = child_processes()
    print(json.dumps(record), flush=True)


def measure(args, name, steps, warmup, cpu_seconds, no_cpu):
    """One workload: `warmup` untimed steps, then `steps` timed steps twice
    (plain, then with per-launch events); the record of its JSON line."""
    import numpy as np
    import torch

    from paper_1508_06904_amd import dss, workloads as wl

    t0 = time.time()
    w = wl.make(name)
    log("workload %s %s generated in %.1fs" % (name, w.x.shape, time.time() - t0))
    plan = dss.Plan.from_workload(w)
    C, H, W = w.x.shape
    ell = args.ell
    g = plan.geometry(H, W, ell)
    x = torch.from_numpy(w.x).to("cuda")
    if w.dtype == "bf16":
        x = x.to(torch.bfloat16)
    x = x.contiguous()
    out = torch.empty((g["out_c"], g["out_h"], g["out_w"]), dtype=torch.float32, device="cuda")
    if args.backward and (ell or args.fashion != "slide" or w.dtype != "f32"):
        log("--backward times the binary32 dense evaluation's gradient step only")
        sys.exit(2)
    if args.fashion == "dilate" and ell:
        log("--fashion dilate evaluates the dense output; it does not combine with --ell")
        sys.exit(2)
    if args.backward:
        need, wf, bf, bwd_flops = plan.backward_geometry(H, W, False)
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
        gw = torch.empty(wf, dtype=torch.float32, device="cuda")
        gb = torch.empty(bf, dtype=torch.float32, device="cuda")
        gen = torch.Generator(device="cuda")
        gen.manual_seed(7)
        gout = torch.randn((g["out_c"], g["out_h"], g["out_w"]), generator=gen, device="cuda")
        g["conv_flops"] = bwd_flops
    elif args.fashion == "dilate":
        _, _, need, dil_flops = plan.dilate_geometry(H, W, g["n_chain"])
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
        g["conv_flops"] = dil_flops
    else:
        ws = plan.workspace(H, W, ell=ell)
    windows = g["out_h"] * g["out_w"]

    def step():
        if args.backward:
            plan.backward(x, gout, with_signal_grad=False, grad_weight=gw, grad_bias=gb, workspace=ws)
        elif args.fashion == "dilate":
            plan.eval_dilate(x, out=out, workspace=ws)
        elif ell == 0:
            plan.eval_dense(x, out=out, workspace=ws)
        else:
            plan.eval_mixed(x, ell, out=out, workspace=ws)

    for i in range(warmup):
        step()
        torch.cuda.synchronize()
        log("warmup %d done" % i)

    def timed(instrumented):
        """K steps between events; with instrumented, the library also records an
        event pair around every kernel launch (the per-kernel durations of the
        roofline and the breakdown)."""
        plan.set_timing(instrumented)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        evs[0].record()
        for i in range(steps):
            step()
            evs[i + 1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(steps))
        med = per[len(per) // 2] if len(per) % 2 else 0.5 * (per[len(per) // 2 - 1] + per[len(per) // 2])
        recs = plan.timings() if instrumented else None
        plan.set_timing(False)
        return evs[0].elapsed_time(evs[-1]), med, wall, recs

    # the throughput: K plain steps; then the same K steps with per-launch events
    # (on small workloads an event pair per launch costs as much as the launch)
    ms_total, ms_median, wall_s, _ = timed(False)
    ms_total_inst, _, _, recs = timed(True)
    ms_per_step = ms_total / steps
    log("timed %d steps: %.3f ms/step (host wall %.3f ms/step); with per-launch events %.3f ms/step" % (
        steps, ms_per_step, 1e3 * wall_s / steps, ms_total_inst / steps))

    kernels = summarize(recs, steps)
    breakdown = [e for e, _ in kernels]
    dom, domd = kernels[0]
    if domd["flops"] > 0:
        ach = (domd["flops"] / domd["n"]) / (domd["ms"] / domd["n"]) / 1e9
        peak = PEAK_TFLOPS[w.dtype]
        roof = {"bound": "mfma", "kernel": dom["kernel"], "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                "frac": ach / peak, "traffic": profiled_traffic(dom["kernel"], name if ell == 0 and args.fashion == "slide"
                                           and not args.backward
                                           else "%s_%s%d%s" % (name, args.fashion, ell,
                                                               "_backward" if args.backward else "")),
                "traffic_unit": "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "per_launch": {"flops": domd["flops"] / domd["n"], "avg_ms": domd["ms"] / domd["n"],
                               "launches_per_step": domd["n"] / steps}}
    else:
        ach = (domd["bytes"] / domd["n"]) / (domd["ms"] / domd["n"]) / 1e6
        roof = {"bound": "hbm", "kernel": dom["kernel"], "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": ach / PEAK_HBM_GBS, "traffic": None,
                "per_launch": {"bytes": domd["bytes"] / domd["n"], "avg_ms": domd["ms"] / domd["n"]}}
    conv_ms = sum(d["ms"] for e, d in kernels if d["flops"] > 0) / steps
    conv_tflops = g["conv_flops"] / (conv_ms * 1e9) if conv_ms > 0 else None

    config = {"workload": name + ": " + WORKLOAD_TEXT[name], "input": [C, H, W],
              "windows_per_step": windows, "receptive_field": [g["B_h"], g["B_w"]],
              "k_star": [g["K_h"], g["K_w"]], "conv_gflop_per_step": g["conv_flops"] / 1e9}
    if args.fashion == "dilate":
        config["fashion"] = "dilated taps on the full-resolution signal (no fragments)"
    if args.backward:
        config["step"] = ("dss_backward_dense: forward keeping every layer's output + weight and bias gradients "
                          "of a random upstream gradient (no signal gradient)")
    if ell:
        config.update({"mixed_level": ell, "output_spacing": [g["step_h"], g["step_w"]],
                       "trimmed": [g["trim_h"], g["trim_w"]], "stuffed": [g["r_h"], g["r_w"]]})
    record = {
        "metric": ("whole-image gradient steps: windows/sec at 1 MI355X" if args.backward else
                   "dense window outputs/sec at 1 MI355X" if ell == 0 else
                   "mixed-fashion window outputs/sec at 1 MI355X (every k*_l-th window per axis)"),
        "value": windows / (ms_per_step / 1e3),
        "unit": "windows/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_median": ms_median,
        "ms_per_step_with_launch_events": ms_total_inst / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded), random He-init weights",
        "config": config,
        "roofline": roof,
        "conv_aggregate": {"tflops": conv_tflops, "frac_of_peak": (conv_tflops / PEAK_TFLOPS[w.dtype]) if conv_tflops else None,
                           "ms_per_step": conv_ms},
        "breakdown": breakdown,
        "cpu_baseline": None,
    }

    if not no_cpu and args.backward:
        record["cpu_baseline"] = cpu_baseline_backward(w, g, cpu_seconds)
    elif not no_cpu:
        record["cpu_baseline"], record["parity_spot_check"] = cpu_baseline(w, g, out, cpu_seconds)
    del plan, out, x
    if "ws" in locals():
        del ws
    torch.cuda.empty_cache()
    return record




def sweep(args, H=240, W=320, maps=128, ws_budget=48e9):
    """Sect. 6.3 runtime experiment shape on one MI355X.  Per L: EvalSlide is one
    dss_eval_dense (Stuff, Frag, Defrag and Trim included, as the paper counts
    it); EvalStride is dss_eval_stride over every window in batches that fit
    `ws_budget` bytes of workspace.  The paper leaves patch extraction and output
    assembly out of the EvalStride time; both figures are reported."""
    import numpy as np
    import torch

    from paper_1508_06904_amd import dss, workloads as wl

    lo, _, hi = args.sweep_layers.partition("-")
    Ls = range(int(lo), int(hi or lo) + 1)
    x = wl.uniform_image(np.random.default_rng(0), 1, H, W)
    xd = torch.from_numpy(x).to("cuda").contiguous()
    rows = []
    for L in Ls:
        layers = wl.init_layers(wl.arch_paper_sweep(L, maps), np.random.default_rng(100 + L))
        plan = dss.Plan(layers, 2, 1)
        g = plan.geometry(H, W)
        n = g["out_h"] * g["out_w"]
        dense = torch.empty((g["out_c"], g["out_h"], g["out_w"]), dtype=torch.float32, device="cuda")
        ws = plan.workspace(H, W)
        reps = max(3, args.steps)
        for _ in range(2):
            plan.eval_dense(xd, out=dense, workspace=ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            plan.eval_dense(xd, out=dense, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        slide_ms = e0.elapsed_time(e1) / reps

        per_ws = plan.stride_geometry(1024)[0] / 1024.0
        batch = int(max(1, min(n, ws_budget // per_ws)))
        sws = torch.empty(max(256, plan.stride_geometry(batch)[0]), dtype=torch.uint8, device="cuda")
        strided = torch.full_like(dense, float("nan"))
        plan.eval_stride(xd, 0, min(batch, n), out=strided, workspace=sws)   # warm-up batch
        torch.cuda.synchronize()
        plan.set_timing(True)
        e0.record()
        for first in range(0, n, batch):
            plan.eval_stride(xd, first, min(batch, n - first), out=strided, workspace=sws)
        e1.record()
        torch.cuda.synchronize()
        stride_ms = e0.elapsed_time(e1)
        recs = plan.timings()
        plan.set_timing(False)
        io_ms = sum(r["ms"] for r in recs if r["kernel"] in ("patch_pack", "window_scatter"))
        conv_ms = sum(r["ms"] for r in recs if r["flops"] > 0)
        stride_flops = sum(r["flops"] for r in recs)
        same = bool(torch.equal(strided, dense))
        row = {"L": L, "B": g["B_h"], "k_star": g["K_h"], "windows": n, "batch": batch,
               "slide_ms": slide_ms, "stride_ms": stride_ms, "stride_ms_without_patch_io": stride_ms - io_ms,
               "speedup": stride_ms / slide_ms, "speedup_paper_protocol": (stride_ms - io_ms) / slide_ms,
               "slide_conv_tflop": g["conv_flops"] / 1e12, "stride_conv_tflop": stride_flops / 1e12,
               "stride_conv_tflops": stride_flops / conv_ms / 1e9 if conv_ms > 0 else None,
               "bit_identical": same}
        log("L=%2d B=%3d windows=%6d  slide %.3f ms  stride %.1f ms (%.1f without patch I/O)  speed-up %.1fx  "
            "identical=%s" % (L, g["B_h"], n, slide_ms, stride_ms, stride_ms - io_ms, stride_ms / slide_ms, same))
        rows.append(row)
        del plan, dense, ws, sws, strided
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "EvalSlide speed-up over patch-by-patch EvalStride at 1 MI355X",
                      "unit": "x", "higher_is_better": True, "dtype": "f32", "data": "synthetic (seeded)",
                      "config": {"workload": "paper runtime-experiment shape: 1x%dx%d U[0,1) image, L 3x3 conv+ReLU "
                                             "layers with %d maps, 2x2 max-pool after every third conv unless last, "
                                             "He-init weights" % (H, W, maps)},
                      "rows": rows}), flush=True)


def calibrate_copy(n=4, nbytes=1 << 30):
    """n plain copies of an nbytes buffer: a kernel whose true HBM traffic is known
    (nbytes read + nbytes written per launch)."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(n):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / n
    # the achievable streaming rate of a plain copy, the practical ceiling the
    # HBM-bound kernels are compared with (besides the 8 TB/s peak)
    print(json.dumps({"calibration": "device copy", "bytes_read_per_launch": nbytes,
                      "bytes_written_per_launch": nbytes, "launches": n, "ms_per_launch": ms,
                      "gbs": 2 * nbytes / ms / 1e6, "frac_of_hbm_peak": 2 * nbytes / ms / 1e6 / PEAK_HBM_GBS}),
          flush=True)


def cpu_baseline_backward(w, g, target_s):
    """Times the oracle's window-by-window backpropagation (float64 numpy, BLAS
    threads) on a bounded seeded sample of the frame's windows."""
    import numpy as np

    from oracle import backward as ob
    from paper_1508_06904_amd import workloads as wl

    try:
        import threadpoolctl
        cores = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    except Exception:
        cores = 1
    si, sj = wl.sample_windows(g["out_h"], g["out_w"], g["K_h"], g["K_w"], per_phase=1, seed=2)
    B = (g["B_h"], g["B_w"])
    rng = np.random.default_rng(3)

    def run(first, n):
        sel = slice(first, first + n)
        patches = np.stack([w.x[:, a:a + B[0], b:b + B[1]] for a, b in zip(si[sel], sj[sel])]).astype(np.float64)
        ob.strided_backward(w.layers, patches, rng.standard_normal((n, g["out_c"])))

    t = time.perf_counter()
    run(0, 1)
    probe = time.perf_counter() - t
    n = int(max(1, min(len(si), target_s / max(probe, 1e-6))))
    t = time.perf_counter()
    for first in range(0, n, 16):
        run(first, min(16, n - first))
    cpu_s = time.perf_counter() - t
    log("cpu baseline (backward): %d windows in %.1fs" % (n, cpu_s))
    return {"value": n / cpu_s, "unit": "windows/s", "cores": cores, "kind": "oracle", "host": host_cpu_info(),
            "sample": "%d seeded windows of the frame (corners, edges, fragment phases); float64 window-by-window "
                      "backpropagation through the strided network" % n, "seconds": cpu_s}


def cpu_baseline(w, g, out, target_s):
    """Times the oracle (plain fp64 EvalStride, OpenMP over windows) on a bounded,
    seeded sample of this frame's windows that covers every fragment phase, and
    compares the GPU output at those windows."""
    import numpy as np

    import oracle
    from paper_1508_06904_amd import workloads as wl

    layers = w.layers
    if w.dtype == "bf16":
        layers = [dict(l, weight=wl.to_bf16_representable(l["weight"])) if l["kind"] == "conv" else l
                  for l in w.layers]
    threads = oracle.threads()
    # output positions are sampled over the phases of the final defragmentation
    # (k*_L / k*_l per axis); output (i, j) is the window at (k*_l,h i, k*_l,w j)
    Gh, Gw = g["K_h"] // g["step_h"], g["K_w"] // g["step_w"]
    sh, sw = g["step_h"], g["step_w"]
    si, sj = wl.sample_windows(g["out_h"], g["out_w"], Gh, Gw, per_phase=1, seed=1)
    nprobe = min(len(si), threads)
    t = time.perf_counter()
    oracle.eval_stride(layers, w.x, windows=(sh * si[:nprobe], sw * sj[:nprobe]))
    probe_s = time.perf_counter() - t
    windows = g["out_h"] * g["out_w"]
    full = windows * probe_s / nprobe <= target_s
    if full:
        # the whole frame fits the time budget: every window
        ii, jj = np.meshgrid(np.arange(g["out_h"]), np.arange(g["out_w"]), indexing="ij")
        si, sj = ii.reshape(-1), jj.reshape(-1)
        n = len(si)
    else:
        n = int(max(nprobe, min(4096, target_s / max(probe_s, 1e-6) * nprobe)))
        if n > len(si):
            reps = -(-n // max(1, len(si))) + 1
            si, sj = wl.sample_windows(g["out_h"], g["out_w"], Gh, Gw, per_phase=reps, seed=1)
        n = min(n, len(si))
        si, sj = si[:n], sj[:n]
    log("cpu baseline: %d windows on %d threads (probe %.2fs for %d)" % (n, threads, probe_s, nprobe))
    t = time.perf_counter()
    ref = oracle.eval_stride(layers, w.x, windows=(sh * si, sw * sj))
    cpu_s = time.perf_counter() - t
    got = out[:, si, sj].T.cpu().numpy().astype(np.float64) if hasattr(out, "cpu") else out
    err = float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-300))
    H, W = w.x.shape[1:]
    sample = ("every window (%d) of the %dx%d frame" % (n, H, W) if full else
              "%d seeded windows of the %dx%d frame covering every fragment phase (i mod %d, j mod %d) "
              "plus corners and edge midpoints%s" % (n, H, W, Gh, Gw, "" if sh == sw == 1 else
                                                      " of the output grid (window spacing %dx%d)" % (sh, sw)))
    base = {"value": n / cpu_s, "unit": "windows/s", "cores": threads, "kind": "oracle",
            "sample": sample + "; fp64 EvalStride per window, plain C with OpenMP over windows",
            "seconds": cpu_s, "extrapolated_full_frame_s": windows * cpu_s / n, "host": host_cpu_info()}
    tol = 2e-2 if w.dtype == "bf16" else 1e-4
    spot = {"windows": n, "max_abs_err_over_max_abs_oracle": err, "tolerance": tol, "pass": err <= tol}
    log("cpu baseline %.2f windows/s; parity spot check %.3e (tol %.0e)" % (base["value"], err, tol))
    return base, spot


if __name__ == "__main__":
    main()
