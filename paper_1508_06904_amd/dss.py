"""Python binding of libdss.so (include/dss.h): argument marshalling only.

Every step of the dense evaluation runs in the library's HIP kernels; torch is
used here for device memory (tensors whose data pointers are handed to the C
ABI) and for the current HIP stream.  There is no fallback: if libdss.so is
missing or a call fails, a `DssError` is raised.

Layers are the dicts produced by `workloads`:
  {"kind": "conv", "cin", "cout", "fh", "fw", "act", "weight": [cout][cin][fh][fw], "bias": [cout]}
  {"kind": "maxpool", "kh", "kw"}
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdss.so")

DSS_F32, DSS_BF16 = 0, 1
DTYPES = {"f32": DSS_F32, "bf16": DSS_BF16}
ACTS = {"none": 0, "relu": 1, "tanh": 2}


class DssError(RuntimeError):
    def __init__(self, status, what, detail):
        super().__init__("%s failed with status %d (%s): %s" % (what, status, _STATUS.get(status, "?"), detail))
        self.status = status


_STATUS = {0: "ok", 1: "invalid", 2: "shape", 3: "unsupported", 4: "nomem", 5: "hip"}


class Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("cin", ctypes.c_int32), ("cout", ctypes.c_int32),
                ("fh", ctypes.c_int32), ("fw", ctypes.c_int32), ("act", ctypes.c_int32),
                ("kh", ctypes.c_int32), ("kw", ctypes.c_int32),
                ("weight", ctypes.POINTER(ctypes.c_float)), ("bias", ctypes.POINTER(ctypes.c_float))]


class Geometry(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("ndim", "in_c", "out_c", "n_chain", "B_h", "B_w", "K_h", "K_w", "r_h", "r_w",
                 "D_h", "D_w", "out_h", "out_w", "dtype", "ell", "step_h", "step_w", "trim_h", "trim_w")] + \
               [("workspace_bytes", ctypes.c_int64), ("conv_flops", ctypes.c_double),
                ("pool_bytes", ctypes.c_double), ("total_bytes", ctypes.c_double)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class LayerGeometry(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("c_h", "c_w", "k_h", "k_w", "kstar_h", "kstar_w", "u_h", "u_w", "U_h", "U_w", "F",
                 "channels", "has_conv", "has_pool", "relaxed", "reserved")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_ if n != "reserved"}


class LaunchRecord(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char_p), ("chain_layer", ctypes.c_int32), ("tile_mode", ctypes.c_int32),
                ("ms", ctypes.c_double), ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


EXPORTS = ("dss_chain_geometry", "dss_chain_layer_geometry", "dss_plan_create", "dss_plan_destroy",
           "dss_plan_geometry", "dss_plan_layer_geometry", "dss_eval_dense", "dss_eval_mixed", "dss_eval_slide",
           "dss_chain_stride_geometry", "dss_plan_stride_geometry", "dss_eval_stride", "dss_chain_dilate_geometry",
           "dss_plan_dilate_geometry", "dss_eval_dilate", "dss_chain_backward_geometry",
           "dss_plan_backward_geometry", "dss_backward_dense", "dss_eval_dense_noalloc", "dss_frag", "dss_defrag",
           "dss_plan_set_timing", "dss_plan_timings", "dss_status_string", "dss_last_error", "dss_version")

_lib = None


def _torch_device_first():
    """With torch in the process there are two HIP runtimes: torch's own copy and
    the system one that libdss.so links.  If the system one brings the device up
    first, torch's then reports no device; bringing torch's up first (when torch
    is installed and sees a device) works in either use.  Nothing happens on a
    machine without a GPU."""
    try:
        import torch
    except ImportError:
        return
    if torch.cuda.is_available():
        torch.cuda.init()


def lib():
    """Load libdss.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise DssError(-1, "loading libdss.so", "%s does not exist; run __graft_entry__.build()" % LIB_PATH)
        _torch_device_first()
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
        L.dss_chain_geometry.argtypes = [P(Layer), I32, I32, I32, I32, I32, I32, I32, P(Geometry)]
        L.dss_chain_layer_geometry.argtypes = [P(Layer), I32, I32, I32, I32, I32, I32, I32, P(LayerGeometry)]
        L.dss_plan_create.argtypes = [P(Layer), I32, I32, I32, I32, P(VP)]
        L.dss_plan_destroy.argtypes = [VP]
        L.dss_plan_destroy.restype = None
        L.dss_plan_geometry.argtypes = [VP, I32, I32, I32, P(Geometry)]
        L.dss_plan_layer_geometry.argtypes = [VP, I32, I32, I32, I32, P(LayerGeometry)]
        L.dss_eval_dense.argtypes = [VP, VP, I32, I32, VP, VP, I64, VP]
        L.dss_eval_mixed.argtypes = [VP, VP, I32, I32, I32, VP, VP, I64, VP]
        L.dss_eval_slide.argtypes = [VP, VP, I32, I32, I32, I32, VP, VP, I64, VP]
        L.dss_chain_stride_geometry.argtypes = [P(Layer), I32, I32, I32, I32, I32, P(I64), P(ctypes.c_double)]
        L.dss_plan_stride_geometry.argtypes = [VP, I32, P(I64), P(ctypes.c_double)]
        L.dss_eval_stride.argtypes = [VP, VP, I32, I32, I64, I32, VP, VP, I64, VP]
        L.dss_chain_dilate_geometry.argtypes = [P(Layer), I32, I32, I32, I32, I32, I32, I32, P(I32), P(I32), P(I64),
                                                P(ctypes.c_double)]
        L.dss_plan_dilate_geometry.argtypes = [VP, I32, I32, I32, P(I32), P(I32), P(I64), P(ctypes.c_double)]
        L.dss_eval_dilate.argtypes = [VP, VP, I32, I32, I32, VP, VP, I64, VP]
        L.dss_chain_backward_geometry.argtypes = [P(Layer), I32, I32, I32, I32, I32, I32, P(I64), P(I64), P(I64),
                                                  P(ctypes.c_double)]
        L.dss_plan_backward_geometry.argtypes = [VP, I32, I32, I32, P(I64), P(I64), P(I64), P(ctypes.c_double)]
        L.dss_backward_dense.argtypes = [VP, VP, I32, I32, VP, VP, VP, VP, VP, I64, VP]
        L.dss_eval_dense_noalloc.argtypes = [VP, VP, I32, I32, VP, VP]
        L.dss_frag.argtypes = [I32, I32, I32, I32, I32, I32, I32, I32, VP, VP, VP]
        L.dss_defrag.argtypes = [I32, I32, I32, I32, I32, I32, I32, I32, VP, VP, VP]
        L.dss_plan_set_timing.argtypes = [VP, I32]
        L.dss_plan_timings.argtypes = [VP, P(LaunchRecord), I32, P(I32)]
        L.dss_status_string.argtypes = [I32]
        L.dss_status_string.restype = ctypes.c_char_p
        L.dss_last_error.argtypes = []
        L.dss_last_error.restype = ctypes.c_char_p
        L.dss_version.argtypes = []
        L.dss_version.restype = ctypes.c_char_p
        for name in ("dss_chain_geometry", "dss_chain_layer_geometry", "dss_plan_create", "dss_plan_geometry",
                     "dss_plan_layer_geometry", "dss_eval_dense", "dss_eval_mixed", "dss_eval_slide", "dss_frag",
                     "dss_defrag", "dss_plan_set_timing", "dss_plan_timings", "dss_plan_stride_geometry",
                     "dss_chain_stride_geometry", "dss_eval_stride", "dss_chain_dilate_geometry",
                     "dss_plan_dilate_geometry", "dss_eval_dilate", "dss_chain_backward_geometry",
                     "dss_plan_backward_geometry", "dss_backward_dense", "dss_eval_dense_noalloc"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status, what):
    if status != 0:
        raise DssError(status, what, lib().dss_last_error().decode())


class _LayerArray:
    """ctypes dss_layer array plus the binary32 weight copies it points into."""

    def __init__(self, layers):
        self.keep = []
        self.arr = (Layer * max(1, len(layers)))()
        for t, l in enumerate(layers):
            if l["kind"] == "conv":
                w = np.ascontiguousarray(l["weight"], dtype=np.float32)
                assert w.shape == (l["cout"], l["cin"], l["fh"], l["fw"])
                b = None if l.get("bias") is None else np.ascontiguousarray(l["bias"], dtype=np.float32)
                self.keep += [w, b]
                self.arr[t] = Layer(0, l["cin"], l["cout"], l["fh"], l["fw"], ACTS[l["act"]], 1, 1,
                                    w.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                    b.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if b is not None
                                    else ctypes.POINTER(ctypes.c_float)())
            else:
                self.arr[t] = Layer(1, 0, 0, 1, 1, 0, l["kh"], l["kw"], ctypes.POINTER(ctypes.c_float)(),
                                    ctypes.POINTER(ctypes.c_float)())
        self.n = len(layers)


def chain_geometry(layers, ndim, in_channels, H, W, dtype="f32", ell=0):
    la = _LayerArray(layers)
    g = Geometry()
    _check(lib().dss_chain_geometry(la.arr, la.n, ndim, in_channels, DTYPES[dtype], H, W, ell, ctypes.byref(g)),
           "dss_chain_geometry")
    return g.as_dict()


def chain_layer_geometry(layers, ndim, in_channels, H, W, j, ell=0):
    la = _LayerArray(layers)
    g = LayerGeometry()
    _check(lib().dss_chain_layer_geometry(la.arr, la.n, ndim, in_channels, H, W, ell, j, ctypes.byref(g)),
           "dss_chain_layer_geometry")
    return g.as_dict()


def chain_stride_geometry(layers, ndim, in_channels, count, dtype="f32"):
    """(workspace bytes, conv flops) of the patch-by-patch baseline on `count` windows (host only)."""
    la = _LayerArray(layers)
    ws = ctypes.c_int64()
    fl = ctypes.c_double()
    _check(lib().dss_chain_stride_geometry(la.arr, la.n, ndim, in_channels, DTYPES[dtype], count, ctypes.byref(ws),
                                           ctypes.byref(fl)), "dss_chain_stride_geometry")
    return ws.value, fl.value


def chain_dilate_geometry(layers, ndim, in_channels, H, W, j, dtype="f32"):
    """(V_h, V_w, workspace bytes, conv flops) of the dilated evaluation after layer j (host only)."""
    la = _LayerArray(layers)
    vh, vw, ws, fl = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64(), ctypes.c_double()
    _check(lib().dss_chain_dilate_geometry(la.arr, la.n, ndim, in_channels, DTYPES[dtype], H, W, j, ctypes.byref(vh),
                                           ctypes.byref(vw), ctypes.byref(ws), ctypes.byref(fl)),
           "dss_chain_dilate_geometry")
    return vh.value, vw.value, ws.value, fl.value


def chain_backward_geometry(layers, ndim, in_channels, H, W, with_signal_grad=True):
    """(workspace bytes, weight-gradient floats, bias-gradient floats, flops) of the backward pass (host only)."""
    la = _LayerArray(layers)
    ws, wf, bf, fl = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_double()
    _check(lib().dss_chain_backward_geometry(la.arr, la.n, ndim, in_channels, H, W, 1 if with_signal_grad else 0,
                                             ctypes.byref(ws), ctypes.byref(wf), ctypes.byref(bf), ctypes.byref(fl)),
           "dss_chain_backward_geometry")
    return ws.value, wf.value, bf.value, fl.value


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _check_buffer(t, what, dtype, numel=None, min_numel=None, device=None):
    """Raises ValueError unless t is a contiguous CUDA tensor of `dtype` (a torch
    dtype, or an element size in bytes) with exactly `numel` (or at least
    `min_numel`) elements, on `device` if given.  The C ABI takes no sizes for
    these buffers, so a wrong one would mean out-of-bounds device accesses."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError("%s must be a contiguous CUDA tensor" % what)
    if isinstance(dtype, int):
        if t.element_size() != dtype or t.is_complex():
            raise ValueError("%s must have %d-byte elements (got %s)" % (what, dtype, t.dtype))
    elif t.dtype != dtype:
        raise ValueError("%s must be %s (got %s)" % (what, dtype, t.dtype))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, the signal on %s" % (what, t.device, device))
    if numel is not None and t.numel() != numel:
        raise ValueError("%s has %d elements, %d expected" % (what, t.numel(), numel))
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError("%s has %d elements, at least %d needed" % (what, t.numel(), min_numel))


def _workspace_args(ws, device):
    """(pointer, bytes) of a caller workspace, or (NULL, 0): the plan's own."""
    if ws is None:
        return ctypes.c_void_p(None), 0
    import torch
    if not isinstance(ws, torch.Tensor) or not ws.is_cuda or not ws.is_contiguous() or ws.device != device:
        raise ValueError("workspace must be a contiguous CUDA tensor on the signal's device")
    return _ptr(ws), ws.numel() * ws.element_size()


class Plan:
    """A dss plan on the current device."""

    def __init__(self, layers, ndim, in_channels, dtype="f32"):
        self.layers = layers
        self.ndim = ndim
        self.in_channels = in_channels
        self.dtype = dtype
        la = _LayerArray(layers)
        h = ctypes.c_void_p()
        _check(lib().dss_plan_create(la.arr, la.n, ndim, in_channels, DTYPES[dtype], ctypes.byref(h)),
               "dss_plan_create")
        self.handle = h

    @classmethod
    def from_workload(cls, wl):
        return cls(wl.layers, wl.ndim, wl.x.shape[0], wl.dtype)

    def close(self):
        if getattr(self, "handle", None):
            lib().dss_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def geometry(self, H, W, ell=0):
        g = Geometry()
        _check(lib().dss_plan_geometry(self.handle, H, W, ell, ctypes.byref(g)), "dss_plan_geometry")
        return g.as_dict()

    def layer_geometry(self, H, W, j, ell=0):
        g = LayerGeometry()
        _check(lib().dss_plan_layer_geometry(self.handle, H, W, ell, j, ctypes.byref(g)), "dss_plan_layer_geometry")
        return g.as_dict()

    def workspace(self, H, W, device=None, ell=0):
        """A new device workspace (uint8 tensor) large enough for dss_eval_dense /
        dss_eval_mixed on an H x W signal at mixed level ell.  Calls that pass no
        workspace use the plan's own one inside the library instead."""
        import torch
        need = self.geometry(H, W, ell)["workspace_bytes"]
        return torch.empty(max(need, 256), dtype=torch.uint8, device=device or "cuda")

    def _check_signal(self, signal):
        import torch
        want = torch.float32 if self.dtype == "f32" else torch.bfloat16
        if not signal.is_cuda or signal.dtype != want or not signal.is_contiguous() or signal.dim() != 3:
            raise ValueError("signal must be a contiguous CUDA %s tensor [C][H][W]" % want)
        if signal.shape[0] != self.in_channels:
            raise ValueError("signal has %d channels, plan expects %d" % (signal.shape[0], self.in_channels))

    def eval_dense(self, signal, out=None, workspace=None, stream=None):
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        g = self.geometry(H, W)
        if out is None:
            out = torch.empty((g["out_c"], g["out_h"], g["out_w"]), dtype=torch.float32, device=signal.device)
        _check_buffer(out, "out", torch.float32, g["out_c"] * g["out_h"] * g["out_w"], device=signal.device)
        wp, wb = _workspace_args(workspace, signal.device)
        _check(lib().dss_eval_dense(self.handle, _ptr(signal), H, W, _ptr(out), wp, wb, _stream(stream)),
               "dss_eval_dense")
        return out

    def eval_dense_noalloc(self, signal, out, stream=None):
        """dss_eval_dense_noalloc: the dense evaluation in the library's fixed
        scratch array (no device allocation, `out` must be given)."""
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        g = self.geometry(H, W)
        _check_buffer(out, "out", torch.float32, g["out_c"] * g["out_h"] * g["out_w"], device=signal.device)
        _check(lib().dss_eval_dense_noalloc(self.handle, _ptr(signal), H, W, _ptr(out), _stream(stream)),
               "dss_eval_dense_noalloc")
        return out

    def eval_mixed(self, signal, ell, out=None, workspace=None, stream=None):
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        g = self.geometry(H, W, ell)
        if out is None:
            out = torch.empty((g["out_c"], g["out_h"], g["out_w"]), dtype=torch.float32, device=signal.device)
        _check_buffer(out, "out", torch.float32, g["out_c"] * g["out_h"] * g["out_w"], device=signal.device)
        wp, wb = _workspace_args(workspace, signal.device)
        _check(lib().dss_eval_mixed(self.handle, _ptr(signal), H, W, ell, _ptr(out), wp, wb, _stream(stream)),
               "dss_eval_mixed")
        return out

    def eval_slide(self, signal, j, out=None, workspace=None, stream=None, ell=0):
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        lg = self.layer_geometry(H, W, j, ell)
        if out is None:
            out = torch.empty((lg["F"], lg["channels"], lg["U_h"], lg["U_w"]), dtype=torch.float32,
                              device=signal.device)
        _check_buffer(out, "out", torch.float32, lg["F"] * lg["channels"] * lg["U_h"] * lg["U_w"],
                      device=signal.device)
        wp, wb = _workspace_args(workspace, signal.device)
        _check(lib().dss_eval_slide(self.handle, _ptr(signal), H, W, ell, j, _ptr(out), wp, wb, _stream(stream)),
               "dss_eval_slide")
        return out

    def dilate_geometry(self, H, W, j):
        """(V_h, V_w, workspace bytes, conv flops) of eval_dilate after layer j."""
        vh, vw, ws, fl = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64(), ctypes.c_double()
        _check(lib().dss_plan_dilate_geometry(self.handle, H, W, j, ctypes.byref(vh), ctypes.byref(vw),
                                              ctypes.byref(ws), ctypes.byref(fl)), "dss_plan_dilate_geometry")
        return vh.value, vw.value, ws.value, fl.value

    def eval_dilate(self, signal, j=None, out=None, workspace=None, stream=None):
        """EvalDilate_j (default j = L, the dense output) as planar binary32 [C_j][V_h][V_w]."""
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        n_chain = self.geometry(H, W)["n_chain"]
        j = n_chain if j is None else j
        vh, vw, _, _ = self.dilate_geometry(H, W, j)
        C = self.in_channels if j == 0 else self.layer_geometry(H, W, j)["channels"]
        if out is None:
            out = torch.empty((C, vh, vw), dtype=torch.float32, device=signal.device)
        _check_buffer(out, "out", torch.float32, C * vh * vw, device=signal.device)
        wp, wb = _workspace_args(workspace, signal.device)
        _check(lib().dss_eval_dilate(self.handle, _ptr(signal), H, W, j, _ptr(out), wp, wb, _stream(stream)),
               "dss_eval_dilate")
        return out

    def backward_geometry(self, H, W, with_signal_grad=True):
        """(workspace bytes, weight-gradient floats, bias-gradient floats, flops) of backward()."""
        ws, wf, bf, fl = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_double()
        _check(lib().dss_plan_backward_geometry(self.handle, H, W, 1 if with_signal_grad else 0, ctypes.byref(ws),
                                                ctypes.byref(wf), ctypes.byref(bf), ctypes.byref(fl)),
               "dss_plan_backward_geometry")
        return ws.value, wf.value, bf.value, fl.value

    def backward(self, signal, grad_out, with_signal_grad=True, grad_weight=None, grad_bias=None, workspace=None,
                 stream=None):
        """Gradients of sum(grad_out * eval_dense(signal)).  Returns (flat weight
        gradients, flat bias gradients, signal gradient or None) as CUDA tensors;
        `split_grads` cuts the flat ones per convolution."""
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        _, wf, bf, _ = self.backward_geometry(H, W, with_signal_grad)
        g = self.geometry(H, W)
        dev = signal.device
        if grad_weight is None:
            grad_weight = torch.empty(max(wf, 1), dtype=torch.float32, device=dev)
        if grad_bias is None:
            grad_bias = torch.empty(max(bf, 1), dtype=torch.float32, device=dev)
        gx = torch.empty_like(signal) if with_signal_grad else None
        _check_buffer(grad_out, "grad_out", torch.float32, g["out_c"] * g["out_h"] * g["out_w"], device=dev)
        _check_buffer(grad_weight, "grad_weight", torch.float32, min_numel=wf, device=dev)
        _check_buffer(grad_bias, "grad_bias", torch.float32, min_numel=bf, device=dev)
        wp, wb = _workspace_args(workspace, dev)
        _check(lib().dss_backward_dense(self.handle, _ptr(signal), H, W, _ptr(grad_out), _ptr(grad_weight),
                                        _ptr(grad_bias), _ptr(gx) if gx is not None else None, wp, wb,
                                        _stream(stream)), "dss_backward_dense")
        return grad_weight, grad_bias, gx

    def split_grads(self, grad_weight, grad_bias):
        """Per-convolution views [cout][cin][fh][fw] and [cout] of the flat gradients."""
        ws, bs, ow, ob = [], [], 0, 0
        for l in self.layers:
            if l["kind"] != "conv":
                continue
            n = l["cout"] * l["cin"] * l["fh"] * l["fw"]
            ws.append(grad_weight[ow:ow + n].view(l["cout"], l["cin"], l["fh"], l["fw"]))
            bs.append(grad_bias[ob:ob + l["cout"]])
            ow += n
            ob += l["cout"]
        return ws, bs

    def stride_geometry(self, count):
        """(workspace bytes, conv flops) of eval_stride on a batch of `count` windows."""
        ws = ctypes.c_int64()
        fl = ctypes.c_double()
        _check(lib().dss_plan_stride_geometry(self.handle, count, ctypes.byref(ws), ctypes.byref(fl)),
               "dss_plan_stride_geometry")
        return ws.value, fl.value

    def eval_stride(self, signal, first, count, out=None, workspace=None, stream=None):
        """Patch-by-patch baseline on windows first..first+count-1 (row-major);
        writes those positions of `out` ([out_c][H-B_h+1][W-B_w+1], allocated if None)."""
        import torch
        self._check_signal(signal)
        _, H, W = signal.shape
        g = self.geometry(H, W)
        if out is None:
            out = torch.zeros((g["out_c"], g["out_h"], g["out_w"]), dtype=torch.float32, device=signal.device)
        _check_buffer(out, "out", torch.float32, g["out_c"] * g["out_h"] * g["out_w"], device=signal.device)
        wp, wb = _workspace_args(workspace, signal.device)
        _check(lib().dss_eval_stride(self.handle, _ptr(signal), H, W, first, count, _ptr(out), wp, wb,
                                     _stream(stream)), "dss_eval_stride")
        return out

    def set_timing(self, on=True):
        _check(lib().dss_plan_set_timing(self.handle, 1 if on else 0), "dss_plan_set_timing")

    def timings(self):
        n = ctypes.c_int32()
        _check(lib().dss_plan_timings(self.handle, None, 0, ctypes.byref(n)), "dss_plan_timings")
        recs = (LaunchRecord * max(1, n.value))()
        _check(lib().dss_plan_timings(self.handle, recs, n.value, ctypes.byref(n)), "dss_plan_timings")
        return [{"kernel": r.kernel.decode(), "layer": r.chain_layer, "ms": r.ms, "flops": r.flops,
                 "bytes": r.bytes, "tile_mode": r.tile_mode} for r in recs[: n.value]]


def frag(x, k_h, k_w, S_h, S_w, out=None, stream=None):
    """dss_frag on a CUDA tensor [S_h*S_w][C][H][W] of 4- or 2-byte elements."""
    import torch
    if not isinstance(x, torch.Tensor) or x.dim() != 4 or x.element_size() not in (2, 4):
        raise ValueError("x must be a 4-D tensor [S_h*S_w][C][H][W] of 2- or 4-byte elements")
    S, C, H, W = x.shape
    if S != S_h * S_w:
        raise ValueError("x holds %d fragments, S_h * S_w = %d" % (S, S_h * S_w))
    _check_buffer(x, "x", x.element_size())
    dt = DSS_BF16 if x.element_size() == 2 else DSS_F32
    if out is None:
        out = torch.empty((k_h * S_h * k_w * S_w, C, H // k_h, W // k_w), dtype=x.dtype, device=x.device)
    # extents that k does not divide are the library's DSS_E_SHAPE, before any access
    if k_h > 0 and k_w > 0 and H % k_h == 0 and W % k_w == 0:
        _check_buffer(out, "out", x.element_size(), S * C * H * W, device=x.device)
    _check(lib().dss_frag(k_h, k_w, S_h, S_w, C, H, W, dt, _ptr(x), _ptr(out), _stream(stream)), "dss_frag")
    return out


def defrag(x, k_h, k_w, S_h, S_w, out=None, stream=None):
    """dss_defrag on a CUDA tensor [(k_h*S_h)*(k_w*S_w)][C][H][W]."""
    import torch
    if not isinstance(x, torch.Tensor) or x.dim() != 4 or x.element_size() not in (2, 4):
        raise ValueError("x must be a 4-D tensor [(k_h*S_h)*(k_w*S_w)][C][H][W] of 2- or 4-byte elements")
    F, C, H, W = x.shape
    if F != k_h * S_h * k_w * S_w:
        raise ValueError("x holds %d fragments, (k_h * S_h) * (k_w * S_w) = %d" % (F, k_h * S_h * k_w * S_w))
    _check_buffer(x, "x", x.element_size())
    dt = DSS_BF16 if x.element_size() == 2 else DSS_F32
    if out is None:
        out = torch.empty((S_h * S_w, C, H * k_h, W * k_w), dtype=x.dtype, device=x.device)
    _check_buffer(out, "out", x.element_size(), F * C * H * W, device=x.device)
    _check(lib().dss_defrag(k_h, k_w, S_h, S_w, C, H, W, dt, _ptr(x), _ptr(out), _stream(stream)), "dss_defrag")
    return out
