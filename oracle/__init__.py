"""Oracle for dense signal scanning -- TEST INFRASTRUCTURE ONLY.

Used by `tests/`, `__graft_entry__.smoke()` and the CPU-baseline leg of
`bench.py`, never by the GPU library.  It shares no code with the GPU path.

* `eval_stride` runs the ordinary strided network on every requested window
  (EvalStride of Definition "processing chain", Sect. 4.2) in double precision,
  in plain C (`evalstride.c`).  Its results are what the main theorem
  (Sect. 4.3) says the dense GPU evaluation must equal.
* `receptive_field` finds B by brute force (smallest patch on which the strided
  network ends in one sample).
* `fragment` holds the literal vec-based Frag/Defrag and Stuff/Trim.
* `bf16` models bfloat16 storage of the intermediate activations on top of the
  dense (dilated) evaluation, for tighter checks of bfloat16 results.

Weights come in cross-correlation order ([cout][cin][fh][fw], tap t multiplies
input sample i+t), the order deep-learning frameworks use.  The paper writes the
convolution with a flipped filter (Sect. 3.3); `_paper_orientation` performs that
flip so that the C code can follow the paper's formula as written.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import fragment  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "evalstride.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ACT_CODES = {"none": 0, "relu": 1, "tanh": 2}


class _Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("cin", ctypes.c_int32), ("cout", ctypes.c_int32),
                ("fh", ctypes.c_int32), ("fw", ctypes.c_int32), ("act", ctypes.c_int32),
                ("kh", ctypes.c_int32), ("kw", ctypes.c_int32),
                ("w", ctypes.POINTER(ctypes.c_double)), ("b", ctypes.POINTER(ctypes.c_double))]


def build(force=True):
    """Compile evalstride.c into liboracle.so with gcc (plain -O2, OpenMP)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                           "-o", tmp, _SRC, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.orc_receptive_field.restype = ctypes.c_int
        lib.orc_receptive_field.argtypes = [ctypes.POINTER(_Layer), ctypes.c_int, ctypes.c_int,
                                            ctypes.c_int]
        lib.orc_eval_stride.restype = ctypes.c_int64
        lib.orc_eval_stride.argtypes = [
            ctypes.POINTER(_Layer), ctypes.c_int, ctypes.c_int,
            ctypes.POINTER(ctypes.c_double), ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.c_int, ctypes.c_int,
            ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64), ctypes.c_int64,
            ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), ctypes.c_int]
        lib.orc_threads.restype = ctypes.c_int
        lib.orc_threads.argtypes = [ctypes.c_int]
        _lib = lib
    return _lib


def _paper_orientation(w):
    """Cross-correlation taps -> the paper's flipped-filter taps (Sect. 3.3):
    paper tap mu (1-based) multiplies sample c+i-mu, i.e. 0-based tap c-1-t of the
    cross-correlation multiplies the same sample as paper tap t."""
    return np.ascontiguousarray(w[:, :, ::-1, ::-1], dtype=np.float64)


class _Chain:
    """Keeps the ctypes layer array and the double-precision weight copies alive."""

    def __init__(self, layers):
        self.keep = []
        arr = (_Layer * max(1, len(layers)))()
        for t, l in enumerate(layers):
            if l["kind"] == "conv":
                w = _paper_orientation(np.asarray(l["weight"]))
                b = np.ascontiguousarray(l["bias"], dtype=np.float64) if l.get("bias") is not None else None
                self.keep += [w, b]
                arr[t] = _Layer(0, l["cin"], l["cout"], l["fh"], l["fw"], ACT_CODES[l["act"]], 1, 1,
                                w.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                b.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if b is not None
                                else ctypes.POINTER(ctypes.c_double)())
            elif l["kind"] == "maxpool":
                arr[t] = _Layer(1, 0, 0, 1, 1, 0, l["kh"], l["kw"],
                                ctypes.POINTER(ctypes.c_double)(), ctypes.POINTER(ctypes.c_double)())
            else:
                raise ValueError(l["kind"])
        self.arr = arr
        self.n = len(layers)


def receptive_field(layers, smax=100000):
    """(B_h, B_w) by brute force."""
    lib = _load()
    ch = _Chain(layers)
    bh = lib.orc_receptive_field(ch.arr, ch.n, 0, smax)
    bw = lib.orc_receptive_field(ch.arr, ch.n, 1, smax)
    return bh, bw


def threads(n=0):
    return _load().orc_threads(n)


def eval_stride(layers, x, windows=None, upto=None, patch=None, threads=0, with_counts=False):
    """EvalStride on windows of x.

    x        [C][H][W] array (any float type; evaluated in float64)
    windows  None (every window) or a pair of int arrays (i, j) of top-left positions
    upto     number of layer descriptors to apply (default: all)
    patch    (ph, pw) patch extents (default: the receptive field)
    Returns  every window: float64 [Cout][H-B_h+1][W-B_w+1];
             listed windows: float64 [nwin][...] flattened per window.
    """
    lib = _load()
    ch = _Chain(layers)
    x = np.ascontiguousarray(x, dtype=np.float64)
    C, H, W = x.shape
    if patch is None:
        patch = receptive_field(layers)
    ph, pw = patch
    if ph < 0 or pw < 0:
        raise ValueError("the layer list has no receptive field")
    full = windows is None
    if full:
        oh, ow = H - ph + 1, W - pw + 1
        if oh <= 0 or ow <= 0:
            raise ValueError("signal smaller than the receptive field")
        ii, jj = np.meshgrid(np.arange(oh, dtype=np.int64), np.arange(ow, dtype=np.int64), indexing="ij")
        wi, wj = ii.reshape(-1).copy(), jj.reshape(-1).copy()
    else:
        wi = np.ascontiguousarray(windows[0], dtype=np.int64)
        wj = np.ascontiguousarray(windows[1], dtype=np.int64)
    upto = len(layers) if upto is None else upto
    nwin = len(wi)
    # the C side returns the per-window element count; size the buffer generously first
    cmax = max([C] + [l["cout"] for l in layers if l["kind"] == "conv"])
    cap = cmax * ph * pw
    out = np.empty((max(1, nwin), cap), dtype=np.float64)
    counts = np.zeros(max(1, upto), dtype=np.int64)
    n_el = lib.orc_eval_stride(ch.arr, ch.n, upto, x.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                               C, H, W, ph, pw,
                               wi.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                               wj.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), nwin,
                               out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                               counts.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), threads)
    if n_el < 0:
        raise ValueError("oracle rejected the request (ill-defined chain or window out of range)")
    # the C side packs n_el values per window contiguously
    res = out.reshape(-1)[: nwin * n_el].reshape(nwin, n_el).copy()
    if full and upto == len(layers):
        cout = n_el
        res = res.reshape(oh, ow, cout).transpose(2, 0, 1).copy()
    if with_counts:
        return res, counts[:upto].copy()
    return res


from . import mixed  # noqa: E402,F401  (needs eval_stride above)
