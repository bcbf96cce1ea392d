"""bfloat16 storage model of the dense evaluation -- TEST INFRASTRUCTURE ONLY.

Only tests use this module; the GPU library never imports it.  It is not part of
the paper's method: it models the precision at which a bfloat16 evaluation keeps
its intermediate activations, so that GPU tests can check bfloat16 results more
tightly than against the exact evaluation alone.

`eval_dilate_bf16_storage(layers, x, fold)` is the oracle's dense evaluation in
the dilated fashion (Definition "evaldilate", `dilate.eval_dilate`, double
precision) with one change: the activated output of every convolution but the
last is first rounded to binary32 and then to the nearest bfloat16, ties to
even, before the next layer reads it.  The last convolution's output is kept
(a bfloat16 evaluation writes it in binary32), and with `fold` so is the output
of the convolution before it (a final 1x1 projection folded into that
convolution's epilogue reads its binary32 activations).  Max-pooling commutes
with the rounding (both are monotone), so it does not matter which of the two
comes first.  Input and weights are expected bfloat16-representable already.

Pins (tests/test_oracle_bf16.py): `round_bf16` against torch's CPU bfloat16
cast on random, halfway, subnormal and large values; a chain whose stored
values are all small integers (exact in bfloat16) equals `eval_dilate` bit for
bit; a single-convolution chain (nothing stored) equals `eval_dilate`; and the
model moves a chain with non-representable activations by about the size of
one bfloat16 rounding.
"""
from __future__ import annotations

import numpy as np

from .dilate import dilate_conv, dilate_max
from .mixed import chain_of, stride_products


def round_bf16(x):
    """Nearest bfloat16 of binary32(x), ties to even, returned as float64.
    Finite inputs only (the activations of the test chains)."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    # add just under half a bfloat16 unit, plus one if the kept part is odd, then cut
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def eval_dilate_bf16_storage(layers, x, fold=False):
    """Dense outputs [C_L][H - B_h + 1][W - B_w + 1] with bfloat16-stored activations."""
    ch = chain_of(layers)
    ks = stride_products(ch)
    convs = [j for j, e in enumerate(ch) if e["conv"] is not None]
    kept = {convs[-1]}
    if fold and len(convs) > 1:
        kept.add(convs[-2])
    t = np.asarray(x, dtype=np.float64)
    for j, e in enumerate(ch):
        if e["conv"] is not None:
            t = dilate_conv(t, e["conv"], ks[j])
            if j not in kept:
                t = round_bf16(t)
        t = dilate_max(t, e["k"][0], e["k"][1], ks[j])
    return t
