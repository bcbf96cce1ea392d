"""Pins for the bfloat16 storage model of the oracle (no GPU).

`oracle.bf16` evaluates a chain densely (the oracle's dilated evaluation, fp64)
with every stored activation rounded to bfloat16.  Its rounding is pinned to
torch's CPU bfloat16 cast (a library routine, round to nearest even); the model
is pinned to the exact evaluation where rounding changes nothing (integer
activations, a chain that stores nothing) and shown to move a chain with
ordinary activations by about one bfloat16 rounding."""
import numpy as np
import pytest

import oracle
from oracle import bf16 as ob
from oracle import dilate
from paper_1508_06904_amd import workloads as wl


def _torch_bf16(x):
    import torch
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(7)
    vals = [rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
            rng.uniform(-1, 1, 20000)]
    # exact halfway cases: the low 16 bits 0x8000 with the kept part even and odd
    hi = rng.integers(0, 0x7F7F, 4000).astype(np.uint32) << 16
    vals.append((hi | 0x8000).view(np.float32))
    vals.append(((hi | 0x10000) | 0x8000).view(np.float32))
    # just below / above halfway, subnormals, the largest finite bfloat16 range
    vals.append(((hi | 0x7FFF)).view(np.float32))
    vals.append(((hi | 0x8001)).view(np.float32))
    vals.append(rng.uniform(-1e-39, 1e-39, 2000).astype(np.float32))
    vals.append(rng.uniform(1e38, 3.3e38, 2000).astype(np.float32) * rng.choice([-1, 1], 2000))
    x = np.concatenate([np.asarray(v, dtype=np.float32) for v in vals])
    np.testing.assert_array_equal(ob.round_bf16(x), _torch_bf16(x))
    # and it is a rounding: idempotent, within half a unit (2^-8 relative)
    r = ob.round_bf16(x)
    np.testing.assert_array_equal(ob.round_bf16(r), r)
    n = np.abs(x) > 1e-37
    assert np.all(np.abs(r[n] - x[n].astype(np.float64)) <= np.abs(x[n]) * 2.0 ** -8)


def test_integer_chain_equals_exact_evaluation():
    """Stored activations that bfloat16 holds exactly (small integers) leave the
    model equal to the exact evaluation bit for bit."""
    arch = [("conv", 2, 4, 2, 2, "relu"), ("pool", 2, 2), ("conv", 4, 3, 2, 2, "relu"), ("pool", 2, 1),
            ("conv", 3, 2, 1, 2, "none")]
    w = wl.custom(arch, 2, 40, 37, seed=3, dtype="bf16", weight_kind="int", value_kind="int")
    # the two stored (pooled) activations are exact in bfloat16, by torch's cast;
    # max-pooling commutes with the monotone rounding, so that is enough
    for upto in (1, 2):
        h = dilate.eval_dilate(w.layers, w.x, upto=upto)
        assert np.all(h == np.round(h)) and np.array_equal(_torch_bf16(h), h)
    np.testing.assert_array_equal(ob.eval_dilate_bf16_storage(w.layers, w.x), dilate.eval_dilate(w.layers, w.x))


def test_single_convolution_stores_nothing():
    arch = [("conv", 3, 5, 3, 2, "tanh")]
    w = wl.custom(arch, 3, 21, 19, seed=5, dtype="bf16")
    np.testing.assert_array_equal(ob.eval_dilate_bf16_storage(w.layers, w.x), dilate.eval_dilate(w.layers, w.x))


@pytest.mark.parametrize("fold", [False, True])
def test_rounding_moves_output_by_about_one_unit(fold):
    """Ordinary activations: the model differs from the exact evaluation (so
    the rounding is applied), by about the relative size of one bfloat16
    rounding per stored layer; with `fold` the activation before the last
    convolution is kept, which changes the result too."""
    arch = [("conv", 3, 8, 3, 3, "tanh"), ("pool", 2, 2), ("conv", 8, 8, 2, 2, "relu"), ("conv", 8, 2, 1, 1, "none")]
    w = wl.custom(arch, 3, 30, 28, seed=9, dtype="bf16")
    exact = dilate.eval_dilate(w.layers, w.x)
    got = ob.eval_dilate_bf16_storage(w.layers, w.x, fold=fold)
    d = np.abs(got - exact).max() / np.abs(exact).max()
    assert 1e-5 < d < 3e-2, d
    other = ob.eval_dilate_bf16_storage(w.layers, w.x, fold=not fold)
    assert np.abs(other - got).max() > 0


def test_model_is_the_dense_evaluation():
    """On a chain with integer data (every stored value exact in bfloat16) the
    dense model agrees window by window with EvalStride, the oracle's per-window
    strided evaluation (Theorem "processing chain")."""
    arch = [("conv", 2, 3, 2, 2, "relu"), ("pool", 2, 2), ("conv", 3, 1, 2, 2, "none")]
    w = wl.custom(arch, 2, 23, 25, seed=11, dtype="bf16", weight_kind="int", value_kind="int")
    np.testing.assert_array_equal(ob.eval_dilate_bf16_storage(w.layers, w.x), oracle.eval_stride(w.layers, w.x))
