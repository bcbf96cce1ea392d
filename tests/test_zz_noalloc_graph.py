"""dss_eval_dense_noalloc under HIP graph capture: one evaluation captured into
a graph (no device allocation happens inside it) and replayed several times,
with the program's own eager work, a new input written into the captured
signal buffer and synchronizations between the replays; every replay must
equal the eager dss_eval_dense of the same input bit for bit."""
import numpy as np
import pytest

from paper_1508_06904_amd import dss, workloads as wl
from tests.gpu_helpers import log, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    dss.lib()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("name", ["c3_512", "c5_4k", "c2_1d_1m"])
def test_noalloc_graph_replays(name):
    import torch
    sizes = {"c3_512": dict(H=150, W=161, widths=(16, 32, 48, 64)),
             "c5_4k": dict(H=190, W=201, widths=(16, 16, 32, 32)), "c2_1d_1m": dict(W=30001)}
    inputs = [wl.make(name, seed=s, **sizes[name]) for s in range(3)]
    w = inputs[0]
    plan = dss.Plan.from_workload(w)
    H, W = w.x.shape[1:]
    g = plan.geometry(H, W)
    shape = (g["out_c"], g["out_h"], g["out_w"])
    eager = []
    for v in inputs:
        eager.append(plan.eval_dense(to_device(v.x, w.dtype), workspace=plan.workspace(H, W)))
    torch.cuda.synchronize()
    x = to_device(w.x, w.dtype).clone()
    out = torch.zeros(shape, device="cuda")
    plan.eval_dense_noalloc(x, out)          # first call on the device: symbol address, kernel attributes
    torch.cuda.synchronize()
    assert torch.equal(out, eager[0])
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan.eval_dense_noalloc(x, out)
    torch.cuda.synchronize()
    for rep in range(6):
        k = rep % len(inputs)
        x.copy_(to_device(inputs[k].x, w.dtype))
        out.fill_(-3.0)                       # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        log("  %s replay %d on input %d" % (name, rep, k))
        assert torch.equal(out, eager[k]), "replay %d differs from the eager evaluation" % rep
    assert np.isfinite(out.cpu().numpy()).all()
