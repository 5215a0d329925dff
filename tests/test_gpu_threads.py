"""Calls from several host threads at once.  Each thread builds plans of its own matrix and
runs the SpMM and the fused layer junction on its own stream, three times over; ctypes
releases the interpreter lock during every library call, so the calls overlap (the block
cache, the per-plan use records and the per-thread read-back buffers are shared or raced
for).  Every result must equal, bit for bit, the one a single thread computed beforehand."""
import threading

import pytest
import torch

from graphgen import configs, dense
from test_gpu_parity import TINY, to_dev

pytestmark = pytest.mark.gpu

GRAPHS = {
    "c1": lambda: configs.load_graph("c1"),
    "c2": lambda: configs.load_graph("c2"),
    "gnp257": TINY["gnp257"],
    "hub_star": TINY["hub_star"],
}
F_IN, F_OUT, REPS = 64, 32, 3


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _run(dg, device, g, X, W):
    plan = dg.Plan(*to_dev(g, device), seed=3, walks_per_node=8, walk_len=4)
    Xd, Wd = X.to(device), W.to(device)
    Y = dg.spmm(plan, Xd)
    T = dg.spmm_update(plan, Xd, Wd, relu=True)
    perm = plan.export()[0]
    torch.cuda.current_stream().synchronize()
    out = (Y.cpu(), T.cpu(), perm)
    plan.destroy()
    return out


def test_threads_share_the_library(dg, device):
    inputs = {}
    for i, (name, make) in enumerate(sorted(GRAPHS.items())):
        g = make()
        X = torch.from_numpy(dense.features_normal(g.n, F_IN, seed=i, stream_id=48))
        W = torch.from_numpy(dense.glorot(F_IN, F_OUT, seed=i))
        inputs[name] = (g, X, W)
    want = {name: _run(dg, device, *args) for name, args in inputs.items()}

    errors, got = [], {}

    def worker(name):
        try:
            stream = torch.cuda.Stream(device=device)       # default priority
            with torch.cuda.stream(stream):
                got[name] = [_run(dg, device, *inputs[name]) for _ in range(REPS)]
        except Exception as e:                               # reported by the main thread
            errors.append((name, repr(e)))

    threads = [threading.Thread(target=worker, args=(name,), daemon=True) for name in inputs]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    for name, runs in got.items():
        Y0, T0, p0 = want[name]
        for Y, T, p in runs:
            assert (p == p0).all(), name
            assert torch.equal(Y, Y0), name
            assert torch.equal(T, T0), name
