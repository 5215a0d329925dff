"""Saved plans: a plan rebuilt from its saved density sums equals the original (perm, S,
K, threshold, sums, schedule sizes) and its SpMM is bit-identical; a buffer that does not
belong to the matrix is refused."""
import numpy as np
import pytest
import torch

import oracle
from graphgen import configs, dense, small

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _dev(g, device):
    return (torch.from_numpy(np.ascontiguousarray(g.rowptr)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.col)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.val)).to(device))


def _same_plan(dg, a, b):
    for x, y in zip(a.export(), b.export()):
        assert np.array_equal(x, y)
    assert a.info() == b.info()


@pytest.mark.parametrize("name,alpha", [("c1", (1, 2)), ("c2", (1, 2)), ("c2", (0xFFFFFFFF, 1024)),
                                        ("star", (1, 3))])
def test_save_load_roundtrip(dg, device, name, alpha):
    if name == "star":
        g = small.star(5000, self_loops=True, normalise=True)
        k, d = 8, 4
    else:
        g = configs.load_graph(name)
        w = configs.WORKLOADS[name]
        k, d = w.walks, w.steps
    rp, c, v = _dev(g, device)
    plan = dg.Plan(rp, c, v, seed=3, walks_per_node=k, walk_len=d, alpha=alpha)
    blob = plan.save()
    assert len(blob) == 80 + 4 * g.n
    loaded = dg.Plan.load(rp, c, v, blob)
    _same_plan(dg, plan, loaded)
    ref = oracle.partition(g, 3, k, d, alpha)
    assert np.array_equal(loaded.export()[0], ref["perm"])
    X = torch.from_numpy(dense.features_normal(g.n, 64, seed=1)).to(device)
    assert torch.equal(dg.spmm(plan, X), dg.spmm(loaded, X))


def test_load_with_other_values_keeps_the_partition(dg, device):
    g = configs.load_graph("c2")
    w = configs.WORKLOADS["c2"]
    rp, c, v = _dev(g, device)
    plan = dg.Plan(rp, c, v, seed=0, walks_per_node=w.walks, walk_len=w.steps)
    mean = dg.aggregator_values(rp, c, "mean")
    loaded = dg.Plan.load(rp, c, mean, plan.save())
    assert np.array_equal(plan.export()[0], loaded.export()[0])
    X = dense.features_normal(g.n, 32, seed=2)
    Y = dg.spmm(loaded, torch.from_numpy(X).to(device)).cpu().numpy()
    gm = type(g)(n=g.n, rowptr=g.rowptr, col=g.col, val=mean.cpu().numpy())
    Yr, B = oracle.spmm(gm, X)
    assert np.all(np.abs(Y - Yr) <= 1e-5 * B)


def test_load_refuses_foreign_buffers(dg, device):
    g = small.random_graph(300, 0.03, seed=5)
    rp, c, v = _dev(g, device)
    plan = dg.Plan(rp, c, v, seed=1, walks_per_node=8, walk_len=4)
    blob = plan.save()
    # same sizes, one column changed: the checksum differs
    c2 = c.clone()
    c2[7] = (c2[7] + 1) % g.n
    with pytest.raises(dg.DualGCNError) as e:
        dg.Plan.load(rp, c2, v, blob)
    assert e.value.status == dg.ERR_INVALID_ARG
    for bad in (blob[:-4], b"X" + blob[1:], blob + b"\0"):
        with pytest.raises(dg.DualGCNError) as e:
            dg.Plan.load(rp, c, v, bad)
        assert e.value.status == dg.ERR_INVALID_ARG
