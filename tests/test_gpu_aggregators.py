"""GPU parity of the aggregator values (GCN, mean, sum/GIN) and of the SpMM on them.

Values: float64 arithmetic rounded once to float32 on both sides; they may differ only
where the device square root is not correctly rounded, so the test allows one float32
ulp and reports how many values match exactly.  SpMM: the usual 1e-5 sum |a||x| bound.
"""
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


GRAPHS = {
    "star": lambda: small.star(300, self_loops=True),
    "gnp": lambda: small.random_graph(200, 0.05, seed=3),
    "rows": lambda: small.from_rows([[0, 1, 2], [1, 0], [2, 2, 0], [], [1], [5, 5, 5, 0]]),
    "c2": lambda: configs.load_graph("c2"),
}


def _dev(g, device):
    return (torch.from_numpy(np.ascontiguousarray(g.rowptr)).to(device),
            torch.from_numpy(np.ascontiguousarray(g.col)).to(device))


def _ulps(a, b):
    ai = a.view(np.int32).astype(np.int64)
    bi = b.view(np.int32).astype(np.int64)
    return np.abs(ai - bi)


@pytest.mark.parametrize("name", sorted(GRAPHS))
@pytest.mark.parametrize("kind,eps", [("gcn", 0.0), ("mean", 0.0), ("sum", 0.0), ("sum", 0.3)])
def test_aggregator_values(dg, device, name, kind, eps):
    g = GRAPHS[name]()
    rp, c = _dev(g, device)
    v = dg.aggregator_values(rp, c, kind, eps).cpu().numpy()
    ref = oracle.aggregator_values(g, {"gcn": oracle.AGG_GCN, "mean": oracle.AGG_MEAN,
                                       "sum": oracle.AGG_SUM}[kind], eps)
    finite = np.isfinite(ref)
    assert np.array_equal(np.isfinite(v), finite)
    assert _ulps(v[finite], ref[finite]).max(initial=0) <= 1
    if kind != "gcn":
        assert np.array_equal(v, ref)                 # one correctly rounded division


@pytest.mark.parametrize("kind", ["mean", "sum"])
def test_spmm_with_other_aggregators_c2(dg, device, kind):
    g = configs.load_graph("c2")
    w = configs.WORKLOADS["c2"]
    rp, c = _dev(g, device)
    val = dg.aggregator_values(rp, c, kind, 0.1)
    plan = dg.Plan(rp, c, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
    X = dense.features_normal(g.n, 64, seed=4)
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    gv = type(g)(n=g.n, rowptr=g.rowptr, col=g.col, val=val.cpu().numpy())
    Yr, B = oracle.spmm(gv, X)
    assert np.all(np.abs(Y - Yr) <= 1e-5 * B)


def test_aggregator_rejects_bad_csr(dg, device):
    g = small.random_graph(20, 0.2, seed=3)
    rp, c = _dev(g, device)
    c = c.clone()
    c[2] = 99
    with pytest.raises(dg.DualGCNError) as e:
        dg.aggregator_values(rp, c, "gcn")
    assert e.value.status == dg.ERR_BAD_CSR
