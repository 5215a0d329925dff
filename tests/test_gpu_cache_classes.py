"""Cache classes of the gathers: a plan of more than 2^18 nodes marks the columns outside the
hottest 65,536 (bit 31 of its sorted copy's columns), and an SpMM whose operand exceeds the
256 MiB memory-side cache reads the marked rows with non-temporal loads.  Results must not
depend on either.  A sparse graph of 2^18 + 7 nodes with 64 hub rows (56 of about 800 entries,
one wavefront each, and 8 of about 12,000 split into parts of the plan's 1024-entry chunk) keeps
the oracle fast
while an F = 256 operand (256 MiB + 7 KiB) takes the class path of the plain SpMM
(spmm_dual_kernel<64, 4, *, true>) and of the fused junction (spmm_xw_kernel<64, true>).
The aggregation is the one of Sec. 1 and Sec. 2.1; every row is checked against the oracle
within 1e-5 sum |a||x| (F = 256: the class path; F = 128, a 128 MiB operand: the plain path)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from graphgen import dense
from graphgen.csr import Graph, csr_from_pairs, normalised_values
from test_gpu_parity import assert_spmm_close, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _hub_graph():
    n = (1 << 18) + 7
    gen = np.random.Generator(np.random.Philox(key=np.array([31, 7], dtype=np.uint64)))
    a, b = gen.integers(0, n, 3 * n), gen.integers(0, n, 3 * n)
    hubs = gen.choice(n, 64, replace=False)
    ha = np.repeat(hubs, [800] * 56 + [12000] * 8)      # long rows, and rows split into parts
    hb = gen.integers(0, n, ha.size)
    src, dst = np.concatenate([a, ha]), np.concatenate([b, hb])
    keep = src != dst
    src, dst = src[keep], dst[keep]
    rows = np.concatenate([src, dst, np.arange(n)])
    cols = np.concatenate([dst, src, np.arange(n)])
    rowptr, col = csr_from_pairs(n, rows, cols)
    return Graph(n=n, rowptr=rowptr, col=col, val=normalised_values(rowptr, col), meta={"kind": "hubs"})


@pytest.fixture(scope="module")
def hub(dg, device):
    g = _hub_graph()
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=8, walk_len=4)
    yield g, plan
    plan.destroy()


def test_large_plan_marks_cold_columns(dg, device, hub):
    g, plan = hub
    info = plan.info()
    assert info["cold_marked"] == 1
    # 2.1M entries: parts of 1024 entries; the 8 longest rows are split, the other hubs not
    assert info["dense_chunk"] == 1024 and info["n_split_rows"] == 8
    small = dg.Plan(*to_dev(g.__class__(n=4096, rowptr=np.arange(4097, dtype=np.int32),
                                        col=np.arange(4096, dtype=np.int32),
                                        val=np.ones(4096, dtype=np.float32)), device),
                    seed=0, walks_per_node=2, walk_len=2)
    assert small.info()["cold_marked"] == 0
    small.destroy()


@pytest.mark.parametrize("F", [256, 128])
def test_spmm_every_row_with_and_without_classes(dg, device, hub, F):
    g, plan = hub
    X = dense.features_normal(g.n, F, seed=F, stream_id=61)
    Y = torch.full((g.n, F), float("nan"), dtype=torch.float32, device=device)
    dg.spmm(plan, torch.from_numpy(X).to(device), Y)
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y.cpu().numpy(), Yr, B, what=f"hub graph F={F}")


def test_fused_junction_on_the_class_path(dg, device, hub):
    """dualgcn_spmm_update with H = NULL runs the fused kernel whatever the route; with
    classes it must still equal the two calls bit for bit."""
    g, plan = hub
    X = torch.from_numpy(dense.features_normal(g.n, 256, seed=3, stream_id=62)).to(device)
    W = torch.from_numpy(dense.glorot(256, 64, seed=4)).to(device)
    T = torch.full((g.n, 64), float("nan"), dtype=torch.float32, device=device)
    st = dg.lib().dualgcn_spmm_update(plan.handle, X.data_ptr(), W.data_ptr(), T.data_ptr(), None,
                                      256, 64, dg.RELU, None)
    assert st == 0
    T_two = dg.update(dg.spmm(plan, X, relu=True, out_bf16=True), W)
    assert torch.equal(T, T_two)
    assert not dg.spmm_update_route(plan, 256, 64)        # two workgroups per CU: the two calls
    assert torch.equal(dg.spmm_update(plan, X, W, relu=True), T_two)


def test_narrow_features_on_the_class_path(dg, device):
    """F = 32 (8-lane groups): an operand of 2^21 + 3 rows is 256 MiB + 384 bytes, so the plain
    SpMM and the fused junction (32 -> 32, fused route) read marked rows non-temporally."""
    n = (1 << 21) + 3
    gen = np.random.Generator(np.random.Philox(key=np.array([32, 1], dtype=np.uint64)))
    a, b = gen.integers(0, n, 2 * n), gen.integers(0, n, 2 * n)
    keep = a != b
    a, b = a[keep], b[keep]
    rows = np.concatenate([a, b, np.arange(n)])
    cols = np.concatenate([b, a, np.arange(n)])
    rowptr, col = csr_from_pairs(n, rows, cols)
    g = Graph(n=n, rowptr=rowptr, col=col, val=normalised_values(rowptr, col), meta={"kind": "sparse"})
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=4, walk_len=3)
    assert plan.info()["cold_marked"] == 1
    X = dense.features_normal(n, 32, seed=8, stream_id=63)
    Xd = torch.from_numpy(X).to(device)
    Y = torch.full((n, 32), float("nan"), dtype=torch.float32, device=device)
    dg.spmm(plan, Xd, Y)
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y.cpu().numpy(), Yr, B, what="F=32 class path")
    W = torch.from_numpy(dense.glorot(32, 32, seed=9)).to(device)
    assert dg.spmm_update_route(plan, 32, 32)
    T = dg.spmm_update(plan, Xd, W, relu=True)
    assert torch.equal(T, dg.update(dg.spmm(plan, Xd, relu=True, out_bf16=True), W))
    plan.destroy()
