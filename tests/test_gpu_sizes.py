"""GPU parity at the full workload sizes, in the launch configuration the benchmark times.

* c4 (R-MAT n=2^21, 63M entries) and c5 (R-MAT n=2^22, 67M entries): the whole
  partition bit-exact against the oracle (every S_v, K_v, the sums, K*, n_sparse
  and the whole order), and the SpMM on sampled rows (random rows, the heaviest
  rows and the rows around the region boundary) within 1e-5 sum |a||x|;
* c5 two-layer GCN forward (256 -> 128 -> 64, bf16 matrix cores): layer 1 on sampled
  rows and the end-to-end output on a few rows, within the bf16 bound;
* c5 fused layer junction (the benchmark's layer-1 kernel): bit-identical to the two-call
  route on every row, and within the bf16 bound of the oracle on sampled rows.
"""
import time

import numpy as np
import pytest
import torch

import oracle
from graphgen import configs, dense
from test_gpu_parity import GCN_TOL, _sample_rows, assert_plan_matches, assert_spmm_close, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _log(msg):
    print(f"[sizes] {msg}", flush=True)


@pytest.mark.parametrize("cfg", ["c4", "c5"])
def test_full_partition_and_sampled_spmm(dg, device, cfg):
    w = configs.WORKLOADS[cfg]
    t0 = time.time()
    g = configs.load_graph(cfg)
    _log(f"{cfg}: n={g.n} nnz={g.nnz} inputs {time.time() - t0:.1f}s")
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps)
    t0 = time.time()
    ref = assert_plan_matches(dg, plan, g, 0, w.walks, w.steps)
    _log(f"{cfg}: partition bit-exact (oracle {time.time() - t0:.1f}s), "
         f"n_sparse={ref['n_sparse']} K*={ref['kstar']}")
    assert 0 < ref["n_sparse"] < g.n
    # 63-67M entries: dense rows are split into parts of the largest chunk, 4096 entries
    info = plan.info()
    assert info["dense_chunk"] == 4096
    rows = _sample_rows(g, ref["perm"], ref["n_sparse"], 4000, seed=11)
    for F in ([w.F] if cfg == "c4" else [128, 64]):
        if cfg == "c4":
            X = configs.load_features(cfg)
        else:
            X = dense.features_normal(g.n, F, seed=F, stream_id=31)
        Y = dg.spmm(plan, torch.from_numpy(X).to(device))
        Ys = Y[torch.from_numpy(rows).long().to(device)].cpu().numpy()
        del Y
        Yr, B = oracle.spmm(g, X, rows)
        assert_spmm_close(Ys, Yr, B, what=f"{cfg} F={F}")
        _log(f"{cfg}: SpMM F={F} ok on {rows.size} rows")
    plan.destroy()


def test_c5_gcn_forward_sampled(dg, device):
    w = configs.WORKLOADS["c5"]
    g = configs.load_graph("c5")
    X = configs.load_features("c5")
    W1, W2 = configs.load_weights("c5")
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps)
    Xd = torch.from_numpy(X).to(device)
    H1 = dg.gcn_layer(plan, Xd, torch.from_numpy(W1).to(device), relu=True)
    del Xd
    Y2 = dg.gcn_layer(plan, H1, torch.from_numpy(W2).to(device))
    perm = plan.export()[0]
    gen = np.random.default_rng(5)
    rows1 = np.unique(np.concatenate([gen.choice(g.n, 1500, replace=False), perm[-4:]])).astype(np.int32)
    idx1 = torch.from_numpy(rows1).long().to(device)
    H1s = H1[idx1].cpu().numpy()
    t0 = time.time()
    Hr, BH = oracle.gcn_layer(g, X, W1, relu=True, rows=rows1)
    assert_spmm_close(H1s, Hr, BH, tol=GCN_TOL, what="c5 layer 1")
    _log(f"c5: layer 1 ok on {rows1.size} rows (oracle {time.time() - t0:.1f}s)")
    rows2 = np.sort(gen.choice(g.n, 12, replace=False)).astype(np.int32)
    Y2s = Y2[torch.from_numpy(rows2).long().to(device)].cpu().numpy()
    t0 = time.time()
    Yr, bound = oracle.gcn_forward_rows(g, X, [W1, W2], rows2)
    assert_spmm_close(Y2s, Yr, bound, tol=GCN_TOL, what="c5 two layers")
    _log(f"c5: two-layer output ok on {rows2.size} rows (oracle {time.time() - t0:.1f}s)")
    plan.destroy()


def test_c5_fused_junction_sampled(dg, device):
    """The bench's fused layer junction at full size: T2 = bf16(relu(A T1)) bf16(W2) bit for bit
    against the two-call route on every row, and against the oracle's float64 layer 1 on
    sampled rows: |T2 - H W2| <= 2e-2 ((|H| + B_H) |W2|), which covers layer 1's bf16 bound
    (1e-2 B_H), the bf16 rounding of H and W2 and the float32 accumulation."""
    w = configs.WORKLOADS["c5"]
    g = configs.load_graph("c5")
    X = configs.load_features("c5")
    W1, W2 = configs.load_weights("c5")
    plan = dg.Plan(*to_dev(g, device), seed=0, walks_per_node=w.walks, walk_len=w.steps)
    W2d = torch.from_numpy(W2).to(device)
    Xd = torch.from_numpy(X).to(device)
    T1 = dg.update(Xd, torch.from_numpy(W1).to(device))
    del Xd
    # the library's route: the fused kernel at the benchmark's shape (2 GiB operand, four
    # workgroups per CU); the two calls where one workgroup fills a CU's LDS
    assert dg.spmm_update_route(plan, 128, 64)
    assert not dg.spmm_update_route(plan, 256, 128)
    T2 = dg.spmm_update(plan, T1, W2d, relu=True)
    T2_two = dg.update(dg.spmm(plan, T1, relu=True, out_bf16=True), W2d)
    assert torch.equal(T2, T2_two), "fused and two-call results differ at full size"
    _log("c5: fused junction bit-identical to the two calls on every row")
    del T2_two, T1
    perm = plan.export()[0]
    gen = np.random.default_rng(17)
    rows = np.unique(np.concatenate([gen.choice(g.n, 1000, replace=False), perm[-6:]])).astype(np.int32)
    T2s = T2[torch.from_numpy(rows).long().to(device)].cpu().numpy().astype(np.float64)
    t0 = time.time()
    H, BH = oracle.gcn_layer(g, X, W1, relu=True, rows=rows)
    W2a = np.abs(W2.astype(np.float64))
    ref = H @ W2.astype(np.float64)
    bound = (np.abs(H) + BH) @ W2a
    err = np.abs(T2s - ref)
    bad = ~(err <= 2e-2 * bound)
    assert not bad.any(), f"{bad.sum()} outside; worst ratio {np.max(err / np.maximum(bound, 1e-300))}"
    _log(f"c5: fused junction ok on {rows.size} rows (oracle {time.time() - t0:.1f}s)")
    plan.destroy()
