"""A seeded sweep over many small random matrices and parameters, beyond the fixed cases of
the other parity tests: for each case the whole plan (S, K, the sums, K*, n_sparse, perm)
bit-exact against the oracle, the SpMM within 1e-5 sum |a||x| of it, and the fused layer
junction bit-identical to the two-call route.

The matrices come from one seeded generator: row lengths from a heavy-tailed law (empty
rows, duplicate columns, asymmetric patterns, hubs beyond one dense chunk in some cases),
random values of both signs.  The parameters: walks k in 1..9 (powers of two and others),
steps d in 1..9, alpha and beta rationals (and the adaptive alpha), every force mode, and
feature widths from 1 to 260 (the vector and the one-feature-per-lane paths).
"""
import numpy as np
import pytest
import torch

import oracle
from graphgen import dense
from graphgen.csr import Graph
from test_gpu_parity import assert_plan_matches, assert_spmm_close, to_dev

pytestmark = pytest.mark.gpu

CASES = 150


@pytest.fixture(scope="module")
def dg(device):
    import paper_2609_01983_amd as dg
    return dg


def _random_matrix(gen, n):
    """CSR with heavy-tailed row lengths; a few cases get one hub row of > 4096 entries."""
    lens = np.minimum(gen.pareto(1.3, n).astype(np.int64), 4 * n)
    lens[gen.random(n) < 0.1] = 0                       # empty rows
    if n > 50 and gen.random() < 0.25:
        lens[gen.integers(n)] = 4096 + int(gen.integers(1, 3000))   # a hub split into parts
    rowptr = np.zeros(n + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum(lens)
    nnz = int(rowptr[-1])
    col = gen.integers(0, n, nnz).astype(np.int32)      # duplicates and asymmetry included
    val = gen.uniform(-1.0, 1.0, nnz).astype(np.float32)
    return Graph(n=n, rowptr=rowptr.astype(np.int32), col=col, val=val, meta=dict(kind="random"))


def _case(i):
    gen = np.random.default_rng(1000 + i)
    n = int(gen.choice([1, 2, 7, 33, 64, 200, 513, 1500]))
    g = _random_matrix(gen, n)
    k = int(gen.choice([1, 2, 3, 4, 8, 9, 16]))
    d = int(gen.integers(1, 10))
    if gen.random() < 0.2:
        marker = oracle.ALPHA_ADAPTIVE if i % 2 else oracle.ALPHA_BALANCED
        alpha = (marker, int(gen.choice([4, 16, 1024])))
    else:
        q = int(gen.integers(1, 8))
        alpha = (int(gen.integers(0, q + 1)), q)
    c = int(gen.integers(1, 6))
    beta = (int(gen.integers(0, 3 * c)), c)
    force = int(gen.choice([0, 0, 0, 1, 2]))
    F = int(gen.choice([1, 3, 4, 16, 33, 64, 128, 260]))
    seed = int(gen.integers(0, 2**62))
    return g, k, d, alpha, beta, force, F, seed


@pytest.mark.parametrize("i", range(CASES))
def test_random_case(dg, device, i):
    g, k, d, alpha, beta, force, F, seed = _case(i)
    print(f"[sweep] case {i}: n={g.n} nnz={g.nnz} k={k} d={d} alpha={alpha} beta={beta} "
          f"force={force} F={F}", flush=True)
    plan = dg.Plan(*to_dev(g, device), seed=seed, walks_per_node=k, walk_len=d, alpha=alpha,
                   beta=beta, force_mode=force)
    assert_plan_matches(dg, plan, g, seed, k, d, alpha, beta, force)
    X = dense.features_normal(g.n, F, seed=i, stream_id=47)
    Y = dg.spmm(plan, torch.from_numpy(X).to(device)).cpu().numpy()
    Yr, B = oracle.spmm(g, X)
    assert_spmm_close(Y, Yr, B, what=f"case {i}")
    if F in (64, 128):
        Xd = torch.from_numpy(X).to(device)
        W = torch.from_numpy(dense.glorot(F, 32, seed=i)).to(device)
        T = dg.spmm_update(plan, Xd, W, relu=True)
        assert torch.equal(T, dg.update(dg.spmm(plan, Xd, relu=True, out_bf16=True), W))
    plan.destroy()
