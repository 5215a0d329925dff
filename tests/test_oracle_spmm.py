"""Pins of the oracle's aggregation SpMM Y = A X and the GCN update (CPU only).

Pinned against brute-force dense products (numpy, separate code), scipy.sparse,
closed forms of special graphs and invariants of the normalised adjacency
D^-1/2 (A + I) D^-1/2 (DualGCN Sec. 1 and Sec. 2.1: aggregation is an SpMM of
the adjacency with the feature matrix; the update multiplies by W).
"""
import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from graphgen import small, dense


def _dense_matrix(g):
    A = np.zeros((g.n, g.n), dtype=np.float64)
    for i in range(g.n):
        for p in range(g.rowptr[i], g.rowptr[i + 1]):
            A[i, g.col[p]] += float(g.val[p])
    return A


def _x(n, f, seed=0):
    return dense.features_normal(n, f, seed=seed, stream_id=40)


@pytest.mark.parametrize("n,p,f", [(1, 0.0, 3), (17, 0.3, 5), (64, 0.1, 16), (50, 0.5, 1)])
def test_spmm_matches_dense_bruteforce(n, p, f):
    g = small.random_graph(n, p, seed=n)
    X = _x(n, f)
    Y, B = oracle.spmm(g, X)
    ref = _dense_matrix(g) @ X.astype(np.float64)
    absref = np.abs(_dense_matrix(g)) @ np.abs(X.astype(np.float64))
    assert np.allclose(Y, ref, rtol=0, atol=1e-12 * (1 + absref.max()))
    assert np.allclose(B, absref, rtol=1e-12, atol=0)


def test_spmm_matches_scipy_with_duplicates_and_empty_rows():
    g = small.from_rows([[0, 2, 2], [], [1, 3], [3, 0, 0, 0]])
    g.val = np.array([0.5, -1.25, 2.0, 3.0, -0.75, 1.5, 0.25, -2.0, 4.0], dtype=np.float32)
    X = _x(4, 7, seed=3)
    A = sp.csr_matrix((g.val.astype(np.float64), g.col, g.rowptr), shape=(4, 4))
    Y, B = oracle.spmm(g, X)
    assert np.allclose(Y, A @ X.astype(np.float64), rtol=0, atol=1e-12)
    assert np.all(Y[1] == 0) and np.all(B[1] == 0)


def test_spmm_scipy_random_larger():
    g = small.random_graph(300, 0.05, seed=5)
    X = _x(300, 33, seed=5)
    A = sp.csr_matrix((g.val.astype(np.float64), g.col, g.rowptr), shape=(300, 300))
    Y, _ = oracle.spmm(g, X)
    assert np.allclose(Y, A @ X.astype(np.float64), rtol=1e-13, atol=1e-13)


def test_edgeless_graph_is_identity():
    g = small.edgeless(10)
    X = _x(10, 4)
    Y, _ = oracle.spmm(g, X)
    assert np.array_equal(Y, X.astype(np.float64))


def test_cycle_averages_three_neighbours():
    n = 12
    g = small.cycle(n, self_loops=True, normalise=True)
    assert np.all(g.val == np.float32(1.0 / 3.0))
    X = _x(n, 6)
    Y, _ = oracle.spmm(g, X)
    Xd = X.astype(np.float64)
    third = float(np.float32(1.0 / 3.0))
    ref = third * (np.roll(Xd, 1, 0) + Xd + np.roll(Xd, -1, 0))
    assert np.allclose(Y, ref, rtol=0, atol=1e-14)


def test_complete_graph_rows_are_column_means():
    n = 9
    g = small.clique(n, self_loops=True, normalise=True)
    X = _x(n, 5)
    Y, _ = oracle.spmm(g, X)
    ref = float(np.float32(1.0 / n)) * X.astype(np.float64).sum(0)
    assert np.allclose(Y, np.broadcast_to(ref, Y.shape), rtol=0, atol=1e-14)


def test_normalised_adjacency_invariants():
    g = small.random_graph(80, 0.08, seed=12)
    d = np.diff(g.rowptr).astype(np.float64)
    s = np.sqrt(d)[:, None]
    Y, _ = oracle.spmm(g, s.astype(np.float32))
    # A sqrt(d) = sqrt(d): each value is rounded once to fp32 (and sqrt(d) too)
    assert np.allclose(Y, s, rtol=2e-7 * d.max(), atol=0)
    # symmetry <A X, Z> = <X, A Z> (values are symmetric bit for bit)
    X, Z = _x(80, 3, 1), _x(80, 3, 2)
    AX, _ = oracle.spmm(g, X)
    AZ, _ = oracle.spmm(g, Z)
    assert abs((AX * Z).sum() - (X * AZ).sum()) < 1e-10
    # linearity
    A2, _ = oracle.spmm(g, (2 * X + Z).astype(np.float32))
    assert np.allclose(A2, 2 * AX + AZ, atol=1e-6)


def test_row_sums_match_normalisation():
    g = small.random_graph(60, 0.1, seed=2)
    ones = np.ones((60, 1), dtype=np.float32)
    Y, _ = oracle.spmm(g, ones)
    d = np.diff(g.rowptr).astype(np.float64)
    ref = np.array([d[i] ** -0.5 * sum(d[j] ** -0.5 for j in g.col[g.rowptr[i]:g.rowptr[i + 1]])
                    for i in range(60)])
    assert np.allclose(Y[:, 0], ref, rtol=1e-6)


def test_bound_equals_result_for_nonnegative_inputs():
    g = small.random_graph(40, 0.2, seed=9)
    X = np.abs(_x(40, 4))
    Y, B = oracle.spmm(g, X)
    assert np.allclose(Y, B, rtol=1e-15, atol=0)


def test_row_subset_matches_full():
    g = small.random_graph(50, 0.2, seed=10)
    X = _x(50, 8)
    Y, B = oracle.spmm(g, X)
    rows = np.array([49, 3, 3, 0])
    Ys, Bs = oracle.spmm(g, X, rows)
    assert np.array_equal(Ys, Y[rows]) and np.array_equal(Bs, B[rows])


# ---------------------------------------------------------------- update phase

def test_xw_matches_numpy():
    X = _x(30, 20)
    W = dense.glorot(20, 7, seed=1)
    T, BT = oracle.xw(X, W)
    assert np.allclose(T, X.astype(np.float64) @ W.astype(np.float64), rtol=1e-13, atol=1e-13)
    assert np.allclose(BT, np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)), rtol=1e-13)


def test_gcn_layer_identity_weight_equals_spmm():
    g = small.random_graph(40, 0.15, seed=6)
    X = _x(40, 6)
    Y, BY = oracle.gcn_layer(g, X, np.eye(6, dtype=np.float32))
    Ys, Bs = oracle.spmm(g, X)
    assert np.allclose(Y, Ys, rtol=0, atol=1e-14)
    assert np.allclose(BY, Bs, rtol=1e-14)


def test_gcn_forward_matches_dense_two_layer():
    g = small.random_graph(45, 0.12, seed=7)
    X = _x(45, 12)
    W1 = dense.glorot(12, 8, seed=1)
    W2 = dense.glorot(8, 5, seed=2)
    A = _dense_matrix(g)
    H1 = np.maximum(A @ (X.astype(np.float64) @ W1.astype(np.float64)), 0)
    Y2 = A @ (H1 @ W2.astype(np.float64))
    rows = np.array([0, 5, 44, 17])
    Y, bound = oracle.gcn_forward_rows(g, X, [W1, W2], rows)
    assert np.allclose(Y, Y2[rows], rtol=1e-12, atol=1e-12)
    absA = np.abs(A)
    B1 = absA @ (np.abs(X.astype(np.float64)) @ np.abs(W1.astype(np.float64)))
    B2 = absA @ ((np.abs(H1) + B1) @ np.abs(W2.astype(np.float64)))
    assert np.allclose(bound, B2[rows], rtol=1e-12)
    # the layer-1 sample on its own
    Y1, BY1 = oracle.gcn_layer(g, X, W1, relu=True, rows=rows)
    assert np.allclose(Y1, H1[rows], rtol=1e-12, atol=1e-12)
    assert np.allclose(BY1, B1[rows], rtol=1e-12)
