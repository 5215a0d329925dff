"""Pins of the oracle's training path (CPU only).

The backward products of a GCN layer follow from the chain rule applied to the
forward of Sec. 1; here they are checked against central finite differences of the
loss (which catch a wrong transpose, a dropped ReLU mask or a sign), the forward
and the transposed aggregation against dense brute force on tiny asymmetric
graphs, and the softmax cross-entropy against its closed form on equal logits.
"""
import math

import numpy as np
import pytest

import oracle
from graphgen import small


def _weighted(rows, seed):
    g = small.from_rows(rows)
    rs = np.random.default_rng(seed)
    g.val[:] = rs.uniform(-1.0, 1.0, g.col.size).astype(np.float32)
    return g


ROWS = [[1, 2, 5], [0], [0, 1, 2, 7], [], [3, 3, 6], [4], [0, 8, 9, 1], [2], [8], [9, 0], [], [10, 11, 0]]


def _dense(g):
    A = np.zeros((g.n, g.n))
    for r in range(g.n):
        for p in range(g.rowptr[r], g.rowptr[r + 1]):
            A[r, g.col[p]] += float(g.val[p])
    return A


def _loss(g, X, Ws, labels, scale):
    return oracle.gcn_train_grads(g, X, Ws, labels, scale)["loss"]


def test_transposed_aggregation_is_dense_transpose():
    g = _weighted(ROWS, 1)
    A = _dense(g)
    G = np.random.default_rng(2).standard_normal((g.n, 3))
    assert np.allclose(oracle.spmm_f64(oracle.transpose_csr(g), G), A.T @ G, rtol=0, atol=1e-12)
    assert np.allclose(oracle.spmm_f64(g, G), A @ G, rtol=0, atol=1e-12)


def test_forward_matches_dense_brute_force():
    g = _weighted(ROWS, 3)
    A = _dense(g)
    rs = np.random.default_rng(4)
    X = rs.standard_normal((g.n, 5))
    Ws = [rs.standard_normal((5, 4)), rs.standard_normal((4, 3))]
    R = oracle.gcn_train_grads(g, X, Ws, np.zeros(g.n, dtype=np.int32), 1.0)
    H1 = np.maximum(A @ (X @ Ws[0]), 0)
    Y = A @ (H1 @ Ws[1])
    assert np.allclose(R["H"][0], H1, atol=1e-12) and np.allclose(R["H"][1], Y, atol=1e-12)


def test_softmax_xent_equal_logits_closed_form():
    n, C, scale = 7, 5, 0.25
    labels = np.array([0, 4, -1, 2, 9, 1, 3], dtype=np.int32)     # -1 and 9: unlabeled
    loss, G = oracle.softmax_xent(np.full((n, C), 2.5), labels, scale)
    assert math.isclose(loss, scale * 5 * math.log(C), rel_tol=1e-14)
    want = np.full((n, C), scale / C)
    want[[2, 4]] = 0.0
    for r in (0, 1, 3, 5, 6):
        want[r, labels[r]] -= scale
    assert np.allclose(G, want, atol=1e-15)


def test_softmax_xent_gradient_by_finite_differences():
    rs = np.random.default_rng(5)
    Y = rs.standard_normal((6, 4)) * 3
    labels = np.array([1, -1, 3, 0, 2, 2], dtype=np.int32)
    loss, G = oracle.softmax_xent(Y, labels, 0.5)
    h = 1e-6
    for r in range(6):
        for c in range(4):
            Yp, Ym = Y.copy(), Y.copy()
            Yp[r, c] += h
            Ym[r, c] -= h
            fd = (oracle.softmax_xent(Yp, labels, 0.5)[0] - oracle.softmax_xent(Ym, labels, 0.5)[0]) / (2 * h)
            assert abs(fd - G[r, c]) < 1e-8
    assert np.allclose(G.sum(axis=1), 0.0, atol=1e-15)          # softmax minus one-hot


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_weight_gradients_by_finite_differences(seed):
    g = _weighted(ROWS, 10 + seed)
    rs = np.random.default_rng(20 + seed)
    X = rs.standard_normal((g.n, 5))
    Ws = [rs.standard_normal((5, 4)), rs.standard_normal((4, 3))]
    labels = rs.integers(-1, 3, g.n).astype(np.int32)
    scale = 1.0 / max(1, int((labels >= 0).sum()))
    R = oracle.gcn_train_grads(g, X, Ws, labels, scale)
    h = 1e-6
    checked = 0
    for li, W in enumerate(Ws):
        for i in range(W.shape[0]):
            for j in range(W.shape[1]):
                Wp = [w.copy() for w in Ws]
                Wm = [w.copy() for w in Ws]
                Wp[li][i, j] += h
                Wm[li][i, j] -= h
                Pp = oracle.gcn_train_grads(g, X, Wp, labels, scale)["P"][0]
                Pm = oracle.gcn_train_grads(g, X, Wm, labels, scale)["P"][0]
                if np.any(np.sign(Pp) != np.sign(Pm)):
                    continue                                     # a ReLU kink inside the step
                fd = (_loss(g, X, Wp, labels, scale) - _loss(g, X, Wm, labels, scale)) / (2 * h)
                assert abs(fd - R["dW"][li][i, j]) < 1e-7 * (1 + abs(fd)), (li, i, j)
                checked += 1
    assert checked >= 28                                         # of 32 entries


def test_three_layers_by_finite_differences():
    g = _weighted(ROWS, 40)
    rs = np.random.default_rng(41)
    X = rs.standard_normal((g.n, 4))
    Ws = [rs.standard_normal((4, 4)), rs.standard_normal((4, 3)), rs.standard_normal((3, 2))]
    labels = rs.integers(0, 2, g.n).astype(np.int32)
    R = oracle.gcn_train_grads(g, X, Ws, labels, 0.1)
    h = 1e-6
    i, j = 2, 1
    Wp = [w.copy() for w in Ws]
    Wm = [w.copy() for w in Ws]
    Wp[0][i, j] += h
    Wm[0][i, j] -= h
    fd = (_loss(g, X, Wp, labels, 0.1) - _loss(g, X, Wm, labels, 0.1)) / (2 * h)
    assert abs(fd - R["dW"][0][i, j]) < 1e-7 * (1 + abs(fd))


def test_weight_grad_and_backward_data_brute_force():
    rs = np.random.default_rng(7)
    X = rs.standard_normal((9, 4))
    G = rs.standard_normal((9, 3))
    W = rs.standard_normal((4, 3))
    M = rs.standard_normal((9, 4))
    dW, B = oracle.weight_grad(X, G)
    dX, BX = oracle.backward_data(G, W, M)
    for i in range(4):
        for j in range(3):
            s = sum(X[r, i] * G[r, j] for r in range(9))
            b = sum(abs(X[r, i] * G[r, j]) for r in range(9))
            assert math.isclose(dW[i, j], s, rel_tol=1e-12, abs_tol=1e-12)
            assert math.isclose(B[i, j], b, rel_tol=1e-12)
    for r in range(9):
        for i in range(4):
            s = sum(G[r, j] * W[i, j] for j in range(3)) if M[r, i] > 0 else 0.0
            assert math.isclose(dX[r, i], s, rel_tol=1e-12, abs_tol=1e-12)
    assert np.array_equal(oracle.backward_data(G, W)[0] != 0, np.ones((9, 4), dtype=bool))


def test_round_bf16_matches_torch_and_ties_go_even():
    import torch
    rs = np.random.default_rng(9)
    x = np.concatenate([rs.standard_normal(20000).astype(np.float32) * 10.0 ** rs.integers(-30, 30, 20000),
                        np.array([0.0, -0.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-40, -1e-40], np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).float().numpy().astype(np.float64)
    got = oracle.round_bf16(x)
    assert np.array_equal(got, want)
    # exact ties: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 and goes to the even 1
    assert oracle.round_bf16(np.float32(1 + 2 ** -8)) == 1.0
    assert oracle.round_bf16(np.float32(1 + 3 * 2 ** -8)) == 1 + 2 ** -6
    assert np.isnan(oracle.round_bf16(np.float32(np.nan)))


def test_bf16_chain_is_the_exact_chain_on_bf16_values():
    # inputs, weights and every intermediate representable in bfloat16: the declared
    # roundings change nothing, so both chains agree to float64 rounding
    g = small.from_rows([[0], [1], [2], [3]])                 # identity: A = I
    X = np.array([[1, 2], [0.5, -1], [-2, 0.25], [4, 1]], dtype=np.float32)
    Ws = [np.array([[1, 0], [0, 1]], np.float32), np.array([[1, -1], [2, 0.5]], np.float32)]
    labels = np.array([0, 1, -1, 1], np.int32)
    a = oracle.gcn_train_grads(g, X, Ws, labels, 1.0)
    b = oracle.gcn_train_grads(g, X, Ws, labels, 1.0, bf16=True)
    assert np.array_equal(a["H"][0], b["H"][0])
    # the aggregated gradients are rounded in the bf16 chain, not in the exact one
    assert np.allclose(a["dW"][1], b["dW"][1], rtol=2 ** -7, atol=1e-12)
    assert abs(a["loss"] - b["loss"]) < 1e-12
