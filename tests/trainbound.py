"""Element-wise error bounds of a two-layer GCN training step against the oracle's exact
float64 chain (oracle.gcn_train_grads without the declared roundings).

The per-stage budgets: one bfloat16 matrix-core product 1e-2 of its |operand| product (two
nearest-even roundings of unit roundoff 2^-8 and float32 sums), one float32 aggregation 1e-5
of |A||operand|, one bfloat16 store 2^-8 of the stored magnitude, the softmax Jacobian half
the largest logit error, and the whole term where a ReLU decision lies within the error of
its input.  They hold whatever the signs, so over the n-row sums of dW they are loose; they
catch a dropped term, a wrong mask or a transposed operand element by element.  Used by the
GPU tests and by __graft_entry__.smoke().
"""
import numpy as np

import oracle

R_MFMA = 1e-2        # one bf16 matrix-core product (two roundings and float32 sums)
R_SPMM = 1e-5        # one float32 aggregation
R_STORE = 2.0 ** -8  # one bfloat16 store (nearest-even: unit roundoff 2^-8, 8 significand bits)


def loss_bound(Y, labels, scale):
    """scale * sum over labeled rows of |terms| of the cross-entropy (the loss's own scale)."""
    Y = np.asarray(Y, dtype=np.float64)
    C = Y.shape[1]
    on = np.flatnonzero((labels >= 0) & (labels < C))
    m = np.abs(Y).max(axis=1)
    return scale * float((np.abs(Y[on, labels[on]]) + m[on] + np.log(C) + 1.0).sum())


def two_layer_bounds(g, X, Ws, labels, scale, ref):
    """Bounds of the loss and of dW1, dW2 for the step X -> T1 = X W1 -> H1 = bf16(relu(A T1))
    -> T2 = H1 W2 -> Y2 = A T2 -> softmax cross-entropy -> dT2 = bf16(A G2) -> dW2 = H1^T dT2,
    dH1 = (dT2 W2^T) [P1 > 0] -> dT1 = bf16(A dH1) -> dW1 = X^T dT1; ref is
    oracle.gcn_train_grads(g, X, Ws, labels, scale) (exact chain)."""
    W1, W2 = Ws
    C = W2.shape[1]
    ga = type(g)(n=g.n, rowptr=g.rowptr, col=g.col, val=np.abs(g.val))
    agg = lambda M: oracle.spmm_f64(ga, M)            # |A| M (= |A|^T M: symmetric)
    aX, aW1, aW2 = (np.abs(a.astype(np.float64)) for a in (X, W1, W2))
    E_T1 = R_MFMA * aX @ aW1
    E_P1 = agg(E_T1) + R_SPMM * agg(aX @ aW1)
    H1r = ref["H"][0]
    E_H1 = E_P1 + R_STORE * (np.abs(H1r) + E_P1)
    aH1 = np.abs(H1r) + E_H1
    E_T2 = E_H1 @ aW2 + R_MFMA * aH1 @ aW2
    E_Y2 = agg(E_T2) + R_SPMM * agg(aH1 @ aW2)
    on = (labels >= 0) & (labels < C)
    rowE = E_Y2.max(axis=1)
    E_G2 = np.where(on[:, None], scale * (0.5 * rowE[:, None] + 1e-6), 0.0)
    E_loss = scale * float((2 * rowE[on]).sum()) + 1e-5 * loss_bound(ref["H"][1], labels, scale)
    G2r = ref["G"][1]
    dT2r = ref["GT"][1]
    E_dT2 = agg(E_G2) + R_SPMM * agg(np.abs(G2r)) + R_STORE * (np.abs(dT2r) + agg(E_G2))
    adT2 = np.abs(dT2r) + E_dT2
    E_dW2 = E_H1.T @ adT2 + np.abs(H1r).T @ E_dT2 + R_MFMA * aH1.T @ adT2
    P1r = ref["P"][0]
    ambiguous = np.abs(P1r) <= E_P1
    keep = (P1r > 0) & ~ambiguous
    full = adT2 @ aW2.T
    E_dH1 = np.where(keep, E_dT2 @ aW2.T + R_MFMA * full, 0.0) + np.where(ambiguous, full * (1 + R_MFMA), 0.0)
    dT1r = ref["GT"][0]
    dH1r = ref["GP"][0]
    E_dT1 = agg(E_dH1) + R_SPMM * agg(np.abs(dH1r)) + R_STORE * (np.abs(dT1r) + agg(E_dH1))
    E_dW1 = aX.T @ E_dT1 + R_MFMA * aX.T @ (np.abs(dT1r) + E_dT1)
    return E_loss, [E_dW1, E_dW2]


def outside(got, want, bound):
    """Number of elements with |got - want| > bound, and the first such index (or None)."""
    err = np.abs(np.asarray(got, dtype=np.float64) - want)
    bad = ~(err <= bound)
    return int(bad.sum()), (tuple(np.argwhere(bad)[0]) if bad.any() else None)
