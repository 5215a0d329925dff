"""CPU oracle of the DualGCN aggregation path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The GPU library never calls it and shares no code with it.

Pieces and the passages they follow (DualGCN paper):

* walks and density -- Sec. 3.2, Theorem 1 and "Neighbor Density": anonymous
  random walks from every node; N_v = sum_i i P_i = S_v / k where S_v sums the
  distinct-node counts of the node's k walks (C part, ``oracle.c``).
* degree -- Sec. 3.2 "Node Degree": the row length read from the row pointers.
* hybrid metric -- Sec. 3.2: H_v = alpha N_v + (1 - alpha) D_v.  With
  alpha = p/q this is kept as the exact integer K_v = q k H_v = p S_v + (q-p) k D_v.
  The adaptive alpha (Sec. 3.2, "Time Complexity") is Var(N) / (Var(N) + Var(D)),
  rounded down to a multiple of 1/q; the balanced alpha sigma_D / (sigma_N + sigma_D)
  gives both terms of H the same spread.
* threshold and mode -- Sec. 3.3 Eq. (1): dense iff H_v >= tau with
  tau = mu_H + 0.5 sigma_H (population statistics over all nodes).  Evaluated
  exactly with Python integers: H >= mu + (b/c) sigma  <=>  c (n K - S1) >= b sqrt(V)
  with S1 = sum K, V = n sum K^2 - S1^2.
* sort -- Sec. 3.2 (proof of Theorem 2): nodes sorted by H ascending, ties by
  node id, then split into the sparse prefix and the dense suffix.
* SpMM -- Sec. 1 / Sec. 2.1 aggregation Y = A X, float64 (C part).
* GCN layer -- Sec. 1 update phase: Y = act(A (X W)), float64 (C part + numpy).

The whole-graph partition is exact and therefore unique; the SpMM and the GCN
layer return float64 values with a per-element magnitude bound.
"""
import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

FORCE_AUTO, FORCE_SPARSE, FORCE_DENSE = 0, 1, 2


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _build
            _build.build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        L.philox4x64_10.argtypes = [P, P, P]
        L.philox4x64_10.restype = None
        L.oracle_walk.argtypes = [P, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_uint32,
                                  ctypes.c_uint64, ctypes.c_uint32, P]
        L.oracle_walk.restype = ctypes.c_uint32
        L.oracle_density.argtypes = [P, P, ctypes.c_int32, ctypes.c_uint64, ctypes.c_uint32,
                                     ctypes.c_uint32, P, ctypes.c_int64, P]
        L.oracle_density.restype = None
        L.oracle_patterns.argtypes = [P, P, ctypes.c_int32, ctypes.c_uint64, ctypes.c_uint32,
                                      ctypes.c_uint32, P]
        L.oracle_patterns.restype = None
        L.oracle_spmm_rows.argtypes = [P, P, P, P, ctypes.c_int32, P, ctypes.c_int64, P, P]
        L.oracle_spmm_rows.restype = None
        L.oracle_spmm_rows_f64.argtypes = [P, P, P, P, ctypes.c_int32, P, ctypes.c_int64, P, P]
        L.oracle_spmm_rows_f64.restype = None
        L.oracle_xw_rows.argtypes = [P, P, ctypes.c_int32, ctypes.c_int32, P, ctypes.c_int64,
                                     P, P]
        L.oracle_xw_rows.restype = None
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _csr(g):
    rowptr = np.ascontiguousarray(g.rowptr, dtype=np.int32)
    col = np.ascontiguousarray(g.col, dtype=np.int32)
    val = np.ascontiguousarray(g.val, dtype=np.float32)
    return rowptr, col, val


# ------------------------------------------------------------------ random stream

def philox(counter, key):
    """One Philox-4x64-10 block: four 64-bit words for a 4-word counter and 2-word key."""
    c = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().philox4x64_10(_p(c), _p(k), _p(out))
    return out


# ------------------------------------------------------------------ walks (Sec. 3.2)

def walk(g, start, w, seed, steps):
    """Labels (length steps+1) of walk ``w`` from node ``start``."""
    rowptr, col, _ = _csr(g)
    out = np.zeros(steps + 1, dtype=np.uint8)
    u = lib().oracle_walk(_p(rowptr), _p(col), g.n, int(start), int(w), int(seed), int(steps),
                          _p(out))
    assert u == out.max()
    return out


def patterns(g, seed, k, steps):
    """uint8 [n, k, steps+1] anonymous walks of every node."""
    rowptr, col, _ = _csr(g)
    out = np.zeros((g.n, k, steps + 1), dtype=np.uint8)
    lib().oracle_patterns(_p(rowptr), _p(col), g.n, int(seed), int(k), int(steps), _p(out))
    return out


def density_sums(g, seed, k, steps, nodes=None):
    """uint32 S_v (sum of distinct-node counts over the k walks) for ``nodes`` (default all)."""
    rowptr, col, _ = _csr(g)
    if nodes is None:
        nodes = np.arange(g.n, dtype=np.int32)
    nodes = np.ascontiguousarray(nodes, dtype=np.int32)
    S = np.zeros(nodes.size, dtype=np.uint32)
    lib().oracle_density(_p(rowptr), _p(col), g.n, int(seed), int(k), int(steps), _p(nodes),
                         nodes.size, _p(S))
    return S


# ------------------------------------------------------------------ partition (Sec. 3.2, 3.3)

def degrees(g):
    """D_v: entries of row v, read from the row pointers."""
    return np.diff(np.asarray(g.rowptr, dtype=np.int64))


def hybrid_keys(S, D, k, alpha=(1, 2)):
    """K_v = q k H_v = p S_v + (q - p) k D_v for alpha = p/q, as uint64."""
    p, q = alpha
    K = np.asarray(S, dtype=np.uint64) * np.uint64(p) + \
        np.asarray(D, dtype=np.uint64) * np.uint64((q - p) * k)
    return K


ALPHA_ADAPTIVE = 0xFFFFFFFF   # alpha numerator that asks for the adaptive weight


def adaptive_alpha(S, D, k, q):
    """Adaptive alpha = p/q (Sec. 3.2, "Time Complexity and Overhead Analysis": alpha
    follows a variance analysis and defaults to 1/2; the paper states no formula).

    Reading: each metric gets its share of the total spread,
    alpha = Var(N) / (Var(N) + Var(D)) with N_v = S_v / k and population variances
    over all nodes, and 1/2 when neither metric varies.  Exact in integers: with
    V_X = n sum X^2 - (sum X)^2 (n^2 times the variance), Var(N) / Var(D) =
    V_S / (k^2 V_D), so p = floor(q V_S / (V_S + k^2 V_D)).
    """
    S = [int(x) for x in np.asarray(S).ravel()]
    D = [int(x) for x in np.asarray(D).ravel()]
    n = len(S)
    VS = n * sum(x * x for x in S) - sum(S) ** 2
    VD = n * sum(x * x for x in D) - sum(D) ** 2
    den = VS + k * k * VD
    return q // 2 if den == 0 else q * VS // den


ALPHA_BALANCED = 0xFFFFFFFE   # alpha numerator that asks for the balanced weight


def balanced_alpha(S, D, k, q):
    """Balanced alpha = p/q: the variance analysis of Sec. 3.2 ("Time Complexity and Overhead
    Analysis"; alpha defaults to 1/2, no formula given) read as balancing the two terms of
    H = alpha N + (1 - alpha) D, so that alpha sigma_N = (1 - alpha) sigma_D, i.e.
    alpha = sigma_D / (sigma_N + sigma_D) with N_v = S_v / k and population standard
    deviations, rounded down to a multiple of 1/q.  A metric that does not vary carries no
    information and gets no weight (alpha = 0 when N is constant, 1 when D is); 1/2 when
    neither varies.

    Taken step by step with exact fractions: the variances as Fractions, then the largest p
    (scanning down from q) with p sigma_N <= (q - p) sigma_D, compared through squares (both
    sides are non-negative)."""
    from fractions import Fraction
    S = np.asarray(S, dtype=np.int64).ravel()
    D = np.asarray(D, dtype=np.int64).ravel()
    n = int(S.size)

    def variance(values, scale):
        # population variance of values / scale: E[x^2] - E[x]^2 from exact integer sums
        s1 = int(values.sum())
        s2 = int((values * values).sum())
        return Fraction(s2, n * scale * scale) - Fraction(s1, n * scale) ** 2

    var_n = variance(S, k)
    var_d = variance(D, 1)
    if var_n == 0 and var_d == 0:
        return q // 2
    if var_n == 0:
        return 0
    if var_d == 0:
        return q
    for p in range(q, -1, -1):
        if p * p * var_n <= (q - p) * (q - p) * var_d:
            return p
    return 0


def moments(K):
    """(S1, S2) = (sum K, sum K^2) as exact Python integers."""
    values, counts = np.unique(np.asarray(K, dtype=np.uint64), return_counts=True)
    S1 = sum(int(v) * int(c) for v, c in zip(values, counts))
    S2 = sum(int(v) * int(v) * int(c) for v, c in zip(values, counts))
    return S1, S2


def is_dense(Kv, n, S1, S2, beta=(1, 2)):
    """Eq. (1): H_v >= mu_H + beta sigma_H, evaluated exactly in integers."""
    b, c = beta
    V = n * S2 - S1 * S1           # n^2 sigma^2 in K units
    lhs = c * (n * int(Kv) - S1)   # c n (K - mu)
    if lhs < 0:
        return False
    return lhs * lhs >= b * b * V


def threshold_key(n, S1, S2, beta=(1, 2)):
    """Least integer K with K >= mu + beta sigma (so dense iff K_v >= this)."""
    b, c = beta
    V = n * S2 - S1 * S1
    guess = int(math.floor((S1 + (b / c) * math.sqrt(V)) / n)) if n else 0
    K = max(guess, 0)
    while K > 0 and is_dense(K - 1, n, S1, S2, beta):
        K -= 1
    while not is_dense(K, n, S1, S2, beta):
        K += 1
    return K


def partition(g, seed, k, steps, alpha=(1, 2), beta=(1, 2), force=FORCE_AUTO, S=None):
    """The whole plan: S, K, K*, dense flags, perm (sorted by (K, v)) and n_sparse.

    alpha = (ALPHA_ADAPTIVE, q) takes the adaptive weight p/q, (ALPHA_BALANCED, q) the
    balanced one; the alpha used is returned under "alpha"."""
    if S is None:
        S = density_sums(g, seed, k, steps)
    D = degrees(g)
    if alpha[0] == ALPHA_ADAPTIVE:
        alpha = (adaptive_alpha(S, D, k, alpha[1]), alpha[1])
    elif alpha[0] == ALPHA_BALANCED:
        alpha = (balanced_alpha(S, D, k, alpha[1]), alpha[1])
    K = hybrid_keys(S, D, k, alpha)
    n = g.n
    S1, S2 = moments(K)
    kstar = threshold_key(n, S1, S2, beta)
    values = np.unique(K)
    dense_values = {int(v) for v in values if is_dense(int(v), n, S1, S2, beta)}
    dense = np.isin(K, np.array(sorted(dense_values), dtype=np.uint64))
    perm = np.lexsort((np.arange(n), K)).astype(np.int32)   # by K, then by node id
    if force == FORCE_SPARSE:
        n_sparse = n
    elif force == FORCE_DENSE:
        n_sparse = 0
    else:
        n_sparse = int(n - dense.sum())
    return dict(S=S, D=D, K=K, S1=S1, S2=S2, kstar=kstar, dense=dense, perm=perm,
                n_sparse=n_sparse, alpha=alpha)


# ------------------------------------------------------------------ SpMM (Sec. 1, 2.1)

def spmm(g, X, rows=None):
    """float64 (Y, B) for the listed rows (default all): Y = A X, B = |A| |X|."""
    rowptr, col, val = _csr(g)
    X = np.ascontiguousarray(X, dtype=np.float32)
    F = X.shape[1] if X.ndim == 2 else 1
    if rows is None:
        rows = np.arange(g.n, dtype=np.int32)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    Y = np.zeros((rows.size, F), dtype=np.float64)
    B = np.zeros((rows.size, F), dtype=np.float64)
    lib().oracle_spmm_rows(_p(rowptr), _p(col), _p(val), _p(X), F, _p(rows), rows.size,
                           _p(Y), _p(B))
    return Y, B


def xw(X, W, rows=None):
    """float64 (T, BT) for the listed rows: T = X W, BT = |X| |W|."""
    X = np.ascontiguousarray(X, dtype=np.float32)
    W = np.ascontiguousarray(W, dtype=np.float32)
    Fin, Fout = W.shape
    if rows is None:
        rows = np.arange(X.shape[0], dtype=np.int32)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    T = np.zeros((rows.size, Fout), dtype=np.float64)
    BT = np.zeros((rows.size, Fout), dtype=np.float64)
    lib().oracle_xw_rows(_p(X), _p(W), Fin, Fout, _p(rows), rows.size, _p(T), _p(BT))
    return T, BT


def _spmm_f64(g, Xc, slot, rows):
    rowptr, col, val = _csr(g)
    Xc = np.ascontiguousarray(Xc, dtype=np.float64)
    F = Xc.shape[1]
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    slot = np.ascontiguousarray(slot, dtype=np.int64)
    Y = np.zeros((rows.size, F), dtype=np.float64)
    lib().oracle_spmm_rows_f64(_p(rowptr), _p(col), _p(val), _p(Xc), F, _p(rows), rows.size,
                               _p(slot), _p(Y))
    return Y


def neighbours(g, rows):
    """Sorted distinct column ids referenced by the listed rows."""
    rp = np.asarray(g.rowptr, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    if rows.size == 0:
        return np.zeros(0, dtype=np.int32)
    parts = [np.asarray(g.col[rp[r]:rp[r + 1]]) for r in rows]
    return np.unique(np.concatenate(parts)).astype(np.int32)


def _absolute(g):
    from types import SimpleNamespace
    return SimpleNamespace(n=g.n, rowptr=g.rowptr, col=g.col, val=np.abs(np.asarray(g.val)))


def gcn_layer(g, X, W, relu=False, rows=None):
    """One GCN layer Y = act(A (X W)) in float64 on the listed rows, with its bound.

    Returns (Y, BY) where BY = |A| (|X| |W|) bounds the magnitude of every
    product term; ReLU does not change it (ReLU is 1-Lipschitz).
    """
    if rows is None:
        rows = np.arange(g.n, dtype=np.int32)
    rows = np.asarray(rows, dtype=np.int32)
    need = neighbours(g, rows)
    T, BT = xw(X, W, need)
    slot = np.full(g.n, -1, dtype=np.int64)
    slot[need] = np.arange(need.size)
    Y = _spmm_f64(g, T, slot, rows)
    BY = _spmm_f64(_absolute(g), BT, slot, rows)
    if relu:
        Y = np.maximum(Y, 0.0)
    return Y, BY


def gcn_forward_rows(g, X, weights, rows):
    """Two-layer (or deeper) forward  act(A (act(A (X W1)) W2))... on the listed output rows.

    ReLU after every layer but the last.  Returns (Y, bound) where ``bound`` is
    the end-to-end magnitude bound of the deviation budget used by the tests:
    for the last layer |A| ((|H| + bound_prev) |W|).
    """
    rows = np.asarray(rows, dtype=np.int32)
    # the set of nodes needed at every depth
    levels = [rows]
    for _ in range(len(weights) - 1):
        levels.append(neighbours(g, levels[-1]))
    H = None
    Hbound = None
    prev_nodes = None
    for li, W in enumerate(weights):
        out_nodes = levels[len(weights) - 1 - li]
        relu = li < len(weights) - 1
        if li == 0:
            Y, BY = gcn_layer(g, X, W, relu=relu, rows=out_nodes)
            H, Hbound = Y, BY
        else:
            slot_prev = np.full(g.n, -1, dtype=np.int64)
            slot_prev[prev_nodes] = np.arange(prev_nodes.size)
            need = neighbours(g, out_nodes)
            Hn = H[slot_prev[need]]
            Bn = Hbound[slot_prev[need]]
            Wd = np.asarray(W, dtype=np.float64)
            T = Hn @ Wd
            BT = (np.abs(Hn) + Bn) @ np.abs(Wd)
            slot = np.full(g.n, -1, dtype=np.int64)
            slot[need] = np.arange(need.size)
            Y = _spmm_f64(g, T, slot, out_nodes)
            BY = _spmm_f64(_absolute(g), BT, slot, out_nodes)
            if relu:
                Y = np.maximum(Y, 0.0)
            H, Hbound = Y, BY
        prev_nodes = out_nodes
    return H, Hbound


# ------------------------------------------------------------------ training (Sec. 1)
# The paper accelerates GCN training: each layer H = act(A (X W)) is followed, in the
# backward pass, by the products of the chain rule.  With G = dL/dH:
#   G_P = G * act'(P)        (P = A (X W); ReLU' is [P > 0])
#   G_T = A^T G_P            (the aggregation transposed)
#   dW  = X^T G_T
#   dX  = G_T W^T            (masked by the previous layer's ReLU')
# The loss is the mean softmax cross-entropy over the labeled rows.

def softmax_xent(Y, labels, scale):
    """(loss, G): loss = scale * sum over labeled rows of -log softmax(Y_v)[label_v] and
    G = dloss/dY = scale (softmax(Y_v) - e_label) on labeled rows, 0 elsewhere.
    Rows whose label is outside [0, C) are unlabeled.  float64."""
    Y = np.asarray(Y, dtype=np.float64)
    labels = np.asarray(labels).astype(np.int64)
    n, C = Y.shape
    m = Y.max(axis=1, keepdims=True)
    e = np.exp(Y - m)
    s = e.sum(axis=1, keepdims=True)
    P = e / s
    on = (labels >= 0) & (labels < C)
    rows = np.flatnonzero(on)
    G = np.zeros_like(Y)
    G[rows] = P[rows]
    G[rows, labels[rows]] -= 1.0
    G *= scale
    logp = Y[rows, labels[rows]] - m[rows, 0] - np.log(s[rows, 0])
    return float(-scale * logp.sum()), G


def transpose_csr(g):
    """The transposed matrix A^T as a CSR graph (entries of column c become row c, in
    row order of A)."""
    from types import SimpleNamespace
    rowptr, col, val = _csr(g)
    rows = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(rowptr.astype(np.int64)))
    order = np.argsort(col, kind="stable")
    tcol = rows[order].astype(np.int32)
    tval = np.asarray(val)[order]
    tptr = np.zeros(g.n + 1, dtype=np.int64)
    np.add.at(tptr, col.astype(np.int64) + 1, 1)
    return SimpleNamespace(n=g.n, rowptr=np.cumsum(tptr).astype(np.int32), col=tcol, val=tval)


def spmm_f64(g, X):
    """A X for a float64 X (every row), float64."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    return _spmm_f64(g, X, np.arange(g.n, dtype=np.int64), np.arange(g.n, dtype=np.int32))


def weight_grad(X, G):
    """(dW, B) = (X^T G, |X|^T |G|) in float64."""
    X = np.asarray(X, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    return X.T @ G, np.abs(X).T @ np.abs(G)


def backward_data(G, W, M=None):
    """(dX, B) = ((G W^T) * [M > 0], (|G| |W|^T) * [M > 0]) in float64; no mask if M is None."""
    G = np.asarray(G, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    dX = G @ W.T
    B = np.abs(G) @ np.abs(W).T
    if M is not None:
        keep = np.asarray(M, dtype=np.float64) > 0
        dX = dX * keep
        B = B * keep
    return dX, B


def round_bf16(a):
    """float64 array of the bfloat16 values nearest (ties to even) to the float32 rounding
    of `a`: the 16 high bits of the float32 pattern after adding 0x7FFF plus the lowest
    kept bit; NaN stays NaN."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isnan(f), np.nan, out)


def gcn_train_grads(g, X, weights, labels, scale, bf16=False):
    """Forward and backward of a GCN (ReLU after every layer but the last, softmax
    cross-entropy on the last) in float64.  Returns a dict with the loss, the weight
    gradients "dW" (one per layer) and the intermediates: per layer "T", "P", "H" of
    the forward and "GP", "GT" of the backward; "G" holds dL/dH of every layer.

    bf16=True applies the declared roundings of the matrix-core path and nothing else:
    both operands of every dense product to bfloat16, hidden activations and aggregated
    gradients stored as bfloat16, the last layer's output stored as float32; all other
    arithmetic stays float64."""
    X = np.asarray(X, dtype=np.float64)
    gt = transpose_csr(g)
    L = len(weights)
    r = round_bf16 if bf16 else (lambda a: a)
    Ws = [np.asarray(W, dtype=np.float64) for W in weights]
    inp, T, P, H = [X], [], [], []
    for li, W in enumerate(Ws):
        T.append(r(inp[-1]) @ r(W))
        P.append(spmm_f64(g, T[-1]))
        if li < L - 1:
            H.append(r(np.maximum(P[-1], 0.0)))
        else:
            H.append(P[-1].astype(np.float32).astype(np.float64) if bf16 else P[-1])
        inp.append(H[-1])
    loss, G_last = softmax_xent(H[-1], labels, scale)
    G = [None] * L
    G[L - 1] = G_last
    GP, GT, dW = [None] * L, [None] * L, [None] * L
    for li in range(L - 1, -1, -1):
        GP[li] = G[li] * (P[li] > 0) if li < L - 1 else G[li]
        GT[li] = r(spmm_f64(gt, GP[li]))
        dW[li] = r(inp[li]).T @ GT[li]
        if li > 0:
            G[li - 1] = GT[li] @ r(Ws[li]).T
    return dict(loss=loss, dW=dW, T=T, P=P, H=H, G=G, GP=GP, GT=GT)


# ------------------------------------------------------------------ aggregators (Sec. 2.1)
# The aggregation phase multiplies by a matrix built from the adjacency; the paper's
# general message-passing form admits other aggregators than the GCN normalisation.
# Values are defined from the row lengths d of the matrix as given (self-loops included
# when present), computed in float64 and rounded once to float32.
AGG_GCN, AGG_MEAN, AGG_SUM = 0, 1, 2


def aggregator_values(g, kind, eps=0.0):
    """float32 values for the structure of g: GCN 1/sqrt(d_r d_c), mean 1/d_r, sum 1
    (1 + eps on self-loop entries, the GIN form)."""
    rowptr = np.asarray(g.rowptr, dtype=np.int64)
    col = np.asarray(g.col, dtype=np.int64)
    d = np.diff(rowptr).astype(np.float64)
    rows = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(rowptr))
    if kind == AGG_GCN:
        v = 1.0 / np.sqrt(d[rows] * d[col])
    elif kind == AGG_MEAN:
        v = 1.0 / d[rows]
    elif kind == AGG_SUM:
        v = np.where(rows == col, 1.0 + float(np.float32(eps)), 1.0)
    else:
        raise ValueError(kind)
    return v.astype(np.float32)
