"""Pins of the oracle's aggregator values (CPU only): closed forms on regular graphs and
stars, and the row sums each normalisation fixes."""
import numpy as np
import pytest

import oracle
from graphgen import small


def test_gcn_values_on_a_star_closed_form():
    L = 9
    g = small.star(L, self_loops=True)
    v = oracle.aggregator_values(g, oracle.AGG_GCN)
    # hub: degree L + 1; leaves: degree 2
    rows = np.repeat(np.arange(g.n), np.diff(g.rowptr))
    for e in range(g.col.size):
        r, c = rows[e], g.col[e]
        dr = L + 1 if r == 0 else 2
        dc = L + 1 if c == 0 else 2
        assert v[e] == np.float32(1.0 / np.sqrt(dr * dc))
    assert v[(rows == 0) & (g.col == 0)][0] == np.float32(1.0 / (L + 1))


def test_gcn_values_regular_graph_rows_sum_to_one():
    g = small.cycle(30, self_loops=True)           # every degree 3
    v = oracle.aggregator_values(g, oracle.AGG_GCN)
    assert np.all(v == np.float32(1.0 / 3.0))
    Y, _ = oracle.spmm(type(g)(n=g.n, rowptr=g.rowptr, col=g.col, val=v), np.ones((g.n, 1), np.float32))
    assert np.allclose(Y, 1.0, atol=1e-6)


def test_mean_rows_sum_to_one():
    g = small.random_graph(50, 0.1, seed=2)
    v = oracle.aggregator_values(g, oracle.AGG_MEAN)
    sums = np.add.reduceat(v.astype(np.float64), g.rowptr[:-1])
    assert np.allclose(sums, 1.0, atol=1e-6)
    d = np.diff(g.rowptr)
    rows = np.repeat(np.arange(g.n), d)
    assert np.all(v == (1.0 / d[rows]).astype(np.float32))


@pytest.mark.parametrize("eps", [0.0, 0.25, -0.5])
def test_sum_is_adjacency_plus_weighted_identity(eps):
    g = small.from_rows([[0, 1, 2], [1, 0], [2, 2, 0], [], [1]])   # a repeated self-loop in row 2
    v = oracle.aggregator_values(g, oracle.AGG_SUM, eps)
    rows = np.repeat(np.arange(g.n), np.diff(g.rowptr))
    loops = rows == g.col
    assert loops.sum() == 4
    assert np.all(v[loops] == np.float32(1.0 + eps)) and np.all(v[~loops] == 1.0)
    # A X with these values: (1 + eps) x_v per self-loop entry plus the neighbours
    X = np.arange(5, dtype=np.float32)[:, None] + 1
    Y, _ = oracle.spmm(type(g)(n=g.n, rowptr=g.rowptr, col=g.col, val=v), X)
    assert np.isclose(Y[2, 0], 2 * (1 + eps) * 3 + 1)
