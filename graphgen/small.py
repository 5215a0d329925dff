"""Tiny named graphs for tests, as CSR with optional self-loops.

All of them are undirected and unweighted; values are filled with the GCN
normalisation when ``normalise`` is set (only meaningful with self-loops), and
with ones otherwise.
"""
import numpy as np

from .csr import Graph, csr_from_pairs, normalised_values


def _build(n, edges, self_loops, normalise, name):
    e = np.asarray(edges, dtype=np.int64).reshape(-1, 2)
    rows = [e[:, 0], e[:, 1]]
    cols = [e[:, 1], e[:, 0]]
    if self_loops:
        rows.append(np.arange(n))
        cols.append(np.arange(n))
    rowptr, col = csr_from_pairs(n, np.concatenate(rows), np.concatenate(cols))
    if normalise:
        val = normalised_values(rowptr, col)
    else:
        val = np.ones(col.size, dtype=np.float32)
    return Graph(n=n, rowptr=rowptr, col=col, val=val, meta=dict(kind=name))


def path(n, self_loops=False, normalise=False):
    return _build(n, [(i, i + 1) for i in range(n - 1)], self_loops, normalise, "path")


def cycle(n, self_loops=False, normalise=False):
    return _build(n, [(i, (i + 1) % n) for i in range(n)], self_loops, normalise, "cycle")


def star(leaves, self_loops=False, normalise=False):
    return _build(leaves + 1, [(0, i) for i in range(1, leaves + 1)], self_loops, normalise, "star")


def clique(n, self_loops=False, normalise=False):
    return _build(n, [(i, j) for i in range(n) for j in range(i + 1, n)], self_loops,
                  normalise, "clique")


def edgeless(n, self_loops=True, normalise=True):
    return _build(n, np.zeros((0, 2), dtype=np.int64), self_loops, normalise, "edgeless")


def random_graph(n, p, seed, self_loops=True, normalise=True):
    gen = np.random.Generator(np.random.Philox(key=np.array([seed, 99], dtype=np.uint64)))
    iu, ju = np.triu_indices(n, 1)
    hit = gen.random(iu.size) < p
    return _build(n, np.stack([iu[hit], ju[hit]], 1), self_loops, normalise, "gnp")


def from_rows(rows):
    """Arbitrary (possibly asymmetric, duplicated, empty-row) CSR from a list of column lists."""
    n = len(rows)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in r], dtype=np.int32)
    val = np.ones(col.size, dtype=np.float32)
    return Graph(n=n, rowptr=rowptr.astype(np.int32), col=col, val=val, meta=dict(kind="rows"))
