"""CSR assembly for the normalised GCN adjacency D^-1/2 (A + I) D^-1/2.

The aggregation operand of a GCN layer is the self-looped adjacency scaled on
both sides by the inverse square root of its degrees (the standard GCN
propagation matrix; the paper multiplies the adjacency by the feature matrix in
its aggregation phase, Sec. 1 and Sec. 2.1).  Degrees are taken in float64 and
each value is rounded once to float32.
"""
from dataclasses import dataclass, field
import hashlib

import numpy as np


@dataclass
class Graph:
    n: int
    rowptr: np.ndarray          # int32 [n+1]
    col: np.ndarray             # int32 [nnz], sorted within each row
    val: np.ndarray             # float32 [nnz]
    meta: dict = field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr.astype(np.int64))

    def max_degree(self) -> int:
        return int(self.degrees().max()) if self.n else 0

    def sha256(self) -> str:
        h = hashlib.sha256()
        for a in (self.rowptr, self.col, self.val):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


def normalised_values(rowptr: np.ndarray, col: np.ndarray) -> np.ndarray:
    """val_ij = fp32(1 / sqrt(d_i * d_j)) with d = row length of A + I (float64)."""
    deg = np.diff(rowptr.astype(np.int64)).astype(np.float64)
    rows = np.repeat(np.arange(len(deg), dtype=np.int64), np.diff(rowptr.astype(np.int64)))
    prod = deg[rows] * deg[col.astype(np.int64)]
    return (1.0 / np.sqrt(prod)).astype(np.float32)


def csr_from_pairs(n: int, rows: np.ndarray, cols: np.ndarray) -> tuple:
    """Sort (row, col) pairs into CSR order; duplicate pairs are kept."""
    key = rows.astype(np.int64)
    key *= np.int64(n)
    key += cols
    key.sort()
    starts = np.arange(n + 1, dtype=np.int64)
    starts *= np.int64(n)
    rowptr = np.searchsorted(key, starts, side="left")
    if rowptr[-1] >= 2**31:
        raise ValueError("nnz does not fit int32 row pointers")
    key -= np.repeat(starts[:-1], np.diff(rowptr))
    return rowptr.astype(np.int32), key.astype(np.int32)


def from_undirected_edges(n: int, lo: np.ndarray, hi: np.ndarray, relabel=None,
                          self_loops: bool = True, meta=None) -> Graph:
    """Symmetrise an undirected edge list, optionally relabel, add I, normalise.

    ``lo``/``hi`` list each undirected edge once (lo != hi).  ``relabel`` is a
    permutation: vertex v becomes relabel[v].
    """
    lo = np.asarray(lo, dtype=np.int64)
    hi = np.asarray(hi, dtype=np.int64)
    if relabel is not None:
        relabel = np.asarray(relabel, dtype=np.int64)
        lo, hi = relabel[lo], relabel[hi]
    parts_r = [lo, hi]
    parts_c = [hi, lo]
    if self_loops:
        ident = np.arange(n, dtype=np.int64)
        parts_r.append(ident)
        parts_c.append(ident)
    rows = np.concatenate(parts_r)
    cols = np.concatenate(parts_c)
    del parts_r, parts_c
    rowptr, col = csr_from_pairs(n, rows, cols)
    del rows, cols
    val = normalised_values(rowptr, col)
    return Graph(n=n, rowptr=rowptr, col=col, val=val, meta=dict(meta or {}))


def transposed(g: Graph) -> Graph:
    """The CSR of the transposed matrix (column c of g becomes row c, entries in row order)."""
    rows = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.rowptr.astype(np.int64)))
    order = np.argsort(g.col, kind="stable")
    counts = np.bincount(g.col.astype(np.int64), minlength=g.n)
    rowptr = np.zeros(g.n + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum(counts)
    return Graph(n=g.n, rowptr=rowptr.astype(np.int32), col=rows[order].astype(np.int32),
                 val=np.asarray(g.val)[order].astype(np.float32), meta=dict(g.meta, transposed=True))
