"""Checks of the seeded input generators (CPU only)."""
import numpy as np

from graphgen import configs, rmat, sbm, small
from graphgen.csr import normalised_values


def _check_normalised_csr(g):
    rp = g.rowptr.astype(np.int64)
    assert rp[0] == 0 and np.all(np.diff(rp) >= 1)          # self-loop: no empty rows
    rows = np.repeat(np.arange(g.n), np.diff(rp))
    # sorted, duplicate-free columns
    key = rows * g.n + g.col
    assert np.all(np.diff(key) > 0)
    # diagonal present
    assert np.isin(np.arange(g.n) * g.n + np.arange(g.n), key).all()
    # symmetric pattern and values
    keyT = g.col.astype(np.int64) * g.n + rows
    order = np.argsort(keyT)
    assert np.array_equal(keyT[order], key)
    assert np.array_equal(g.val[order], g.val)
    # value definition
    d = np.diff(rp).astype(np.float64)
    ref = (1.0 / np.sqrt(d[rows] * d[g.col])).astype(np.float32)
    assert np.array_equal(g.val, ref)


def test_c1_exact_size_and_structure():
    g = configs.load_graph("c1")
    assert g.n == 4096 and g.nnz == 2 * 32768 + 4096
    _check_normalised_csr(g)


def test_c2_size():
    g = configs.load_graph("c2")
    assert g.n == 1 << 17 and g.nnz == 1_310_720
    _check_normalised_csr(g)


def test_rmat_is_deterministic_and_distinct():
    lo, hi = rmat.undirected_edges(1 << 10, 3000, seed=5)
    lo2, hi2 = rmat.undirected_edges(1 << 10, 3000, seed=5)
    assert np.array_equal(lo, lo2) and np.array_equal(hi, hi2)
    assert np.all(lo < hi)
    assert np.unique(lo * (1 << 10) + hi).size == 3000


def test_first_occurrences_matches_unique():
    gen = np.random.default_rng(0)
    for bits, count in [(10, 5000), (40, 20000), (60, 30000)]:
        k = gen.integers(0, 1 << bits, count).astype(np.int64)
        k[count // 2:] = k[:count - count // 2]
        _, first = np.unique(k, return_index=True)
        first.sort()
        assert np.array_equal(rmat.first_occurrences(k, bits), k[first])


def test_small_sbm_structure():
    g = sbm.graph(n=1 << 12, communities=8, p_in=0.2, m_inter=500, seed=3, smin=64, smax=256)
    _check_normalised_csr(g)
    sizes = np.array(g.meta["sizes"])
    off = np.concatenate([[0], np.cumsum(sizes)])
    # intra-community density close to p_in
    rp = g.rowptr.astype(np.int64)
    intra = 0
    pairs = 0
    for c in range(8):
        a, b = off[c], off[c + 1]
        cols = g.col[rp[a]:rp[b]]
        intra += np.count_nonzero((cols >= a) & (cols < b)) - (b - a)   # drop self-loops
        pairs += (b - a) * (b - a - 1)
    assert abs(intra / pairs - 0.2) < 0.02


def test_normalised_values_small():
    g = small.star(3, self_loops=True, normalise=True)
    d = np.diff(g.rowptr)
    assert d.tolist() == [4, 2, 2, 2]
    assert np.array_equal(g.val, normalised_values(g.rowptr, g.col))
    assert g.val[0] == np.float32(0.25)
