"""Stochastic block model with power-law bridges.

512 dense communities of 64..1024 nodes (sizes log-uniform) occupy contiguous id
ranges; every pair inside a community is an edge with probability ``p_in``.
The remaining nodes belong to no community.  On top of that, ``m_inter``
distinct bridge edges join nodes of different communities, their endpoints
drawn from a Chung-Lu model with Zipf weights w_i ~ rank_i^(-1/(gamma-1)).
"""
import numpy as np

from . import rng as _rng
from .csr import from_undirected_edges


def community_sizes(gen, count: int, smin: int, smax: int) -> np.ndarray:
    u = gen.random(count)
    return np.floor(smin * (smax / smin) ** u).astype(np.int64).clip(smin, smax)


def undirected_edges(n: int, communities: int = 512, smin: int = 64, smax: int = 1024,
                     p_in: float = 0.2, m_inter=None, gamma: float = 2.1, seed: int = 0):
    gen = _rng.stream(seed, _rng.GRAPH)
    sizes = community_sizes(gen, communities, smin, smax)
    if sizes.sum() > n:
        raise ValueError("communities do not fit")
    offsets = np.zeros(communities + 1, dtype=np.int64)
    np.cumsum(sizes, out=offsets[1:])
    comm = np.full(n, -1, dtype=np.int64)
    for c in range(communities):
        comm[offsets[c]:offsets[c + 1]] = c

    los, his = [], []
    tri_cache = {}
    for c in range(communities):
        s = int(sizes[c])
        if s not in tri_cache:
            tri_cache[s] = np.triu_indices(s, 1)
        ti, tj = tri_cache[s]
        hit = gen.random(ti.size) < p_in
        los.append(ti[hit] + offsets[c])
        his.append(tj[hit] + offsets[c])
    intra_lo = np.concatenate(los)
    intra_hi = np.concatenate(his)

    if m_inter is None:
        m_inter = n
    ranks = gen.permutation(n) + 1
    w = ranks.astype(np.float64) ** (-1.0 / (gamma - 1.0))
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    accepted = np.empty(0, dtype=np.int64)
    batch = int(m_inter * 1.5) + 1024
    while accepted.size < m_inter:
        a = np.searchsorted(cdf, gen.random(batch), side="right").clip(0, n - 1)
        b = np.searchsorted(cdf, gen.random(batch), side="right").clip(0, n - 1)
        lo = np.minimum(a, b)
        hi = np.maximum(a, b)
        ok = (lo != hi) & ((comm[lo] != comm[hi]) | (comm[lo] < 0))
        keys = lo[ok] * np.int64(n) + hi[ok]
        allk = np.concatenate([accepted, keys])
        _, first = np.unique(allk, return_index=True)
        first.sort()
        accepted = allk[first]
        batch = int((m_inter - accepted.size) * 2) + 1024
    accepted = accepted[:m_inter]
    lo = np.concatenate([intra_lo, accepted // n])
    hi = np.concatenate([intra_hi, accepted % n])
    info = dict(sizes=sizes.tolist(), community_nodes=int(sizes.sum()),
                intra_edges=int(intra_lo.size), inter_edges=int(m_inter))
    return lo, hi, info


def graph(n: int = 1 << 18, communities: int = 512, p_in: float = 0.2, m_inter=None,
          gamma: float = 2.1, seed: int = 0, smin: int = 64, smax: int = 1024):
    lo, hi, info = undirected_edges(n, communities, smin, smax, p_in, m_inter, gamma, seed)
    g = from_undirected_edges(n, lo, hi, relabel=None,
                              meta=dict(kind="sbm", n=n, seed=seed, p_in=p_in,
                                        gamma=gamma, **info))
    g.meta["max_degree"] = g.max_degree()
    return g
