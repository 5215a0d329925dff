"""R-MAT power-law graphs (Chakrabarti, Zhan & Faloutsos, SDM 2004).

Each edge draw descends ``scale = log2(n)`` levels of the adjacency matrix and
at every level picks a quadrant with probabilities (a, b, c, d).  Self-loops are
dropped, each undirected edge is kept once, and draws continue until exactly
``m`` distinct undirected edges exist; the first ``m`` in draw order are kept.
The vertex ids are then shuffled by a seeded permutation (as Graph500 does) so
that hub rows are not clustered at low ids.
"""
import numpy as np

from . import rng as _rng
from .csr import from_undirected_edges

# quadrant probabilities a=.57, b=.19, c=.19, d=.05 as cut points on a uniform
# 32-bit word (each off from the exact value by less than 2^-32)
_TA = np.uint32(round(0.57 * 2**32))
_TAB = np.uint32(round(0.76 * 2**32))
_TABC = np.uint32(round(0.95 * 2**32))


def _draw(gen: np.random.Generator, count: int, scale: int):
    """``count`` edge draws; one uniform 32-bit word per level, in cache-sized chunks.

    With x1 = r >= a, x2 = r >= a+b, x3 = r >= a+b+c the quadrant's source bit
    is x2 (quadrants c, d) and its destination bit is x1 ^ x2 ^ x3 (b, d).
    """
    src = np.empty(count, dtype=np.uint32)
    dst = np.empty(count, dtype=np.uint32)
    chunk = 1 << 18
    for a in range(0, count, chunk):
        b = min(count, a + chunk)
        s = np.zeros(b - a, dtype=np.uint32)
        d = np.zeros(b - a, dtype=np.uint32)
        for level in range(scale):
            r = gen.integers(0, 2**32, size=b - a, dtype=np.uint32)
            x2 = r >= _TAB
            dbit = (r >= _TA) ^ x2 ^ (r >= _TABC)
            s |= np.left_shift(x2, level, dtype=np.uint32)
            d |= np.left_shift(dbit, level, dtype=np.uint32)
        src[a:b] = s
        dst[a:b] = d
    return src, dst


def first_occurrences(keys: np.ndarray, key_bits: int) -> np.ndarray:
    """Distinct values of ``keys`` (non-negative, < 2^key_bits) in first-occurrence order.

    Each key is packed with its position into one 64-bit word and sorted, so the
    first word of every run of equal keys carries that key's first position.
    Keys too wide to share a word with the position are first split into buckets
    by their top bits (a stable radix pass), and the packing is done per bucket.
    """
    count = keys.size
    if count == 0:
        return keys.copy()
    pos_bits = max(1, int(count - 1).bit_length())
    spare = 64 - pos_bits
    top_bits = max(0, key_bits - spare)
    if top_bits > 16:
        raise ValueError("keys too wide for bucketed first-occurrence search")
    k = keys.view(np.uint64) if keys.dtype == np.int64 else keys.astype(np.uint64)
    pos = np.arange(count, dtype=np.uint64)
    low_bits = key_bits - top_bits
    low_mask = np.uint64((1 << low_bits) - 1)
    pos_mask = np.uint64((1 << pos_bits) - 1)
    if top_bits == 0:
        segments = [(0, count)]
        order = None
    else:
        bucket = (k >> np.uint64(low_bits)).astype(np.uint16)
        order = np.argsort(bucket, kind="stable")
        edges = np.searchsorted(bucket[order], np.arange((1 << top_bits) + 1), side="left")
        segments = [(int(edges[i]), int(edges[i + 1])) for i in range(1 << top_bits)
                    if edges[i + 1] > edges[i]]
    firsts = []
    for a, b in segments:
        sel = slice(a, b) if order is None else order[a:b]
        packed = np.sort(((k[sel] & low_mask) << np.uint64(pos_bits)) | pos[sel])
        low = packed >> np.uint64(pos_bits)
        start = np.ones(packed.size, dtype=bool)
        start[1:] = low[1:] != low[:-1]
        firsts.append((packed[start] & pos_mask).astype(np.int64))
    first = np.concatenate(firsts)
    first.sort()
    return keys[first]


def undirected_edges(n: int, m: int, seed: int = 0):
    """Return (lo, hi) arrays of exactly m distinct undirected non-loop edges."""
    scale = int(n).bit_length() - 1
    if 1 << scale != n:
        raise ValueError("R-MAT needs n to be a power of two")
    if m > n * (n - 1) // 2:
        raise ValueError("too many edges requested")
    gen = _rng.stream(seed, _rng.GRAPH)
    accepted = np.empty(0, dtype=np.int64)
    batch = int(m * 1.3) + 1024
    while accepted.size < m:
        s, d = _draw(gen, batch, scale)
        keep = s != d
        s, d = s[keep], d[keep]
        keys = (np.minimum(s, d).astype(np.int64) << np.int64(scale)) | np.maximum(s, d)
        prev = accepted.size
        # distinct keys in first-draw order; earlier batches come first
        accepted = first_occurrences(np.concatenate([accepted, keys]), 2 * scale)
        gained = accepted.size - prev
        need = m - accepted.size
        if need > 0:
            rate = max(gained / batch, 1e-3)
            batch = int(need / rate * 1.2) + 1024
    accepted = accepted[:m]
    return accepted >> np.int64(scale), accepted & np.int64(n - 1)


def graph(n: int, m: int, seed: int = 0, relabel: bool = True):
    lo, hi = undirected_edges(n, m, seed)
    perm = _rng.stream(seed, _rng.RELABEL).permutation(n) if relabel else None
    g = from_undirected_edges(n, lo, hi, relabel=perm,
                              meta=dict(kind="rmat", n=n, m=m, seed=seed,
                                        abcd=(0.57, 0.19, 0.19, 0.05)))
    g.meta["max_degree"] = g.max_degree()
    return g
