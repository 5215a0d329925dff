"""Pins of the oracle's random stream and anonymous random walks (CPU only).

The walker must reproduce (DualGCN Sec. 3.2, Theorem 1):
* the Philox-4x64-10 stream -- checked against numpy's own Philox bit generator;
* the anonymous labelling -- restricted-growth strings, hand-derived pattern
  counts (tests/golden/arw_closed_forms.txt), exact pattern distributions and
  exact expectations found by enumerating every walk (independent code below).
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from graphgen import small

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- Philox

def _numpy_block(counter, key):
    """numpy's Philox returns block P(c + 1) first after its counter is set to c."""
    c = [int(x) for x in counter]
    value = sum(w << (64 * i) for i, w in enumerate(c))
    value = (value - 1) % (1 << 256)
    prev = np.array([(value >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.asarray(key, dtype=np.uint64), counter=prev)
    return bg.random_raw(4).astype(np.uint64)


@pytest.mark.parametrize("counter,key", [
    ([0, 0, 0, 0], [0, 0]),
    ([1, 0, 0, 0], [7, 0]),
    ([0, 5, 0, 0], [0, 0]),          # borrow across the first word
    ([123456789, 15, 1, 0], [0, 0]),
    ([2**64 - 1, 2**64 - 1, 3, 9], [2**63 + 5, 2**40 + 1]),
])
def test_philox_matches_numpy(counter, key):
    assert np.array_equal(oracle.philox(counter, key), _numpy_block(counter, key))


def test_philox_random_cases_match_numpy():
    gen = np.random.default_rng(11)
    for _ in range(200):
        c = gen.integers(0, 2**63, 4, dtype=np.uint64) * np.uint64(2) + gen.integers(0, 2, 4,
                                                                                     dtype=np.uint64)
        k = gen.integers(0, 2**63, 2, dtype=np.uint64)
        assert np.array_equal(oracle.philox(c, k), _numpy_block(c, k))


# ---------------------------------------------------------------- enumeration (independent)

def _adjacency(g):
    return [list(map(int, g.col[g.rowptr[v]:g.rowptr[v + 1]])) for v in range(g.n)]


def enumerate_patterns(g, start, d):
    """Exact distribution {pattern: probability} of the d-step anonymous walk from start."""
    adj = _adjacency(g)
    dist = {}

    def rec(path, prob):
        if len(path) == d + 1:
            first = {}
            lab = tuple(first.setdefault(x, len(first) + 1) for x in path)
            dist[lab] = dist.get(lab, 0) + prob
            return
        nb = adj[path[-1]]
        if not nb:
            rec(path + [path[-1]], prob)
            return
        for y in nb:
            rec(path + [y], prob * Fraction(1, len(nb)))

    rec([start], Fraction(1))
    return dist


def _graph(kind, size, loops):
    return {"clique": small.clique, "path": small.path, "star": small.star}[kind](size, bool(loops))


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#")[0].split()
            if line:
                yield line


# ---------------------------------------------------------------- label invariants

def _restricted_growth(lab):
    if lab[0] != 1:
        return False
    top = 1
    for x in lab[1:]:
        if x < 1 or x > top + 1:
            return False
        top = max(top, x)
    return True


def test_patterns_are_restricted_growth_strings():
    g = small.random_graph(40, 0.15, seed=3, self_loops=True)
    P = oracle.patterns(g, seed=5, k=6, steps=7)
    for lab in P.reshape(-1, 8):
        assert _restricted_growth(lab)


def test_no_self_loops_means_no_repeated_label():
    g = small.random_graph(40, 0.2, seed=4, self_loops=False)
    deg = np.diff(g.rowptr)
    # nodes of positive degree only: isolated nodes stay put by definition
    P3 = oracle.patterns(g, seed=1, k=4, steps=6)
    for v in np.flatnonzero(deg > 0):
        for lab in P3[v]:
            assert np.all(lab[1:] != lab[:-1])


def test_empty_row_keeps_walk_in_place():
    g = small.from_rows([[1], [], [0, 1]])
    lab = oracle.walk(g, 1, 0, seed=9, steps=6)
    assert lab.tolist() == [1] * 7
    lab = oracle.walk(g, 0, 0, seed=9, steps=3)
    assert lab.tolist() == [1, 2, 2, 2]


def test_distinct_count_is_max_label_and_density_sums():
    g = small.random_graph(30, 0.2, seed=8)
    P = oracle.patterns(g, seed=2, k=5, steps=5)
    S = oracle.density_sums(g, seed=2, k=5, steps=5)
    assert np.array_equal(S, P.max(axis=2).sum(axis=1).astype(np.uint32))
    S_sub = oracle.density_sums(g, seed=2, k=5, steps=5, nodes=np.array([7, 3, 3]))
    assert S_sub.tolist() == [S[7], S[3], S[3]]


# ---------------------------------------------------------------- pattern counts (golden)

@pytest.mark.parametrize("row", list(_rows("arw_closed_forms.txt")))
def test_distinct_pattern_counts(row):
    kind, size, loops, start, d, expected = row[0], *map(int, row[1:])
    g = _graph(kind, size, loops)
    exact = enumerate_patterns(g, start, d)
    assert len(exact) == expected          # pins the enumerator to the hand count
    # enough sampled walks hit every possible pattern and nothing else; with
    # k = 25 / p_min a pattern is missed with probability below e^-25
    k = int(25 / float(min(exact.values()))) + 1
    seen = set()
    for w in range(k):
        seen.add(tuple(oracle.walk(g, start, w, seed=17, steps=d).tolist()))
    assert seen == set(exact)


def test_pattern_distribution_chi_square():
    # a small irregular graph: triangle with a pendant path and a self-loop
    g = small.from_rows([[1, 2], [0, 2, 3], [0, 1], [1, 4], [3, 4]])
    d, start, k = 4, 1, 20000
    exact = enumerate_patterns(g, start, d)
    counts = {}
    for w in range(k):
        t = tuple(oracle.walk(g, start, w, seed=123, steps=d).tolist())
        counts[t] = counts.get(t, 0) + 1
    assert set(counts) <= set(exact)
    chi2 = sum((counts.get(t, 0) - k * float(p)) ** 2 / (k * float(p)) for t, p in exact.items())
    dof = len(exact) - 1
    # deterministic (fixed seed); 99.99th percentile of chi-square ~ dof + 6 sqrt(2 dof)
    assert chi2 < dof + 6 * math.sqrt(2 * dof) + 10


@pytest.mark.parametrize("row", list(_rows("arw_expectations.txt")))
def test_density_expectation(row):
    kind, size, loops, start, d, num, den = row[0], *map(int, row[1:])
    g = _graph(kind, size, loops)
    exact = enumerate_patterns(g, start, d)
    mean = sum(max(t) * p for t, p in exact.items())
    assert mean == Fraction(num, den)      # pins the enumerator to the hand derivation
    var = sum((max(t) - mean) ** 2 * p for t, p in exact.items())
    k = 40000
    S = oracle.density_sums(g, seed=31, k=k, steps=d, nodes=np.array([start]))[0]
    sampled = S / k
    assert abs(sampled - float(mean)) < 5 * math.sqrt(float(var) / k) + 1e-12


def test_density_orders_equal_degree_nodes():
    """Fig. 2 motivation (Sec. 2.3): same degree, denser neighbourhood -> larger N."""
    star = small.star(4)
    k5 = small.clique(5)
    k = 20000
    n_star = oracle.density_sums(star, 1, k, 4, nodes=np.array([0]))[0] / k
    n_k5 = oracle.density_sums(k5, 1, k, 4, nodes=np.array([0]))[0] / k
    assert n_star < n_k5


def test_neighbour_choice_is_uniform_over_row_entries():
    """Row 0 lists node 1 twice and node 2 once, so a step from 0 reaches 1 w.p. 2/3.

    Node 1 has a second neighbour (3), node 2 has none but 0, so the two-step
    pattern [1, 2, 3] occurs only through node 1 and then node 3: p = 2/3 * 1/2.
    """
    g = small.from_rows([[1, 1, 2], [0, 3], [0], [1]])
    k = 30000
    hits = sum(oracle.walk(g, 0, w, seed=5, steps=2).tolist() == [1, 2, 3] for w in range(k))
    p = (2 / 3) * (1 / 2)
    assert abs(hits / k - p) < 5 * math.sqrt(p * (1 - p) / k)


def test_walk_counter_layout():
    """Step s of walk w from v uses the 32-bit half (low for even s) of word (s div 2) mod 4 of
    Philox block (v, w, s div 8, 0), key (seed, 0); the blocks come from numpy's Philox."""
    g = small.clique(9)                       # 8 neighbours per row, no self-loops
    seed, v, w, d = 77, 3, 5, 19              # three blocks, odd and even steps
    lab = oracle.walk(g, v, w, seed, d)
    cur, seen, expect = v, [v], [1]
    for s in range(d):
        word = int(_numpy_block([v, w, s // 8, 0], [seed, 0])[(s // 2) % 4])
        half = (word >> (32 * (s % 2))) & 0xFFFFFFFF
        row = g.col[g.rowptr[cur]:g.rowptr[cur + 1]]
        idx = (half * len(row)) >> 32
        cur = int(row[idx])
        if cur not in seen:
            seen.append(cur)
        expect.append(seen.index(cur) + 1)
    assert lab.tolist() == expect
