"""Pins of the oracle's dual-metric partition (CPU only).

DualGCN Sec. 3.2: H_v = alpha N_v + (1 - alpha) D_v with N_v = S_v / k; nodes are
sorted by H and split; Sec. 3.3 Eq. (1): dense iff H >= tau = mu_H + 0.5 sigma_H.

The oracle evaluates Eq. (1) in exact integers.  Here it is checked against an
independent evaluation with Fractions and a 60-digit decimal square root, against
the textbook degree-only sort that alpha = 0 reduces to, and against the
invariants of a sorted split.
"""
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest

import oracle
from graphgen import small, configs


def _tau_decimal(H):
    """tau = mu + sigma / 2 with population sigma, as a 60-digit Decimal."""
    getcontext().prec = 60
    n = len(H)
    mu = sum(H, Fraction(0)) / n
    var = sum(((h - mu) ** 2 for h in H), Fraction(0)) / n
    sigma = (Decimal(var.numerator) / Decimal(var.denominator)).sqrt()
    return Decimal(mu.numerator) / Decimal(mu.denominator) + sigma / 2


def _check_plan(P, n):
    perm, K = P["perm"], P["K"]
    assert np.array_equal(np.sort(perm), np.arange(n))
    Ks = K[perm]
    assert np.all(Ks[1:] >= Ks[:-1])
    ties = Ks[1:] == Ks[:-1]
    assert np.all(perm[1:][ties] > perm[:-1][ties])
    ns = P["n_sparse"]
    assert np.all(Ks[:ns] < P["kstar"]) and np.all(Ks[ns:] >= P["kstar"])


@pytest.mark.parametrize("seed,n,p", [(0, 30, 0.1), (1, 60, 0.05), (2, 25, 0.4), (3, 80, 0.03)])
def test_threshold_matches_fraction_definition(seed, n, p):
    g = small.random_graph(n, p, seed=seed)
    k, d = 6, 4
    P = oracle.partition(g, seed=seed, k=k, steps=d)
    S = oracle.density_sums(g, seed, k, d)
    D = np.diff(g.rowptr)
    H = [Fraction(1, 2) * Fraction(int(s), k) + Fraction(1, 2) * int(dv) for s, dv in zip(S, D)]
    tau = _tau_decimal(H)
    dense_ref = np.array([Decimal(h.numerator) / Decimal(h.denominator) >= tau for h in H])
    assert np.array_equal(P["dense"], dense_ref)
    assert P["n_sparse"] == n - dense_ref.sum()
    _check_plan(P, n)
    # K* is the least integer key meeting the threshold
    Kstar = P["kstar"]
    q_k = 2 * k
    assert Decimal(Kstar) / q_k >= tau
    assert Decimal(Kstar - 1) / q_k < tau


def test_alpha_zero_is_degree_only_sort():
    g = configs.load_graph("c1")
    P = oracle.partition(g, seed=0, k=8, steps=4, alpha=(0, 1))
    D = np.diff(g.rowptr)
    assert np.array_equal(P["perm"], np.argsort(D, kind="stable"))
    _check_plan(P, g.n)


def test_alpha_one_is_density_only_sort():
    g = small.random_graph(70, 0.08, seed=4)
    P = oracle.partition(g, seed=3, k=5, steps=5, alpha=(1, 1))
    S = oracle.density_sums(g, 3, 5, 5)
    assert np.array_equal(P["perm"], np.argsort(S, kind="stable"))


def test_equal_scores_make_every_node_dense():
    # a cycle with alpha = 0: every degree is 3, sigma = 0, H = tau -> dense (ties go dense)
    g = small.cycle(20, self_loops=True, normalise=True)
    P = oracle.partition(g, seed=0, k=4, steps=3, alpha=(0, 1))
    assert P["n_sparse"] == 0 and P["dense"].all()
    assert np.array_equal(P["perm"], np.arange(20))


def test_forced_modes_only_move_the_split():
    g = small.random_graph(50, 0.1, seed=1)
    auto = oracle.partition(g, 0, 4, 4)
    sp_ = oracle.partition(g, 0, 4, 4, force=oracle.FORCE_SPARSE)
    de = oracle.partition(g, 0, 4, 4, force=oracle.FORCE_DENSE)
    assert sp_["n_sparse"] == 50 and de["n_sparse"] == 0
    for P in (sp_, de):
        assert np.array_equal(P["perm"], auto["perm"]) and P["kstar"] == auto["kstar"]


def test_beta_generalises_threshold():
    g = small.random_graph(60, 0.1, seed=6)
    for beta in [(0, 1), (1, 1), (3, 2)]:
        P = oracle.partition(g, 1, 4, 4, beta=beta)
        K = P["K"].astype(np.float64)
        mu, sd = K.mean(), K.std()
        tau = mu + beta[0] / beta[1] * sd
        ok = np.abs(K - tau) > 1e-9 * (1 + tau)        # away from float ties
        assert np.array_equal(P["dense"][ok], (K >= tau)[ok])


def test_c1_plan_invariants_and_moments():
    g = configs.load_graph("c1")
    P = oracle.partition(g, seed=0, k=8, steps=4)
    _check_plan(P, g.n)
    K = P["K"]
    assert P["S1"] == sum(int(x) for x in K)
    assert P["S2"] == sum(int(x) ** 2 for x in K)
    assert 0 < P["n_sparse"] < g.n
    S = P["S"]
    assert np.all(S >= 8) and np.all(S <= 8 * 5)        # 1 <= distinct <= d+1 per walk
