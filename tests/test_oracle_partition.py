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


# ---------------------------------------------------------------- adaptive alpha
# The adaptive weight is alpha = Var(N) / (Var(N) + Var(D)) (population variances,
# N = S / k), 1/2 when neither varies.  Graphs whose walks are deterministic (every
# row has at most one entry) fix N and D by hand, independently of the walk stream.

def _pairs_and_empties(pairs, empties):
    """`pairs` 2-cycles u <-> v (one entry per row, no self-loops) and `empties` empty rows."""
    rows = []
    for i in range(pairs):
        rows += [[2 * i + 1], [2 * i]]
    return small.from_rows(rows + [[] for _ in range(empties)])


def _triangles_and_empties(tri, empties):
    """`tri` directed 3-cycles a -> b -> c -> a and `empties` empty rows."""
    rows = []
    for i in range(tri):
        a = 3 * i
        rows += [[a + 1], [a + 2], [a]]
    return small.from_rows(rows + [[] for _ in range(empties)])


@pytest.mark.parametrize("k,q", [(4, 1024), (7, 1000), (1, 2)])
def test_adaptive_alpha_equal_spreads_is_half(k, q):
    # N is 2 on the paired rows and 1 on the empty ones; D is 1 and 0: the same
    # spread, so alpha = 1/2 whatever the mix
    g = _pairs_and_empties(5, 13)
    S = oracle.density_sums(g, 9, k, 3)
    assert sorted(set(S.tolist())) == [k, 2 * k]
    assert oracle.adaptive_alpha(S, oracle.degrees(g), k, q) == q // 2


@pytest.mark.parametrize("k", [3, 8])
def test_adaptive_alpha_triangles_closed_form(k):
    # N is 3 or 1 (d >= 2), D is 1 or 0 on the same rows: Var(N) = 4 Var(D), alpha = 4/5
    g = _triangles_and_empties(4, 9)
    S = oracle.density_sums(g, 2, k, 4)
    assert sorted(set(S.tolist())) == [k, 3 * k]
    D = oracle.degrees(g)
    for q in (5, 1000, 1024, 65535):
        assert oracle.adaptive_alpha(S, D, k, q) == (4 * q) // 5
    # Fraction check of the same closed form on the raw values
    N = [Fraction(int(s), k) for s in S]
    mN = sum(N) / len(N)
    vN = sum((x - mN) ** 2 for x in N) / len(N)
    mD = Fraction(int(D.sum()), len(D))
    vD = sum((int(x) - mD) ** 2 for x in D) / len(D)
    assert vN / (vN + vD) == Fraction(4, 5)


def test_adaptive_alpha_degenerate_cases():
    # neither metric varies: the default 1/2
    g = small.edgeless(12, self_loops=False, normalise=False)
    S = oracle.density_sums(g, 0, 4, 3)
    assert oracle.adaptive_alpha(S, oracle.degrees(g), 4, 1024) == 512
    # constant degree, varying density: alpha = 1 (density alone separates nodes)
    g = small.cycle(20, self_loops=True, normalise=True)
    S = oracle.density_sums(g, 1, 6, 4)
    assert len(set(S.tolist())) > 1
    assert oracle.adaptive_alpha(S, oracle.degrees(g), 6, 1024) == 1024
    # constant density, varying degree: alpha = 0 (rows holding only repeated
    # self-loops keep every walk at its start, while their lengths differ)
    g = small.from_rows([[0] * 3, [1], [2] * 5, [3] * 2])
    S = oracle.density_sums(g, 0, 4, 3)
    assert set(S.tolist()) == {4}
    assert oracle.adaptive_alpha(S, oracle.degrees(g), 4, 1024) == 0


# ---------------------------------------------------------------- balanced alpha
# The balanced weight gives both terms of H the same spread: alpha sigma_N = (1 - alpha)
# sigma_D, alpha = sigma_D / (sigma_N + sigma_D).  Pinned by closed forms on the same
# deterministic-walk graphs, by 60-digit square roots, and by its degenerate cases.

@pytest.mark.parametrize("k,q", [(4, 1024), (7, 1000), (1, 2), (16, 65535)])
def test_balanced_alpha_equal_spreads_is_half(k, q):
    g = _pairs_and_empties(5, 13)
    S = oracle.density_sums(g, 9, k, 3)
    assert oracle.balanced_alpha(S, oracle.degrees(g), k, q) == q // 2


@pytest.mark.parametrize("k", [3, 8])
def test_balanced_alpha_triangles_closed_form(k):
    # N is 3 or 1, D is 1 or 0 on the same rows: sigma_N = 2 sigma_D, alpha = 1/3 (where
    # the variance rule gives 4/5: the two readings weigh the metrics oppositely)
    g = _triangles_and_empties(4, 9)
    S = oracle.density_sums(g, 2, k, 4)
    D = oracle.degrees(g)
    for q in (3, 5, 1000, 1024, 65535):
        assert oracle.balanced_alpha(S, D, k, q) == q // 3
    assert oracle.adaptive_alpha(S, D, k, 1000) == 800


def test_balanced_alpha_degenerate_cases():
    g = small.edgeless(12, self_loops=False, normalise=False)          # nothing varies
    S = oracle.density_sums(g, 0, 4, 3)
    assert oracle.balanced_alpha(S, oracle.degrees(g), 4, 1024) == 512
    g = small.cycle(20, self_loops=True, normalise=True)               # constant degree
    S = oracle.density_sums(g, 1, 6, 4)
    assert len(set(S.tolist())) > 1
    assert oracle.balanced_alpha(S, oracle.degrees(g), 6, 1024) == 1024
    g = small.from_rows([[0] * 3, [1], [2] * 5, [3] * 2])               # constant density
    S = oracle.density_sums(g, 0, 4, 3)
    assert set(S.tolist()) == {4}
    assert oracle.balanced_alpha(S, oracle.degrees(g), 4, 1024) == 0


@pytest.mark.parametrize("seed", range(6))
def test_balanced_alpha_against_60_digit_square_roots(seed):
    """floor(q sigma_D / (sigma_N + sigma_D)) with the standard deviations as 60-digit square
    roots of the exact variances, against the oracle's exact search."""
    gen = np.random.default_rng(seed)
    g = small.random_graph(int(gen.integers(20, 300)), float(gen.uniform(0.01, 0.2)), seed=seed)
    k = int(gen.choice([2, 8, 16]))
    S = oracle.density_sums(g, seed, k, 4)
    D = oracle.degrees(g)
    getcontext().prec = 60
    n = len(S)
    vn = Fraction(sum(int(x) ** 2 for x in S), n * k * k) - Fraction(int(S.sum()), n * k) ** 2
    vd = Fraction(sum(int(x) ** 2 for x in D), n) - Fraction(int(D.sum()), n) ** 2
    sn = (Decimal(vn.numerator) / Decimal(vn.denominator)).sqrt()
    sd = (Decimal(vd.numerator) / Decimal(vd.denominator)).sqrt()
    for q in (7, 1024, 65535):
        want = int((Decimal(q) * sd / (sn + sd)).to_integral_value(rounding="ROUND_FLOOR"))
        assert oracle.balanced_alpha(S, D, k, q) == want


def test_balanced_partition_uses_the_chosen_alpha():
    g = small.random_graph(80, 0.07, seed=11)
    P = oracle.partition(g, 5, 8, 4, alpha=(oracle.ALPHA_BALANCED, 1024))
    p = P["alpha"][0]
    assert P["alpha"][1] == 1024 and 0 < p < 1024
    fixed = oracle.partition(g, 5, 8, 4, alpha=(p, 1024))
    assert np.array_equal(P["perm"], fixed["perm"]) and P["kstar"] == fixed["kstar"]
    N = P["S"] / 8.0
    D = P["D"].astype(np.float64)
    a = D.std() / (N.std() + D.std())
    assert p <= a * 1024 < p + 1 + 1e-9
    _check_plan(P, g.n)


def test_adaptive_partition_uses_the_chosen_alpha():
    g = small.random_graph(80, 0.07, seed=11)
    P = oracle.partition(g, 5, 8, 4, alpha=(oracle.ALPHA_ADAPTIVE, 1024))
    p = P["alpha"][0]
    assert P["alpha"][1] == 1024 and 0 <= p <= 1024
    fixed = oracle.partition(g, 5, 8, 4, alpha=(p, 1024))
    assert np.array_equal(P["perm"], fixed["perm"]) and P["kstar"] == fixed["kstar"]
    # the weight against a float evaluation of the variances
    N = P["S"] / 8.0
    D = P["D"].astype(np.float64)
    a = N.var() / (N.var() + D.var())
    assert p <= a * 1024 < p + 1 + 1e-9
    _check_plan(P, g.n)
