"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: values the
paper prints for its worked examples (tests/golden/), exact rationals for the
hardness construction, the identities of Lemma 2.2, closed forms, brute force
on tiny instances and invariance under permutation of keys.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import fw_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rand_instance(rng, n, d, temp=1.0):
    z = rng.standard_normal(n) * temp
    V = rng.standard_normal((n, d))
    return z, O.weights(z), V


# ---------------------------------------------------------------------------
# Worked examples printed in the paper
# ---------------------------------------------------------------------------

def test_example_2_3_values():
    g = _golden("example_2_3.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    for key, val in g["es"].items():
        A = [int(x) for x in key.split(",")]
        assert O.forced_error(p, v, A) == pytest.approx(float(Fraction(val)), rel=1e-14)
    best, ES = O.best_subset(p, v, g["k"])
    assert best.tolist() == g["best_set"]
    assert ES == pytest.approx(float(Fraction(g["ES"])), rel=1e-14)
    top = O.top_mass_set(np.log(p), g["k"])
    assert sorted(top.tolist()) == g["top_mass_set"]
    es_top = O.forced_error(p, v, top)
    assert es_top / ES == pytest.approx(float(Fraction(g["kappa"])), rel=1e-13)
    assert O.closed_fraction(es_top, ES) == pytest.approx(float(Fraction(g["closed_fraction"])), rel=1e-13)


def test_example_2_3_swap_rule():
    g = _golden("example_2_3.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    for method in ("direct", "gform"):
        S, traj, ns = O.swap_rule(p, v, g["k"], max_iters=8, method=method)
        assert S.tolist() == g["swap_final"]
        assert ns == g["n_swaps"]
        want = [float(Fraction(x)) for x in g["swap_trajectory"]]
        assert np.allclose(traj[: ns + 1], want, rtol=1e-13)
        assert np.all(np.isnan(traj[ns + 1:]))


def test_example_A3_table_and_tie_rule():
    g = _golden("example_A3.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    for key, val in g["es"].items():
        A = [int(x) for x in key.split(",")]
        assert O.forced_error(p, v, A) == pytest.approx(float(Fraction(val)), rel=1e-14, abs=1e-15)
    for s, want in g["lexicographic_best"].items():
        best, ES = O.best_subset(p, v, int(s))
        exact = g["exact_in_float64"][s]
        if exact:
            assert best.tolist() == want
        else:  # tied optimum: any tied set is correct, the value is pinned
            ties = [k for k, val in g["es"].items() if len(k.split(",")) == int(s)
                    and Fraction(val) == min(Fraction(x) for kk, x in g["es"].items()
                                             if len(kk.split(",")) == int(s))]
            assert ",".join(map(str, best.tolist())) in ties
        assert ES == pytest.approx(float(min(Fraction(x) for kk, x in g["es"].items()
                                             if len(kk.split(",")) == int(s))), abs=1e-15)
    # uniform masses: the top-mass set is the lowest indices
    for s in (1, 2, 3):
        assert O.top_mass_set(np.zeros(4), s).tolist() == list(range(s))


def test_example_A3_not_submodular_statements():
    """The printed increments: adding key 0 to {2} keeps es at 1/2, adding it
    to {1,2} raises es from 0 to 1/2; adding it to {1} raises es from 1/2 to 1,
    adding it to {1,3} lowers es from 1/2 to 1/6."""
    v = np.arange(4.0)[:, None]
    p = np.full(4, 0.25)
    es = lambda A: O.forced_error(p, v, A)
    assert es([2]) == es([0, 2]) == 0.5
    assert es([1, 2]) == 0.0 and es([0, 1, 2]) == 0.5
    assert es([1]) == 0.5 and es([0, 1]) == 1.0
    assert es([1, 3]) == 0.5 and es([0, 1, 3]) == pytest.approx(1 / 6, rel=1e-14)


def test_row_dense_topk_example_2_3():
    """Example 2.3 through the batched top-k evaluator, budgets given out of
    order: mu = 1/2; the top-1 set is {0} (keys 0 and 1 tie in mass, the lower
    index wins), m = -1, gap 3/2, dropped 11/20; the top-2 set {0,1} has m = 0,
    gap 1/2 (the example's value), dropped 1/10; keeping all three keys gives
    m = mu, gap 0, dropped 0."""
    g = _golden("example_2_3.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    r = O.row_dense_topk(np.log(p), v, (3, 1, 2))
    assert r["o"][0] == pytest.approx(0.5, rel=1e-14)
    assert r["topk_idx"].tolist() == [0, 1, 2]
    np.testing.assert_allclose(r["o_s"][:, 0], [0.5, -1.0, 0.0], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(r["gap"], [0.0, 1.5, float(Fraction(g["es"]["0,1"]))], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(r["dropped"], [0.0, 0.55, 0.1], rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("seed", range(4))
def test_row_dense_topk_per_budget_first_form(seed):
    """Every budget's forced output, gap and dropped mass come from that
    budget's own top-mass set: checked against plain loops over the set
    ranked by (logit desc, index asc) and against Lemma 2.2's first form
    es(S) = (1 - p(S)) ||m_{S^c} - m_S||."""
    rng = np.random.default_rng(1200 + seed)
    n, d = 17, 4
    z = np.round(rng.standard_normal(n) * 2.0, 1)  # rounding creates logit ties
    V = rng.standard_normal((n, d))
    ks = (11, 3, 7, n)
    r = O.row_dense_topk(z, V, ks)
    e = [math.exp(z[j] - max(z)) for j in range(n)]
    p = [x / sum(e) for x in e]
    order = sorted(range(n), key=lambda j: (-z[j], j))
    assert r["topk_idx"].tolist() == order[: max(ks)]
    for t, k in enumerate(ks):
        S, Sc = order[:k], order[k:]
        pS = sum(p[j] for j in S)
        mS = [sum(p[j] * V[j][c] for j in S) / pS for c in range(d)]
        np.testing.assert_allclose(r["o_s"][t], mS, rtol=1e-12, atol=1e-14)
        assert r["dropped"][t] == pytest.approx(sum(p[j] for j in Sc), rel=1e-12, abs=1e-15)
        if not Sc:
            assert r["gap"][t] == 0.0
            continue
        pSc = sum(p[j] for j in Sc)
        mSc = [sum(p[j] * V[j][c] for j in Sc) / pSc for c in range(d)]
        first = (1.0 - pS) * math.sqrt(sum((mSc[c] - mS[c]) ** 2 for c in range(d)))
        assert r["gap"][t] == pytest.approx(first, rel=1e-10)


def test_row_best_subset_example_2_3():
    """Example 2.3 through the per-row exhaustive evaluator: best set {0,2}
    (the paper's {1,3}) at 9/22, top-mass set {0,1} at 1/2, closed fraction
    2/11, and the top-mass set drops mass 1/10."""
    g = _golden("example_2_3.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    r = O.row_best_subset(np.log(p), v, g["k"])
    assert r["best_idx"].tolist() == g["best_set"]
    assert r["topk_idx"].tolist() == g["top_mass_set"]
    assert r["best_gap"] == pytest.approx(float(Fraction(g["ES"])), rel=1e-14)
    assert r["topk_gap"] == pytest.approx(float(Fraction(g["es"]["0,1"])), rel=1e-14)
    assert r["closed"] == pytest.approx(float(Fraction(g["closed_fraction"])), rel=1e-13)
    assert r["dropped_topk"] == pytest.approx(0.1, rel=1e-13)


def test_balancing_stops_at_a_local_optimum():
    """A row on which the balancing selector stops above the candidate-set
    optimum (exact rationals in the fixture): no swap improves A*_s, so it
    returns A*_s with zero swaps, while ES_pool is lower; kappa_bal =
    es(A_bal) / ES_pool = 22/7, and never below 1."""
    g = _golden("balancing_local_optimum.json")
    F = lambda x: float(Fraction(x))
    v = np.array(g["v"], float)[:, None]
    p = np.array([F(x) for x in g["p"]])
    for key, val in g["swap_es"].items():
        assert O.forced_error(p, v, [int(x) for x in key.split(",")]) == pytest.approx(F(val), rel=1e-13)
    r = O.row_pool(np.log(p), v, g["s"], g["extra"], max_iters=8)
    assert r["top"].tolist() == g["top"]
    assert r["bal_idx"].tolist() == g["bal_set"] and r["n_swaps"] == g["n_swaps"]
    assert r["best_idx"].tolist() == g["best_set"]
    assert r["es_top"] == pytest.approx(F(g["es_top"]), rel=1e-13)
    assert r["es_bal"] == pytest.approx(F(g["es_top"]), rel=1e-13)
    assert r["es_pool"] == pytest.approx(F(g["ES_pool"]), rel=1e-12)
    assert r["kappa_hat"] == pytest.approx(F(g["kappa_hat"]), rel=1e-12)
    assert r["kappa_bal"] == pytest.approx(F(g["kappa_bal"]), rel=1e-12)
    assert r["c_hat"] == pytest.approx(F(g["c_hat"]), rel=1e-12)
    S, traj, ns = O.swap_rule(p, v, g["s"], 8, method="direct")
    assert S.tolist() == sorted(g["bal_set"]) and ns == 0


# ---------------------------------------------------------------------------
# Hardness construction (Appendix A.2) in exact rationals
# ---------------------------------------------------------------------------

def _balanced_split_exists(w):
    """Independent subset-sum check: some half-size subset with half the sum."""
    m, W = len(w), sum(w)
    if W % 2:
        return False
    reach = {(0, 0)}
    for x in w:
        reach |= {(c + 1, s + x) for (c, s) in reach if c < m // 2}
    return (m // 2, W // 2) in reach


@pytest.mark.parametrize("seed", range(12))
def test_hardness_family_exact(seed):
    rng = np.random.default_rng(1000 + seed)
    m = int(rng.choice([4, 6, 8, 10]))
    w = [int(x) for x in rng.integers(0, 9, size=m)]
    W = sum(w)
    s = m // 2
    # Lemma A.5: g_A = (m sum_A w - |A| W)/m^2; Lemma A.6: p(A) = 1/2, es = 2|g_A|
    exact = {}
    for A in itertools.combinations(range(m), s):
        gA = Fraction(m * sum(w[i] for i in A) - s * W, m * m)
        exact[A] = 2 * abs(gA)
    ES_exact = min(exact.values())
    p = np.full(m, 1.0 / m)
    v = np.array(w, float)[:, None]
    best, ES = O.best_subset(p, v, s)
    assert ES == pytest.approx(float(ES_exact), abs=1e-12)
    assert exact[tuple(best.tolist())] == ES_exact
    # Proposition 2.4 / Lemma A.6: ES = 0 iff a balanced split exists, else >= 2/m^2
    if _balanced_split_exists(w):
        assert ES_exact == 0 and ES < 1e-12
    else:
        assert ES_exact >= Fraction(2, m * m) and ES >= 2.0 / m ** 2 - 1e-12


def test_hardness_all_pairs_tie():
    """w = (1,1,1,4): every pair has es = 3/4 exactly (dyadic), so the tie
    rule must return the lexicographically smallest pair {0,1}."""
    p = np.full(4, 0.25)
    v = np.array([1, 1, 1, 4.0])[:, None]
    es = O.subset_errors(p, v, O.combinations_table(4, 2))
    assert np.all(es == 0.75)
    best, ES = O.best_subset(p, v, 2)
    assert best.tolist() == [0, 1] and ES == 0.75
    best, ES = O.best_subset(p, np.array([1, 2, 3, 4.0])[:, None], 2)
    assert best.tolist() == [0, 3] and ES == 0.0


def test_swap_values_example_2_3():
    """Every single swap from Example 2.3's top-mass set {0,1}: dropping 0
    for 2 gives {1,2} at 27/22, dropping 1 for 2 gives {0,2} at 9/22 (the
    example's optimum); both evaluators agree."""
    g = _golden("example_2_3.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    for method in ("direct", "gform"):
        vals, Sin, Sout = O.swap_values(p, v, [1, 0], method)
        assert Sin.tolist() == [0, 1] and Sout.tolist() == [2]
        np.testing.assert_allclose(vals[:, 0], [float(Fraction(g["es"]["1,2"])), float(Fraction(g["es"]["0,2"]))],
                                   rtol=1e-13)


def test_swap_rule_stops_on_a_tie():
    """The balancing selector stops when no swap strictly decreases es
    (Section 2.1).  On the hardness instance w = (1,1,1,4) with uniform
    masses every pair has es = 3/4 exactly, so every swap ties the current
    set: no swap is taken, the trajectory is [3/4] and the set stays the
    top-mass set {0,1}; the same holds inside a candidate set of every key."""
    p = np.full(4, 0.25)
    v = np.array([1, 1, 1, 4.0])[:, None]
    for method in ("direct", "gform"):
        S, traj, ns = O.swap_rule(p, v, 2, 6, method=method)
        assert ns == 0 and S.tolist() == [0, 1]
        assert traj[0] == 0.75 and np.all(np.isnan(traj[1:]))
    r = O.row_pool(np.log(p), v, 2, 2, max_iters=6)
    assert r["n_swaps"] == 0 and r["bal_idx"].tolist() == [0, 1]
    assert r["kappa_bal"] == 1.0 and r["kappa_hat"] == 1.0


# ---------------------------------------------------------------------------
# Lemma 2.2 identities, the 2 D mbar bound and the k = n zero
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(10))
def test_lemma_2_2_identities(seed):
    rng = np.random.default_rng(seed)
    n, d = int(rng.integers(3, 40)), int(rng.integers(1, 9))
    z, p, V = _rand_instance(rng, n, d, temp=rng.uniform(0.3, 3))
    mu = O.dense_output(p, V)
    assert np.allclose(mu, sum(p[j] * V[j] for j in range(n)), rtol=1e-13, atol=1e-13)
    u = p[:, None] * (V - mu)
    assert np.linalg.norm(u.sum(axis=0)) < 1e-13 * (1 + np.abs(u).sum())
    for _ in range(5):
        k = int(rng.integers(1, n))
        A = np.sort(rng.choice(n, size=k, replace=False))
        Ac = np.setdiff1d(np.arange(n), A)
        es = O.forced_error(p, V, A)
        pA = p[A].sum()
        mA = (p[A, None] * V[A]).sum(0) / pA
        mAc = (p[Ac, None] * V[Ac]).sum(0) / p[Ac].sum()
        first = (1 - pA) * np.linalg.norm(mAc - mA)
        second = np.linalg.norm(u[A].sum(0)) / pA
        assert es == pytest.approx(first, rel=1e-10, abs=1e-13)
        assert es == pytest.approx(second, rel=1e-10, abs=1e-13)
        assert O.dropped_mass(p, A) == pytest.approx(1 - pA, abs=1e-14)
        w = p[A] / O.kept_mass(p, A)
        assert w.sum() == pytest.approx(1.0, abs=1e-14)
    # es(A*_k) <= 2 D mbar_k
    D = np.max(np.linalg.norm(V - mu, axis=1))
    for k in range(1, n + 1):
        top = O.top_mass_set(z, k)
        es = O.forced_error(p, V, top)
        assert es <= 2 * D * O.dropped_mass(p, top) + 1e-12
    top = O.top_mass_set(z, n)
    assert O.forced_error(p, V, top) < 1e-13
    assert O.dropped_mass(p, top) == 0.0


def test_softmax_closed_form_and_shift():
    p = O.weights(np.array([0.0, math.log(3.0)]))
    assert p == pytest.approx([0.25, 0.75], rel=1e-15)
    rng = np.random.default_rng(7)
    z = rng.standard_normal(50) * 3
    assert O.weights(z).sum() == pytest.approx(1.0, abs=1e-14)
    assert np.allclose(O.weights(z), O.weights(z + 123.25), rtol=1e-12)
    q, K = rng.standard_normal(5), rng.standard_normal((7, 5))
    bias = rng.standard_normal(7)
    assert np.allclose(O.logits(q, K, 0.5, bias), [0.5 * q @ K[j] + bias[j] for j in range(7)])


# ---------------------------------------------------------------------------
# Closed forms for k = 1, k = n-1, k = n, and brute force on tiny rows
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_closed_forms(seed):
    rng = np.random.default_rng(50 + seed)
    n, d = int(rng.integers(3, 11)), int(rng.integers(1, 6))
    z, p, V = _rand_instance(rng, n, d)
    mu = O.dense_output(p, V)
    dev = np.linalg.norm(V - mu, axis=1)
    best, ES = O.best_subset(p, V, 1)  # m_{j} = v_j
    assert best.tolist() == [int(np.argmin(dev))]
    assert ES == pytest.approx(dev.min(), rel=1e-12)
    best, ES = O.best_subset(p, V, n - 1)  # dropping j: es = p_j |v_j - mu| / (1 - p_j)
    drop = p * dev / (1 - p)
    j = int(np.argmin(drop))
    assert best.tolist() == [i for i in range(n) if i != j]
    assert ES == pytest.approx(drop.min(), rel=1e-10)
    best, ES = O.best_subset(p, V, n)
    assert best.tolist() == list(range(n)) and ES < 1e-13


@pytest.mark.parametrize("seed", range(8))
def test_top_mass_brute_force(seed):
    """pbar(A*_k) is the least achievable dropped mass over all |A| = k."""
    rng = np.random.default_rng(90 + seed)
    n = int(rng.integers(2, 11))
    z = np.round(rng.standard_normal(n), 1)  # rounding creates ties
    p = O.weights(z)
    for k in range(1, n + 1):
        top = O.top_mass_set(z, k)
        brute = min(1 - p[list(A)].sum() for A in itertools.combinations(range(n), k))
        assert O.dropped_mass(p, top) == pytest.approx(brute, abs=1e-14)
        # ties to the lower index: the set is the first k of the (z desc, j asc) order
        order = sorted(range(n), key=lambda j: (-z[j], j))
        assert top.tolist() == order[:k]
    assert O.top_mass_set(np.array([1.0, 2.0, 2.0, 0.0]), 2).tolist() == [1, 2]
    assert O.top_mass_set(np.array([2.0, 2.0, 2.0]), 2).tolist() == [0, 1]


@pytest.mark.parametrize("seed", range(6))
def test_best_subset_permutation_invariance(seed):
    rng = np.random.default_rng(200 + seed)
    n, d = int(rng.integers(4, 11)), int(rng.integers(1, 5))
    z, p, V = _rand_instance(rng, n, d, temp=1.5)
    k = int(rng.integers(1, n))
    best, ES = O.best_subset(p, V, k)
    # brute force by a different route: itertools + direct definition one by one
    vals = {A: O.forced_error(p, V, A) for A in itertools.combinations(range(n), k)}
    assert ES == pytest.approx(min(vals.values()), rel=1e-12)
    perm = rng.permutation(n)
    best2, ES2 = O.best_subset(p[perm], V[perm], k)
    assert ES2 == pytest.approx(ES, rel=1e-12)
    if sorted(vals.values())[1] > ES * (1 + 1e-9):  # unique optimum
        assert sorted(perm[best2].tolist()) == best.tolist()


# ---------------------------------------------------------------------------
# Swap rule: ordering, local optimality, agreement of the two searches
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(8))
def test_swap_rule_invariants(seed):
    rng = np.random.default_rng(300 + seed)
    n, d = int(rng.integers(5, 13)), int(rng.integers(1, 8))
    z, p, V = _rand_instance(rng, n, d, temp=2.0)
    k = int(rng.integers(1, n))
    top = O.top_mass_set(z, k)
    S, traj, ns = O.swap_rule(p, V, k, 64, start=top, method="direct")
    S2, traj2, ns2 = O.swap_rule(p, V, k, 64, start=top, method="gform")
    assert S.tolist() == S2.tolist() and ns == ns2
    assert np.allclose(traj[: ns + 1], traj2[: ns + 1], rtol=1e-10)
    es_swap = O.forced_error(p, V, S)
    es_top = O.forced_error(p, V, top)
    _, ES = O.best_subset(p, V, k)
    assert ES <= es_swap * (1 + 1e-12) and es_swap <= es_top * (1 + 1e-12)
    assert traj[0] == pytest.approx(es_top, rel=1e-14)
    assert np.all(np.diff(traj[: ns + 1]) < 0)
    assert traj[ns] == pytest.approx(es_swap, rel=1e-14)
    # local optimum: no single swap decreases es (checked one pair at a time)
    if ns < 64:
        for i in S:
            for j in np.setdiff1d(np.arange(n), S):
                T = np.sort(np.concatenate([S[S != i], [j]]))
                assert O.forced_error(p, V, T) >= es_swap * (1 - 1e-12)
    c = O.closed_fraction(es_top, ES)
    assert -1e-12 <= c <= 1.0


def test_swap_rule_max_iters_and_edges():
    rng = np.random.default_rng(5)
    z, p, V = _rand_instance(rng, 12, 3, temp=3.0)
    S, traj, ns = O.swap_rule(p, V, 4, 0, start=O.top_mass_set(z, 4))
    assert ns == 0 and traj.shape == (1,)
    S, traj, ns = O.swap_rule(p, V, 12, 5, start=O.top_mass_set(z, 12))
    assert ns == 0 and traj[0] < 1e-13


# ---------------------------------------------------------------------------
# Dropped-mass curve, allocation, compaction
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_dropped_mass_curve(seed):
    rng = np.random.default_rng(400 + seed)
    G, n, d = 4, int(rng.integers(2, 11)), 3
    Qw, K = rng.standard_normal((G, d)), rng.standard_normal((n, d))
    r = O.importance(Qw, K, 0.7)
    assert r.sum() == pytest.approx(1.0, abs=1e-14)
    assert np.allclose(r, np.mean([O.weights(O.logits(Qw[g], K, 0.7)) for g in range(G)], axis=0))
    c = O.dropped_mass_curve(r)
    assert c.shape == (n + 1,)
    assert c[0] == pytest.approx(1.0, abs=1e-14) and c[n] == 0.0
    assert np.all(np.diff(c) <= 0)
    for k in range(n + 1):
        brute = min(sum(r[j] for j in range(n) if j not in A) for A in itertools.combinations(range(n), k))
        assert c[k] == pytest.approx(brute, abs=1e-15)


def _alloc_brute(r, budget, floor):
    H, n = r.shape
    f = min(floor, n)
    cand = sorted(((-r[h, j], h, j) for h in range(H) for j in range(n - f)))
    quota = budget - H * f
    kept = cand[:quota]
    keep = np.zeros((H, n), bool)
    keep[:, n - f:] = True
    for _, h, j in kept:
        keep[h, j] = True
    return keep, (-kept[-1][0] if kept else math.inf)


@pytest.mark.parametrize("seed", range(6))
def test_allocation(seed):
    rng = np.random.default_rng(500 + seed)
    H, n, floor = int(rng.integers(1, 6)), int(rng.integers(4, 40)), int(rng.integers(0, 5))
    r = np.round(rng.random((H, n)), 2)  # coarse values create ties at tau
    budget = int(rng.integers(H * min(floor, n), H * n + 1))
    a = O.allocate(r, budget, floor)
    keep, tau = _alloc_brute(r, budget, floor)
    assert np.array_equal(a["keep"], keep)
    assert a["tau"] == tau
    assert a["counts"].sum() == budget and np.all(a["counts"] >= min(floor, n))
    nf = np.zeros((H, n), bool)
    nf[:, : n - min(floor, n)] = True
    if a["quota"] > 0:
        assert r[nf & ~a["keep"]].max(initial=-1) <= a["tau"] <= r[nf & a["keep"]].min()
    assert np.allclose(a["dropped"], (r * ~keep).sum(1))


def test_allocation_rejects_bad_budget():
    with pytest.raises(ValueError):
        O.allocate(np.ones((2, 8)), 3, 2)
    with pytest.raises(ValueError):
        O.allocate(np.ones((2, 8)), 17, 2)


def test_compaction_and_bytes():
    rng = np.random.default_rng(9)
    H, hpl, n, d = 4, 2, 10, 3
    K = rng.integers(0, 1 << 16, (H, n, d)).astype(np.uint16)
    V = rng.integers(0, 1 << 16, (H, n, d)).astype(np.uint16)
    keep = rng.random((H, n)) < 0.4
    keep[:, -1] = True
    c = O.compact(K, V, keep, hpl, elem_bytes=2)
    counts = keep.sum(1)
    assert c["offsets"].tolist() == [0] + np.cumsum(counts).tolist()
    for h in range(H):
        pos = [j for j in range(n) if keep[h, j]]
        lo, hi = c["offsets"][h], c["offsets"][h + 1]
        assert c["kept_pos"][lo:hi].tolist() == pos
        assert np.array_equal(c["k_out"][lo:hi], K[h, pos])
        assert np.array_equal(c["v_out"][lo:hi], V[h, pos])
    row = 2 * d * 2
    assert c["bytes_held"][0] == counts.sum() * row
    assert c["bytes_held"][1] == (max(counts[0], counts[1]) + max(counts[2], counts[3])) * 2 * row
    assert c["bytes_held"][2] == H * n * row


def test_dense_topk_batch_consistency():
    rng = np.random.default_rng(11)
    H, G, n, d = 2, 3, 20, 4
    q, K, V = rng.standard_normal((H, G, d)), rng.standard_normal((H, n, d)), rng.standard_normal((H, n, d))
    scale = np.array([0.5, 1.5])
    bias = np.zeros(n)
    bias[0] = 4.0
    out = O.dense_topk(q, K, V, scale, bias, (3, 7, 20))
    for h in range(H):
        for g in range(G):
            z = scale[h] * (K[h] @ q[h, g]) + bias
            p = np.exp(z - z.max())
            p /= p.sum()
            assert np.allclose(out["o"][h, g], p @ V[h])
            for t, k in enumerate((3, 7, 20)):
                S = out["topk_idx"][h, g, :k]
                assert out["dropped"][t, h, g] == pytest.approx(1 - p[S].sum(), abs=1e-14)
            assert out["gap"][2, h, g] < 1e-13
            assert np.allclose(out["o_s"][2, h, g], out["o"][h, g])


# ---------------------------------------------------------------------------
# Candidate set, ES_pool, pool-restricted balancing, certificate statistics
# (Definition 2.5, Lemma 2.2, the appendix's absolute forms)
# ---------------------------------------------------------------------------

def test_pool_example_2_3():
    g = _golden("example_2_3_pool.json")
    v = np.array(g["v"], float)[:, None]
    p = np.array([float(Fraction(x)) for x in g["p"]])
    F = lambda x: float(Fraction(x))
    e = O.single_key_errors(p, v)
    assert e == pytest.approx([F(x) for x in g["single_key_errors"]], rel=1e-13)
    r = O.row_pool(np.log(p), v, g["s"], g["extra"], max_iters=8)
    assert r["top"].tolist() == g["top"] and r["extras"].tolist() == g["extras"]
    assert r["best_idx"].tolist() == g["best_set"] and r["bal_idx"].tolist() == g["bal_set"]
    assert r["es_pool"] == pytest.approx(F(g["ES_pool"]), rel=1e-13)
    assert r["kappa_hat"] == pytest.approx(F(g["kappa_hat"]), rel=1e-13)
    assert r["c_hat"] == pytest.approx(F(g["c_hat"]), rel=1e-12)
    assert r["n_swaps"] == g["n_swaps"]
    assert r["dropped"] == pytest.approx(F(g["dropped"]), rel=1e-13)
    assert r["phi"] == pytest.approx(F(g["phi"]), rel=1e-13)
    assert r["diam"] == pytest.approx(F(g["diam"]), rel=1e-13)
    assert r["sigma"] ** 2 == pytest.approx(F(g["sigma_sq"]), rel=1e-13)
    assert r["bound_diam"] == pytest.approx(F(g["bound_diam"]), rel=1e-13)
    assert r["bound_var"] ** 2 == pytest.approx(F(g["bound_var_sq"]), rel=1e-13)


@pytest.mark.parametrize("seed", range(4))
def test_pool_brute_force(seed):
    """The candidate set and ES_pool against plain loops over the definitions
    on small rows: extras are the largest p_j ||v_j - mu|| outside A*_s (ties to
    the lower index), and ES_pool is the smallest es over the pool's s-subsets
    with the full row's masses and dense output; ES <= ES_pool <= es(A*_s)."""
    rng = np.random.default_rng(700 + seed)
    n, d, s, extra = 9, 3, 3, 3
    z, p, V = _rand_instance(rng, n, d, temp=1.5)
    if seed == 3:  # equal single-key errors: the lower index must win
        V[5] = V[6]
        z[5] = z[6]
        p = O.weights(z)
    top, extras = O.candidate_pool(z, V, s, extra)
    mu = sum(p[j] * V[j] for j in range(n))
    err = [p[j] * math.sqrt(sum((V[j][c] - mu[c]) ** 2 for c in range(d))) for j in range(n)]
    ranked = sorted(range(n), key=lambda j: (-z[j], j))
    assert top.tolist() == ranked[:s]
    rest = sorted((j for j in range(n) if j not in ranked[:s]), key=lambda j: (-err[j], j))
    assert extras.tolist() == rest[:extra]
    pool = sorted(ranked[:s] + rest[:extra])
    brute = min((O.forced_error(p, V, list(A)), A) for A in itertools.combinations(pool, s))
    best, es_pool = O.pool_best_subset(p, V, np.concatenate([top, extras]), s)
    assert best.tolist() == list(brute[1])
    assert es_pool == pytest.approx(brute[0], rel=1e-12)
    _, ES = O.best_subset(p, V, s)
    assert ES <= es_pool * (1 + 1e-12)
    assert es_pool <= O.forced_error(p, V, top) * (1 + 1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_pool_of_every_key_is_the_full_search(seed):
    """With every key in the candidate set, ES_pool is ES and the
    pool-restricted balancing selector is the full one (both pinned above)."""
    rng = np.random.default_rng(710 + seed)
    n, d, s = 8, 2, 3
    z, p, V = _rand_instance(rng, n, d, temp=2.0)
    r = O.row_pool(z, V, s, n - s, max_iters=16)
    best, ES = O.best_subset(p, V, s)
    assert r["best_idx"].tolist() == best.tolist()
    assert r["es_pool"] == pytest.approx(ES, rel=1e-12)
    S, traj, ns = O.swap_rule(p, V, s, max_iters=16, method="direct")
    assert r["bal_idx"].tolist() == S.tolist() and r["n_swaps"] == ns
    np.testing.assert_allclose(r["traj"], traj, rtol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_pool_swap_invariants(seed):
    """The pool-restricted trajectory decreases strictly, its set stays in the
    pool, no single in-pool swap improves the final set, and it lies between
    ES_pool and es(A*_s)."""
    rng = np.random.default_rng(720 + seed)
    n, d, s, extra = 12, 4, 4, 4
    z, p, V = _rand_instance(rng, n, d, temp=2.5)
    r = O.row_pool(z, V, s, extra, max_iters=20)
    pool = set(r["top"].tolist()) | set(r["extras"].tolist())
    S = r["bal_idx"]
    assert set(S.tolist()) <= pool
    t = r["traj"][: r["n_swaps"] + 1]
    assert np.all(np.diff(t) < 0)
    for i in S:
        for j in pool - set(S.tolist()):
            A = sorted(set(S.tolist()) - {int(i)} | {j})
            assert O.forced_error(p, V, A) >= r["es_bal"] * (1 - 1e-12)
    assert r["es_pool"] <= r["es_bal"] * (1 + 1e-12)
    assert r["es_bal"] <= r["es_top"] * (1 + 1e-12)
    assert r["kappa_hat"] >= 1 - 1e-12 and 0 <= r["c_hat"] <= 1


@pytest.mark.parametrize("seed", range(3))
def test_certificate_identities_and_bounds(seed):
    """Phi = es(S) p(S) = ||g_S|| (Lemma 2.2); sigma^2 = sum_j p_j ||v_j||^2 -
    ||mu||^2; D bounds every deviation; es(A*_s) <= 2 D pbar (Lemma 2.2) and
    every kept set satisfies es(S) <= sqrt(pbar / (1 - pbar)) sigma."""
    rng = np.random.default_rng(730 + seed)
    n, d, s = 8, 3, 3
    z, p, V = _rand_instance(rng, n, d, temp=1.0 + seed)
    top = O.top_mass_set(z, s)
    c = O.certificate(p, V, top)
    es_top = O.forced_error(p, V, top)
    assert c["phi"] == pytest.approx(es_top * O.kept_mass(p, top), rel=1e-12)
    mu = p @ V
    assert c["sigma"] ** 2 == pytest.approx(float(p @ (V * V).sum(1) - mu @ mu), rel=1e-10)
    assert c["diam"] == pytest.approx(max(math.dist(V[j], mu) for j in range(n)), rel=1e-13)
    assert es_top <= c["bound_diam"] * (1 + 1e-12)
    for k in range(1, n):
        for A in itertools.combinations(range(n), k):
            cA = O.certificate(p, V, list(A))
            assert O.forced_error(p, V, list(A)) <= cA["bound_var"] * (1 + 1e-12)


def test_cell_median():
    assert O.cell_median(np.array([0.1, 0.3, 0.2])) == pytest.approx(0.2)
    assert O.cell_median(np.array([0.1, 0.4, 0.2, 0.3])) == pytest.approx(0.25)
    assert O.ratio(0.0, 0.0) == 1.0 and O.ratio(1.0, 0.0) == math.inf


# ---------------------------------------------------------------------------
# Group vote (Section 2.1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(3))
def test_group_vote_of_one_row_is_its_top_mass_set(seed):
    """A group of one row (the multi-head family of the paper) votes exactly
    that row's top-mass set, at ratio 1."""
    rng = np.random.default_rng(800 + seed)
    z, p, V = _rand_instance(rng, 12, 3, temp=2.0)
    r = O.group_vote(z[None, :], V, 4)
    assert r["vote"].tolist() == O.top_mass_set(z, 4).tolist()
    assert r["es_vote"][0] == r["es_top"][0] and r["ratio"][0] == 1.0


@pytest.mark.parametrize("seed", range(3))
def test_group_vote_brute_force(seed):
    """The vote set holds the most summed mass of all s-subsets (ties to the
    lexicographically first), each row's error is the forced-weight error of
    that set, and identical rows vote their common top-mass set."""
    rng = np.random.default_rng(810 + seed)
    m, n, d, s = 3, 8, 2, 3
    Z = rng.standard_normal((m, n)) * 2.0
    V = rng.standard_normal((n, d))
    if seed == 2:
        Z[:, 6] = Z[:, 5]  # tied summed masses: the lower index first
    r = O.group_vote(Z, V, s)
    P = np.exp(Z - Z.max(1, keepdims=True))
    P /= P.sum(1, keepdims=True)
    best = max(itertools.combinations(range(n), s), key=lambda A: (round(P[:, list(A)].sum(), 12), [-a for a in A]))
    assert sorted(r["vote"].tolist()) == list(best)
    for i in range(m):
        assert r["es_vote"][i] == pytest.approx(O.forced_error(P[i], V, list(best)), rel=1e-12)
        assert r["dropped"][i] == pytest.approx(1.0 - P[i, list(best)].sum(), rel=1e-10)
    same = O.group_vote(np.repeat(Z[:1], 4, axis=0), V, s)
    assert same["vote"].tolist() == O.top_mass_set(Z[0], s).tolist()
    assert np.all(same["ratio"] == 1.0)



# ---------------------------------------------------------------------------
# Budget-enforced ContourKV and SnapKV's max-pooled score (Section 4; the
# appendix's audit of SnapKV)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(3))
def test_allocation_with_cap(seed):
    """A cap of n changes nothing; with a cap every cell keeps at most cap
    entries, the total is exact, and the result equals a greedy fill in the
    global order (score desc, cell asc, position asc) that skips full cells."""
    rng = np.random.default_rng(900 + seed)
    H, n, f = 5, 30, 3
    r = rng.random((H, n))
    if seed == 2:
        r[:, 4] = r[:, 5] = 0.5  # ties inside and across cells
        r[1, 10:14] = 0.5
    for budget, cap in ((60, 14), (40, 8), (H * 14, 14)):
        a = O.allocate(r, budget, f, cap)
        assert a["counts"].sum() == budget and a["counts"].max() <= cap and a["counts"].min() >= f
        keep = np.zeros((H, n), bool)
        keep[:, n - f:] = True
        order = sorted(((-r[h, j], h, j) for h in range(H) for j in range(n - f)))
        left = budget - H * f
        for _, h, j in order:
            if left == 0:
                break
            if keep[h].sum() < cap:
                keep[h, j] = True
                left -= 1
        assert np.array_equal(a["keep"], keep)
    nocap = O.allocate(r, 50, f)
    assert np.array_equal(O.allocate(r, 50, f, n)["keep"], nocap["keep"])
    with pytest.raises(ValueError):
        O.allocate(r, H * 8 + 1, f, 8)


def test_allocation_uniform_cap_is_per_cell_top():
    """budget = H * cap forces every cell to keep exactly its floor plus its
    cap - floor best keys (a uniform per-head budget)."""
    rng = np.random.default_rng(910)
    H, n, f, cap = 4, 25, 2, 7
    r = rng.random((H, n))
    a = O.allocate(r, H * cap, f, cap)
    for h in range(H):
        best = np.lexsort((np.arange(n - f), -r[h, : n - f]))[: cap - f]
        assert set(np.nonzero(a["keep"][h, : n - f])[0].tolist()) == set(best.tolist())


@pytest.mark.parametrize("kernel", [1, 3, 7])
def test_maxpool_scores(kernel):
    """Kernel 1 is the identity; otherwise the pooled score equals scipy's
    maximum filter (edge replication adds no new maximum) and bounds the score
    from above."""
    scipy_nd = pytest.importorskip("scipy.ndimage")
    rng = np.random.default_rng(920 + kernel)
    r = rng.random((3, 40))
    out = O.maxpool_scores(r, kernel)
    if kernel == 1:
        assert np.array_equal(out, r)
    ref = scipy_nd.maximum_filter1d(r, size=kernel, axis=1, mode="nearest")
    assert np.array_equal(out, ref)
    assert np.all(out >= r)


# ---------------------------------------------------------------------------
# Free weights: ef, EF and the Frank-Wolfe estimate (Section 2.1, the
# definitions after Definition 2.1; Proposition A.1; the appendix's "Penalty")
# ---------------------------------------------------------------------------

def _frac_vec(xs):
    return np.array([float(Fraction(str(x))) for x in xs])


def test_hull_distance_constructed():
    g = _golden("frank_wolfe.json")
    V = np.array(g["triangle"]["V"], float)
    for c in g["triangle"]["cases"]:
        dist = O.hull_distance(V, _frac_vec(c["mu"]), [0, 1, 2])
        assert dist ** 2 == pytest.approx(float(Fraction(c["dist_sq"])), rel=1e-13, abs=1e-26), c["note"]
    c = g["collinear"]
    V = np.array(c["V"], float)
    assert O.hull_distance(V, _frac_vec(c["mu"]), range(4)) ** 2 == pytest.approx(float(Fraction(c["dist_sq"])), rel=1e-13)


def test_frank_wolfe_example_2_3():
    """Example 2.3: EF(2) = 0 although ES(2) = 9/22, so pi = +inf; EF(1) is the
    distance to the nearest value, 1/2."""
    g = _golden("frank_wolfe.json")["example_2_3"]
    F = lambda x: float(Fraction(x))
    v = np.array(g["v"], float)[:, None]
    p = _frac_vec(g["p"])
    mu = O.dense_output(p, v)
    assert O.exact_free_error(v, mu, range(3), 2) == pytest.approx(F(g["EF_2"]), abs=1e-15)
    assert O.exact_free_error(v, mu, range(3), 1) == pytest.approx(F(g["EF_1"]), rel=1e-13)
    fw1 = O.frank_wolfe(v, mu, range(3), 1, 16)
    assert fw1["ef"] == pytest.approx(F(g["EF_1"]), rel=1e-13) and fw1["support"].tolist() == [1]
    r = O.row_pool(np.log(p), v, g["s"], g["extra"], max_iters=8, fw_iters=16)
    assert r["ef_fw"] <= 1e-15
    assert r["fw_support"].tolist() == g["fw_support_2"]
    assert r["geo_idx"].tolist() == g["geo_2"]
    assert r["es_geo"] == pytest.approx(F(g["es_geo_2"]), rel=1e-13)
    assert r["es_pool"] == pytest.approx(F(g["ES_pool_2"]), rel=1e-13)
    assert r["pi_hat"] > 1e12


def test_geometric_set_pads_in_rank_order():
    g = _golden("frank_wolfe.json")["geo_padding"]
    v = np.array(g["v"], float)[:, None]
    p = _frac_vec(g["p"])
    mu = np.array([float(Fraction(g["mu"]))])
    assert O.dense_output(p, v)[0] == mu[0]  # dyadic: exact
    top = O.top_mass_set(np.log(p), 4)
    assert top.tolist() == g["rank_order"]
    fw = O.frank_wolfe(v, mu, range(4), g["s"], 16)
    assert fw["support"].tolist() == g["fw_support"] and fw["steps"] == g["fw_steps"] and fw["ef"] == 0.0
    geo = O.geometric_set(fw["support"], top, g["s"])
    assert geo.tolist() == g["geo"]
    assert O.forced_error(p, v, geo) == pytest.approx(float(Fraction(g["es_geo"])), rel=1e-13)


@pytest.mark.parametrize("seed", range(4))
def test_free_error_brute_force_and_bounds(seed):
    """On small rows with every key a candidate: EF(s) <= sigma / sqrt(s)
    (Proposition A.1), EF(s) <= ES(s) (es >= ef, Lemma 2.2's proof), EF(d+1) = 0
    (Caratheodory), EF nonincreasing in s, EF(1) = min_j ||v_j - mu||; the
    Frank-Wolfe estimate is an upper bound on EF(s) and exact at s = 1."""
    rng = np.random.default_rng(900 + seed)
    n, d = 6, 1 + seed % 3
    z, p, V = _rand_instance(rng, n, d, temp=1.0 + seed)
    mu = O.dense_output(p, V)
    dev = np.linalg.norm(V - mu, axis=1)
    sigma = math.sqrt(float(np.sum(p * dev ** 2)))
    ef = [O.exact_free_error(V, mu, range(n), s) for s in range(1, n + 1)]
    for s in range(1, n + 1):
        assert ef[s - 1] <= sigma / math.sqrt(s) + 1e-12
        assert ef[s - 1] <= O.best_subset(p, V, s)[1] + 1e-12
        fw = O.frank_wolfe(V, mu, range(n), s, 200)
        assert fw["ef"] >= ef[s - 1] - 1e-12
        assert fw["support"].size <= s and abs(fw["weights"].sum() - 1.0) < 1e-12
        assert np.all(fw["weights"] > 0)
    assert np.all(np.diff(ef) <= 1e-12)
    assert ef[d] <= 1e-12
    assert ef[0] == pytest.approx(dev.min(), rel=1e-13)
    assert O.frank_wolfe(V, mu, range(n), 1, 50)["ef"] == pytest.approx(dev.min(), rel=1e-13)


@pytest.mark.parametrize("seed", range(3))
def test_frank_wolfe_one_dimension_closed_form(seed):
    """d = 1 with every key a candidate: mu lies between the smallest and the
    largest value, and one step from the nearest value toward the farthest
    value on the other side of mu lands on mu, so EF_FW(s) = 0 for s >= 2."""
    rng = np.random.default_rng(950 + seed)
    n = 5 + seed
    z, p, V = _rand_instance(rng, n, 1, temp=2.0)
    mu = O.dense_output(p, V)
    D = float(np.abs(V - mu).max())
    for s in range(2, n + 1):
        fw = O.frank_wolfe(V, mu, range(n), s, 1)
        assert fw["steps"] == 1 and fw["ef"] <= 1e-14 * D
        near = int(np.argmin(np.abs(V[:, 0] - mu[0])))
        far = int(np.argmin(V[:, 0])) if V[near, 0] > mu[0] else int(np.argmax(V[:, 0]))
        assert sorted(fw["support"].tolist()) == sorted([near, far])


@pytest.mark.parametrize("seed", range(3))
def test_frank_wolfe_convergence_rate_and_descent(seed):
    """Without the support cap (s = number of keys) the iterates descend and
    obey the Frank-Wolfe rate with exact line search:
    ||x_t - mu||^2 - dist(mu, hull)^2 <= 4 diam^2 / (t + 2)."""
    rng = np.random.default_rng(980 + seed)
    n, d = 6, 4
    V = rng.standard_normal((n, d))
    mu = rng.standard_normal(d) * (0.3 if seed == 0 else 2.0)  # inside / outside the hull
    dist = O.hull_distance(V, mu, range(n))
    diam = max(np.linalg.norm(V[i] - V[j]) for i in range(n) for j in range(n))
    prev = math.inf
    for t in range(0, 40):
        fw = O.frank_wolfe(V, mu, range(n), n, t)
        e2 = fw["ef"] ** 2
        assert e2 - dist ** 2 <= 4 * diam ** 2 / (t + 2) + 1e-12
        assert fw["ef"] <= prev + 1e-12 and fw["ef"] >= dist - 1e-12
        prev = fw["ef"]


@pytest.mark.parametrize("seed", range(2))
def test_frank_wolfe_permutation(seed):
    """Relabelling the keys relabels the support and keeps EF_FW."""
    rng = np.random.default_rng(990 + seed)
    n, d, s = 8, 5, 3
    z, p, V = _rand_instance(rng, n, d)
    mu = O.dense_output(p, V)
    perm = rng.permutation(n)
    a = O.frank_wolfe(V, mu, range(n), s, 30)
    b = O.frank_wolfe(V[perm], mu, range(n), s, 30)
    assert b["ef"] == pytest.approx(a["ef"], rel=1e-10, abs=1e-14)
    assert sorted(perm[b["support"]].tolist()) == a["support"].tolist()
