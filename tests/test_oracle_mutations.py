"""Planted mistakes in the oracle must fail at least one pin.

Each mutant replaces one oracle function with a plausible error (dropped
renormalisation, wrong tie direction, wrong sign, argmax for argmin, prefix in
place of suffix, Phi reported for es, one budget's set used for every budget,
an inverted ratio, a non-strict stopping rule, ...) and runs the pins that
should catch it.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import fw_oracle as O
from tests import test_oracle_pins as P


def _fails(fn, *args):
    try:
        fn(*args)
    except (AssertionError, ValueError, IndexError):
        return True
    return False


def _run_all_pins():
    """True if any pin fails under the current (mutated) oracle."""
    checks = [
        (P.test_example_2_3_values,), (P.test_example_2_3_swap_rule,),
        (P.test_example_A3_table_and_tie_rule,), (P.test_example_A3_not_submodular_statements,),
        (P.test_hardness_all_pairs_tie,), (P.test_softmax_closed_form_and_shift,),
        (P.test_compaction_and_bytes,), (P.test_dense_topk_batch_consistency,),
    ]
    checks += [(P.test_hardness_family_exact, s) for s in range(4)]
    checks += [(P.test_lemma_2_2_identities, s) for s in range(3)]
    checks += [(P.test_closed_forms, s) for s in range(3)]
    checks += [(P.test_top_mass_brute_force, s) for s in range(3)]
    checks += [(P.test_swap_rule_invariants, s) for s in range(3)]
    checks += [(P.test_dropped_mass_curve, s) for s in range(3)]
    checks += [(P.test_allocation, s) for s in range(3)]
    checks += [(P.test_pool_example_2_3,), (P.test_cell_median,)]
    checks += [(P.test_pool_brute_force, s) for s in range(4)]
    checks += [(P.test_pool_of_every_key_is_the_full_search, s) for s in range(3)]
    checks += [(P.test_pool_swap_invariants, s) for s in range(3)]
    checks += [(P.test_certificate_identities_and_bounds, s) for s in range(3)]
    checks += [(P.test_group_vote_of_one_row_is_its_top_mass_set, s) for s in range(3)]
    checks += [(P.test_group_vote_brute_force, s) for s in range(3)]
    checks += [(P.test_allocation_with_cap, s) for s in range(3)]
    checks += [(P.test_allocation_uniform_cap_is_per_cell_top,)]
    checks += [(P.test_maxpool_scores, k) for k in (1, 3, 7)]
    checks += [(P.test_row_dense_topk_example_2_3,), (P.test_row_best_subset_example_2_3,),
               (P.test_balancing_stops_at_a_local_optimum,), (P.test_swap_rule_stops_on_a_tie,),
               (P.test_swap_values_example_2_3,)]
    checks += [(P.test_row_dense_topk_per_budget_first_form, s) for s in range(4)]
    checks += [(P.test_hull_distance_constructed,), (P.test_frank_wolfe_example_2_3,),
               (P.test_geometric_set_pads_in_rank_order,)]
    checks += [(P.test_free_error_brute_force_and_bounds, s) for s in range(4)]
    checks += [(P.test_frank_wolfe_one_dimension_closed_form, s) for s in range(3)]
    checks += [(P.test_frank_wolfe_convergence_rate_and_descent, s) for s in range(3)]
    checks += [(P.test_frank_wolfe_permutation, s) for s in range(2)]
    return any(_fails(*c) for c in checks)


def _no_renorm(p, V, S):
    S = np.asarray(S, np.int64)
    return np.asarray(p)[S] @ np.asarray(V)[S]


def _ties_high(z, k):
    z = np.asarray(z, np.float64)
    return np.lexsort((-np.arange(z.size), -z))[:k]


def _dropped_is_kept(p, S):
    return O.kept_mass(p, S)


def _neg_softmax(z):
    z = -np.asarray(z, np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def _argmax_best(p, V, k):
    combos = O.combinations_table(len(p), k)
    es = O.subset_errors(p, V, combos)
    i = int(np.argmax(es))
    return combos[i].copy(), float(es[i])


def _ratio_closed(es_top, es_best):
    return 0.0 if es_top == 0 else es_best / es_top


def _prefix_curve(r):
    srt = np.sort(np.asarray(r, np.float64))[::-1]
    return np.concatenate([[0.0], np.cumsum(srt)])


def _no_bias_logits(q, K, scale, bias=None):
    return float(scale) * (np.asarray(q, np.float64) @ np.asarray(K, np.float64).T)


def _gap_transposed(p, V, S):
    # mixes up keys and dimensions of V: uses the first |S| columns
    S = np.asarray(S, np.int64)
    mu = np.asarray(p) @ np.asarray(V)
    pS = np.asarray(p)[S]
    m = (pS @ np.asarray(V)[S]) / pS.sum()
    return float(np.linalg.norm(m - mu) + abs(m[0] - mu[0]))


def _alloc_ties_high(r, budget, floor):
    r = np.asarray(r, np.float64)
    H, n = r.shape
    f = min(floor, n)
    quota = budget - H * f
    if quota < 0 or quota > H * (n - f):
        raise ValueError("budget")
    keep = np.zeros((H, n), bool)
    keep[:, n - f:] = True
    hh, jj = np.meshgrid(np.arange(H), np.arange(n - f), indexing="ij")
    hh, jj = hh.ravel(), jj.ravel()
    vals = r[:, : n - f].ravel()
    order = np.lexsort((-jj, -hh, -vals))[:quota]
    keep[hh[order], jj[order]] = True
    tau = float(vals[order[-1]]) if quota > 0 else np.inf
    return dict(keep=keep, counts=keep.sum(1), tau=tau, quota=quota,
                dropped=np.where(keep, 0.0, r).sum(1))


def _extras_by_mass(z, V, s, extra):
    z = np.asarray(z, np.float64)
    top = O.top_mass_set(z, s)
    rest = np.setdiff1d(np.arange(z.size), top)
    return top, rest[np.lexsort((rest, -z[rest]))[:extra]]


def _extras_may_repeat_top(z, V, s, extra):
    z = np.asarray(z, np.float64)
    e = O.single_key_errors(O.weights(z), V)
    allk = np.arange(z.size)
    return O.top_mass_set(z, s), allk[np.lexsort((allk, -e))[:extra]]


def _pool_renormalised(p, V, pool, s):
    keys = np.sort(np.asarray(pool, np.int64))
    q = np.asarray(p)[keys] / np.asarray(p)[keys].sum()
    Vk = np.asarray(V)[keys]
    best, es = O.best_subset(q, Vk, s)
    return keys[best], es


def _sigma_unweighted(p, V, S):
    c = _ORIG_CERT(p, V, S)
    mu = np.asarray(p) @ np.asarray(V)
    c["sigma"] = float(np.sqrt(np.mean(np.linalg.norm(np.asarray(V) - mu, axis=1) ** 2)))
    return c


def _var_bound_inverted(p, V, S):
    c = _ORIG_CERT(p, V, S)
    m = c["dropped"]
    c["bound_var"] = float(np.sqrt((1 - m) / m) * c["sigma"]) if m > 0 else np.inf
    return c


_ORIG_CERT = O.certificate


def _vote_by_max(Z, V, s):
    # votes on the largest single-row mass instead of the summed mass
    Z = np.asarray(Z, np.float64)
    P = O.weights(Z)
    score = P.max(axis=0)
    vote = np.lexsort((np.arange(score.size), -score))[:s]
    r = _ORIG_VOTE(Z, V, s)
    r["vote"] = vote
    vs = np.sort(vote)
    r["es_vote"] = np.array([O.forced_error(P[i], V, vs) for i in range(Z.shape[0])])
    return r


_ORIG_VOTE = O.group_vote


def _cap_counts_floor_twice(r, budget, floor, cap=None):
    # caps the non-floor part at cap instead of cap - floor
    return _ORIG_ALLOC(r, budget, floor, None if cap is None else cap + floor)


def _maxpool_one_sided(r, kernel):
    r = np.asarray(r, np.float64)
    out = np.empty_like(r)
    for j in range(r.shape[-1]):
        out[..., j] = r[..., j: j + kernel].max(axis=-1)
    return out


_ORIG_ALLOC = O.allocate
_ORIG_ROW_DENSE = O.row_dense_topk
_ORIG_ROW_BEST = O.row_best_subset
_ORIG_ROW_POOL = O.row_pool


def _dense_gap_times_kept_mass(z, V, ks):
    # reports Phi = p(S) es(S) instead of es(S)
    r = _ORIG_ROW_DENSE(z, V, ks)
    r["gap"] = r["gap"] * (1.0 - r["dropped"])
    return r


def _dense_kmax_set_for_every_budget(z, V, ks):
    # evaluates every budget on the largest budget's set
    r = _ORIG_ROW_DENSE(z, V, ks)
    i = int(np.argmax(ks))
    for t in range(len(ks)):
        r["o_s"][t], r["gap"][t], r["dropped"][t] = r["o_s"][i], r["gap"][i], r["dropped"][i]
    return r


def _best_dropped_is_kept(z, V, k):
    r = _ORIG_ROW_BEST(z, V, k)
    r["dropped_topk"] = 1.0 - r["dropped_topk"]
    return r


def _pool_kappa_bal_inverted(z, V, s, extra, max_iters, fw_iters=64):
    r = _ORIG_ROW_POOL(z, V, s, extra, max_iters, fw_iters)
    r["kappa_bal"] = O.ratio(r["es_pool"], r["es_bal"])
    return r


def _swap_non_strict(p, V, k, max_iters, start=None, method="auto"):
    # accepts a swap that only ties the current error
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    if start is None:
        start = O.top_mass_set(np.log(p), k)
    S = np.sort(np.asarray(start, np.int64))
    method = "direct" if (method == "direct" or (method == "auto" and p.size <= 32)) else "gform"
    traj = np.full(max_iters + 1, np.nan)
    cur = O.forced_error(p, V, S)
    traj[0] = cur
    it = 0
    if k == 0 or k == p.size:
        return S, traj, 0
    while it < max_iters:
        es_new, i, j = O._best_swap(p, V, S, method)
        if not es_new <= cur:
            break
        S = np.sort(np.concatenate([S[S != i], [j]]))
        it += 1
        cur = O.forced_error(p, V, S)
        traj[it] = cur
    return S, traj, it

_ORIG_FW = O.frank_wolfe
_ORIG_HULL = O.hull_distance
_ORIG_ROW_POOL_FW = O.row_pool


def _fw_variant(vertex="argmin", step="square", start="nearest", cap=0):
    def fw(V, mu, keys, s, max_iters):
        V = np.asarray(V, np.float64)
        mu = np.asarray(mu, np.float64)
        keys = np.sort(np.asarray(keys, np.int64))
        P = V[keys]
        w = np.zeros(keys.size)
        w[0 if start == "first" else int(np.argmin(np.linalg.norm(P - mu, axis=1)))] = 1.0
        steps = 0
        while steps < max_iters:
            x = w @ P
            r = x - mu
            j = int(np.argmin(P @ r)) if vertex == "argmin" else int(np.argmax(P @ r))
            dvec = P[j] - x
            gap = -float(r @ dvec)
            if vertex == "argmin" and not gap > 0.0:
                break
            if w[j] == 0.0 and np.count_nonzero(w) >= s + cap:
                break
            nrm = float(dvec @ dvec)
            if nrm == 0.0:
                break
            eta = min(1.0, gap / (nrm if step == "square" else math.sqrt(nrm)))
            if vertex != "argmin":
                eta = min(1.0, abs(eta))
            w = (1.0 - eta) * w
            w[j] += eta
            steps += 1
        return dict(ef=float(np.linalg.norm(w @ P - mu)), support=keys[w > 0.0], weights=w[w > 0.0], steps=steps)
    return fw


def _hull_negative_weights(V, mu, S):
    # accepts affine projections outside the hull
    V = np.asarray(V, np.float64)
    mu = np.asarray(mu, np.float64)
    S = [int(j) for j in S]
    best = math.inf
    for size in range(1, len(S) + 1):
        for F in itertools.combinations(S, size):
            v0 = V[F[0]]
            if size == 1:
                w = np.ones(1)
            else:
                B = (V[list(F[1:])] - v0).T
                t = np.linalg.lstsq(B, mu - v0, rcond=None)[0]
                w = np.concatenate([[1.0 - t.sum()], t])
            best = min(best, float(np.linalg.norm(w @ V[list(F)] - mu)))
    return best


def _exact_free_one_fewer(V, mu, keys, s):
    keys = [int(j) for j in keys]
    m = max(1, min(s, len(keys)) - 1)
    return min(O.hull_distance(V, mu, F) for F in itertools.combinations(keys, m))


def _geo_pads_ascending(support, top, s):
    out = [int(j) for j in support]
    for j in sorted(int(t) for t in top):
        if len(out) >= s:
            break
        if j not in out:
            out.append(j)
    return np.sort(np.asarray(out, np.int64))


def _pool_pi_inverted(z, V, s, extra, max_iters, fw_iters=64):
    r = _ORIG_ROW_POOL_FW(z, V, s, extra, max_iters, fw_iters)
    r["pi_hat"] = O.ratio(r["ef_fw"], r["es_pool"])
    return r


MUTANTS = {
    "frank_wolfe_vertex_argmax": ("frank_wolfe", _fw_variant(vertex="argmax")),
    "frank_wolfe_step_over_norm": ("frank_wolfe", _fw_variant(step="norm")),
    "frank_wolfe_starts_at_first_key": ("frank_wolfe", _fw_variant(start="first")),
    "frank_wolfe_support_cap_plus_one": ("frank_wolfe", _fw_variant(cap=1)),
    "hull_distance_negative_weights": ("hull_distance", _hull_negative_weights),
    "exact_free_error_one_key_fewer": ("exact_free_error", _exact_free_one_fewer),
    "geometric_set_pads_ascending": ("geometric_set", _geo_pads_ascending),
    "pool_pi_hat_inverted": ("row_pool", _pool_pi_inverted),
    "group_vote_by_max_mass": ("group_vote", _vote_by_max),
    "allocation_cap_ignores_floor": ("allocate", _cap_counts_floor_twice),
    "maxpool_one_sided_window": ("maxpool_scores", _maxpool_one_sided),
    "pool_extras_by_mass": ("candidate_pool", _extras_by_mass),
    "pool_extras_repeat_top": ("candidate_pool", _extras_may_repeat_top),
    "pool_renormalised_within_pool": ("pool_best_subset", _pool_renormalised),
    "certificate_sigma_unweighted": ("certificate", _sigma_unweighted),
    "certificate_variance_bound_inverted": ("certificate", _var_bound_inverted),
    "forced_output_without_renormalisation": ("forced_output", _no_renorm),
    "top_mass_ties_to_higher_index": ("top_mass_set", _ties_high),
    "dropped_mass_is_kept_mass": ("dropped_mass", _dropped_is_kept),
    "softmax_sign_flip": ("weights", _neg_softmax),
    "best_subset_argmax": ("best_subset", _argmax_best),
    "closed_fraction_as_ratio": ("closed_fraction", _ratio_closed),
    "curve_as_prefix_sum": ("dropped_mass_curve", _prefix_curve),
    "logits_drop_bias": ("logits", _no_bias_logits),
    "gap_extra_term": ("forced_error", _gap_transposed),
    "allocation_ties_high": ("allocate", _alloc_ties_high),
    "dense_topk_gap_times_kept_mass": ("row_dense_topk", _dense_gap_times_kept_mass),
    "dense_topk_kmax_set_for_every_budget": ("row_dense_topk", _dense_kmax_set_for_every_budget),
    "best_subset_dropped_is_kept": ("row_best_subset", _best_dropped_is_kept),
    "pool_kappa_bal_inverted": ("row_pool", _pool_kappa_bal_inverted),
    "swap_rule_non_strict_stop": ("swap_rule", _swap_non_strict),
}


def test_unmutated_oracle_passes_all_pins():
    assert not _run_all_pins()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(O, attr, fn)
    assert _run_all_pins(), f"no pin catches mutant {name}"
