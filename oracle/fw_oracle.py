"""CPU oracle for forced-weight subset evaluation over attention rows.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or run
this module: only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP library and imports none of it.

Every function is a plain, slow, float64 transcription of a definition in
"Trust the Mass: Forced Weights in KV-Cache Eviction" (Shi, Gu; arXiv
2608.25230).  Numbering follows the paper: Section 2.1 (Definition 2.1,
Lemma 2.2, Example 2.3, the balancing selector), Section 2.2 (Definition 2.5),
Section 4 ("ContourKV", "Setup and measured memory"), Appendix A.

Notation map (paper -> here): budget s -> k; kept set A -> S; mass p_j -> p;
mu -> dense output o; m_A -> forced output o_S; es(A) -> gap; 1 - p(A) ->
dropped mass; top-mass set A*_s -> top-k set; balancing selector -> swap rule.

Readings where the paper is silent (each also listed in the design notes):
  * ties in the top-mass set go to the lower key index, and the set is chosen
    on the logits (exp is monotone, so this is the set of largest masses);
  * among best subsets of equal error the lexicographically smallest ascending
    index tuple wins; among equally good swaps the smallest (out, in) pair;
  * the closed fraction is 0 when the top-k error is 0 (nothing to close);
  * the swap rule accepts a swap only on a strict decrease and stops after
    ``max_iters`` swaps;
  * the dropped-mass curve is indexed by the number of kept keys, 0..n, and is
    a suffix sum of the sorted importances;
  * the ContourKV budget counts the recency floor, is exact (ties at the
    threshold broken by (cell, position) ascending) and has no per-cell cap.

Parity status: every function here is pinned by the not-gpu tests against
something other than itself: worked examples of the paper and constructed
instances in exact rationals (tests/golden/), closed forms, Lemma 2.2's
identities, brute force over all subsets, permutation invariance and the
hardness family.  Each pin was checked by planting plausible mistakes in a
copy of this module (tests/test_oracle_mutations.py); no function is
"parity unpinned".
"""
from __future__ import annotations

import functools
import itertools
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# Instance (Definition 2.1): weights of one query row and the dense output
# ----------------------------------------------------------------------------


def logits(q: np.ndarray, K: np.ndarray, scale: float, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Attention logits of query rows ``q`` [..., d] against keys ``K`` [n, d]:
    z_j = scale * <q, k_j> + bias_j.  At an attention head, p is one softmax
    query row (Definition 2.1 and the text after it)."""
    z = float(scale) * (np.asarray(q, np.float64) @ np.asarray(K, np.float64).T)
    if bias is not None:
        z = z + np.asarray(bias, np.float64)
    return z


def weights(z: np.ndarray) -> np.ndarray:
    """Softmax along the last axis: the strictly positive probability vector p
    of Definition 2.1."""
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def dense_output(p: np.ndarray, V: np.ndarray) -> np.ndarray:
    """mu = sum_j p_j v_j, the dense attention output (Definition 2.1)."""
    return np.asarray(p, np.float64) @ np.asarray(V, np.float64)


# ----------------------------------------------------------------------------
# Top-mass set and the forced-weight operator (Definition 2.1)
# ----------------------------------------------------------------------------


def top_mass_set(z: np.ndarray, k: int) -> np.ndarray:
    """A*_k: the k keys of largest mass, in rank order (largest first), ties to
    the lower index.  Ranked on the logits z, which order the masses the same
    way."""
    z = np.asarray(z, np.float64)
    order = np.lexsort((np.arange(z.size), -z))
    return order[:k]


def kept_mass(p: np.ndarray, S: Sequence[int]) -> float:
    """p(S) = sum_{j in S} p_j."""
    return float(np.sum(np.asarray(p, np.float64)[np.asarray(S, np.int64)]))


def dropped_mass(p: np.ndarray, S: Sequence[int]) -> float:
    """pbar(S) = 1 - p(S), summed over the dropped keys themselves."""
    keep = np.zeros(len(p), bool)
    keep[np.asarray(S, np.int64)] = True
    return float(np.sum(np.asarray(p, np.float64)[~keep]))


def forced_output(p: np.ndarray, V: np.ndarray, S: Sequence[int]) -> np.ndarray:
    """m_S = sum_{j in S} (p_j / p(S)) v_j: what a deployed sparse operator
    returns once the kept weights are renormalised (Definition 2.1)."""
    S = np.asarray(S, np.int64)
    pS = np.asarray(p, np.float64)[S]
    return (pS @ np.asarray(V, np.float64)[S]) / pS.sum()


def forced_error(p: np.ndarray, V: np.ndarray, S: Sequence[int]) -> float:
    """es(S) = || mu - m_S ||_2, computed directly from its definition.  When S
    holds every key, m_S = mu exactly (the masses sum to one), so es = 0 rather
    than the rounding residue of two differently ordered sums."""
    if np.unique(np.asarray(S, np.int64)).size == len(p):
        return 0.0
    mu = dense_output(p, V)
    return float(np.linalg.norm(forced_output(p, V, S) - mu))


def row_dense_topk(z: np.ndarray, V: np.ndarray, ks: Sequence[int]) -> Dict[str, np.ndarray]:
    """For one row with logits z and values V: dense output o, and for every
    budget k the top-k set (rank order), forced output o_S, gap ||o_S - o||
    and dropped mass."""
    p = weights(z)
    o = dense_output(p, V)
    kmax = max(ks)
    top = top_mass_set(z, kmax)
    o_s, gap, drop = [], [], []
    for k in ks:
        S = top[:k]
        o_s.append(forced_output(p, V, S))
        gap.append(forced_error(p, V, S))
        drop.append(dropped_mass(p, S))
    return dict(p=p, o=o, o_s=np.array(o_s), gap=np.array(gap), dropped=np.array(drop),
                topk_idx=top)


def dense_topk(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: np.ndarray,
               bias: Optional[np.ndarray], ks: Sequence[int]) -> Dict[str, np.ndarray]:
    """Batched ``row_dense_topk`` over q [H][G][d], K, V [H][n][d]."""
    H, G, d = q.shape
    nk = len(ks)
    out = dict(o=np.zeros((H, G, d)), o_s=np.zeros((nk, H, G, d)), gap=np.zeros((nk, H, G)),
               dropped=np.zeros((nk, H, G)), topk_idx=np.zeros((H, G, max(ks)), np.int64))
    for h in range(H):
        Z = logits(q[h], K[h], scale[h], bias)
        for g in range(G):
            r = row_dense_topk(Z[g], V[h], ks)
            out["o"][h, g] = r["o"]
            out["o_s"][:, h, g] = r["o_s"]
            out["gap"][:, h, g] = r["gap"]
            out["dropped"][:, h, g] = r["dropped"]
            out["topk_idx"][h, g] = r["topk_idx"]
    return out


# ----------------------------------------------------------------------------
# Exhaustive best subset (Section 2.2, Definition 2.5, with the whole row as
# the candidate set) and the closed fraction
# ----------------------------------------------------------------------------


@functools.lru_cache(maxsize=16)
def combinations_table(n: int, k: int) -> np.ndarray:
    """All size-k subsets of range(n), ascending tuples in lexicographic order."""
    return np.array(list(itertools.combinations(range(n), k)), dtype=np.int64).reshape(-1, k)


def subset_errors(p: np.ndarray, V: np.ndarray, combos: np.ndarray, chunk: int = 1 << 15) -> np.ndarray:
    """es(A) for every row A of ``combos`` from the definition: the kept
    numerator sum_{j in A} p_j v_j is an indicator-matrix product."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    mu = p @ V
    pV = p[:, None] * V
    n = p.size
    out = np.empty(len(combos))
    for lo in range(0, len(combos), chunk):
        c = combos[lo:lo + chunk]
        ind = np.zeros((len(c), n))
        np.put_along_axis(ind, c, 1.0, axis=1)
        num = ind @ pV
        den = ind @ p
        out[lo:lo + chunk] = np.linalg.norm(num / den[:, None] - mu, axis=1)
    return out


def best_subset(p: np.ndarray, V: np.ndarray, k: int) -> Tuple[np.ndarray, float]:
    """ES(k) = min over |A| = k of es(A), by exhaustive enumeration in
    lexicographic order; the first minimum (the lexicographically smallest
    tuple) wins exact ties.  Returns (ascending indices, ES)."""
    combos = combinations_table(len(p), k)
    es = subset_errors(p, V, combos)
    i = int(np.argmin(es))
    best = combos[i].copy()
    # report the winner's error through the same evaluator as any other set's
    return best, forced_error(p, V, best)


def closed_fraction(es_top: float, es_best: float) -> float:
    """c = 1 - ES(k)/es(A*_k) (Definition 2.5); 0 when es(A*_k) = 0."""
    if es_top == 0.0:
        return 0.0
    return 1.0 - es_best / es_top


def row_best_subset(z: np.ndarray, V: np.ndarray, k: int) -> Dict[str, object]:
    p = weights(z)
    top = top_mass_set(z, k)
    es_top = forced_error(p, V, top)
    best, es_best = best_subset(p, V, k)
    return dict(best_idx=best, best_gap=es_best, topk_gap=es_top,
                closed=closed_fraction(es_top, es_best), dropped_topk=dropped_mass(p, top),
                topk_idx=top)


# ----------------------------------------------------------------------------
# Swap rule: the balancing selector of Section 2.1
# ----------------------------------------------------------------------------


def swap_values(p: np.ndarray, V: np.ndarray, S: Sequence[int], method: str = "direct"
                ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """es(S - i + j) for every kept key i and dropped key j, as an array
    [|S|][n - |S|] over the kept keys ascending (rows) and the dropped keys
    ascending (columns); returns (values, kept keys, dropped keys).

    ``direct`` evaluates every candidate set from the definition.  ``gform``
    uses Lemma 2.2's second form es(A) = ||g_A|| / p(A) with
    g_A = sum_{j in A} p_j (v_j - mu): ||g - u_i + u_j||^2 expands into norms,
    inner products with g and the cross terms u_i . u_j, taken as one float64
    matrix product."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    n = p.size
    Sin = np.sort(np.asarray(S, np.int64))
    Sout = np.setdiff1d(np.arange(n), Sin)
    if method == "direct":
        cands = [np.sort(np.concatenate([Sin[Sin != i], [j]])) for i in Sin for j in Sout]
        vals = subset_errors(p, V, np.array(cands, np.int64)).reshape(Sin.size, Sout.size)
        return vals, Sin, Sout
    mu = p @ V
    U = p[:, None] * (V - mu)
    g = U[Sin].sum(axis=0)
    P = p[Sin].sum()
    a_in, a_out = U[Sin] @ g, U[Sout] @ g
    b_in, b_out = np.einsum("ij,ij->i", U[Sin], U[Sin]), np.einsum("ij,ij->i", U[Sout], U[Sout])
    cross = U[Sin] @ U[Sout].T
    num = (g @ g) + b_in[:, None] + b_out[None, :] - 2.0 * a_in[:, None] + 2.0 * a_out[None, :] - 2.0 * cross
    den = (P - p[Sin][:, None] + p[Sout][None, :]) ** 2
    return np.sqrt(np.maximum(num, 0.0) / den), Sin, Sout


def _best_swap(p: np.ndarray, V: np.ndarray, S: np.ndarray, method: str) -> Tuple[float, int, int]:
    """(min es over all single swaps, kept key i, dropped key j); ties to the
    smallest (i, j): the first minimum in (i asc, j asc) order."""
    vals, Sin, Sout = swap_values(p, V, S, method)
    t = int(np.argmin(vals))
    i, j = divmod(t, Sout.size)
    return float(vals.flat[t]), int(Sin[i]), int(Sout[j])


def swap_rule(p: np.ndarray, V: np.ndarray, k: int, max_iters: int,
              start: Optional[Sequence[int]] = None, method: str = "auto"
              ) -> Tuple[np.ndarray, np.ndarray, int]:
    """Balancing selector: start at A*_k and repeatedly take the single
    (kept, dropped) swap that most decreases es, stopping when no swap
    decreases it or after ``max_iters`` swaps.  Returns (ascending final set,
    gap trajectory of length max_iters+1 padded with NaN, number of swaps).
    The trajectory holds es of each accepted set, from the definition."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    if start is None:
        z = np.log(p)
        start = top_mass_set(z, k)
    S = np.sort(np.asarray(start, np.int64))
    if method == "auto":
        method = "direct" if p.size <= 32 else "gform"
    traj = np.full(max_iters + 1, np.nan)
    cur = forced_error(p, V, S)
    traj[0] = cur
    it = 0
    if k == 0 or k == p.size:
        return S, traj, 0
    while it < max_iters:
        es_new, i, j = _best_swap(p, V, S, method)
        if not es_new < cur:
            break
        S = np.sort(np.concatenate([S[S != i], [j]]))
        it += 1
        cur = forced_error(p, V, S)
        traj[it] = cur
    return S, traj, it


# ----------------------------------------------------------------------------
# Dropped-mass curve (Definition 2.1's least achievable dropped mass, as a
# function of the budget) over a window-averaged importance score (Section 4)
# ----------------------------------------------------------------------------


def importance(Qw: np.ndarray, K: np.ndarray, scale: float, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Observation-window score: r_j = mean over the window's query rows of the
    softmax weight p_{g,j}."""
    return weights(logits(Qw, K, scale, bias)).mean(axis=0)


def dropped_mass_curve(r: np.ndarray) -> np.ndarray:
    """curve[k] = sum of all but the k largest scores, k = 0..n: the least
    dropped score when keeping k keys.  Summed from the smallest upward."""
    srt = np.sort(np.asarray(r, np.float64))  # ascending
    suffix = np.cumsum(srt)[::-1]  # suffix[k] = sum of the n-k smallest
    return np.concatenate([suffix, [0.0]])


# ----------------------------------------------------------------------------
# ContourKV allocation and ragged storage (Section 4)
# ----------------------------------------------------------------------------


def allocate(r: np.ndarray, budget: int, floor: int, cap: Optional[int] = None) -> Dict[str, object]:
    """One score r and one threshold tau shared by all cells.  Each cell keeps
    its last ``floor`` positions plus its non-floor keys of score >= tau, with
    tau set so that exactly ``budget`` entries are kept in total (floor
    included); ties at tau go to (cell, position) ascending.  With ``cap``
    (budget enforcement), no cell keeps more than ``cap`` entries: each cell
    offers only its cap - floor best non-floor keys (score desc, position
    asc) to the shared threshold."""
    r = np.asarray(r, np.float64)
    H, n = r.shape
    f = min(floor, n)
    quota = budget - H * f
    per_cell = n - f if cap is None else max(0, min(cap, n) - f)
    if quota < 0 or quota > H * per_cell:
        raise ValueError("budget outside [H*floor, H*min(cap, n)]")
    keep = np.zeros((H, n), bool)
    keep[:, n - f:] = True
    cand_h, cand_j = [], []
    for h in range(H):
        js = np.arange(n - f)
        order = np.lexsort((js, -r[h, : n - f]))[:per_cell]
        cand_h.append(np.full(order.size, h))
        cand_j.append(js[order])
    cand_h = np.concatenate(cand_h) if H else np.zeros(0, np.int64)
    cand_j = np.concatenate(cand_j) if H else np.zeros(0, np.int64)
    vals = r[cand_h, cand_j]
    order = np.lexsort((cand_j, cand_h, -vals))[:quota]
    keep[cand_h[order], cand_j[order]] = True
    tau = float(vals[order[-1]]) if quota > 0 else math.inf
    counts = keep.sum(axis=1)
    return dict(keep=keep, counts=counts, tau=tau, quota=quota,
                dropped=np.where(keep, 0.0, r).sum(axis=1))


def maxpool_scores(r: np.ndarray, kernel: int) -> np.ndarray:
    """SnapKV's pooling of the observation-window score (the appendix's audit
    runs it with kernel 7): each position takes the largest score within
    kernel // 2 positions on either side, positions outside the cell
    ignored."""
    r = np.asarray(r, np.float64)
    half = kernel // 2
    n = r.shape[-1]
    out = np.empty_like(r)
    for j in range(n):
        out[..., j] = r[..., max(0, j - half): j + half + 1].max(axis=-1)
    return out


def compact(K: np.ndarray, V: np.ndarray, keep: np.ndarray, heads_per_layer: int,
            elem_bytes: int) -> Dict[str, object]:
    """Physical per-cell eviction stored ragged: each cell's kept rows, in
    ascending position, packed one cell after another, plus the bytes three
    storage layouts hold (ragged, every layer padded to its widest cell, the
    full cache under a mask)."""
    H, n = keep.shape
    d = K.shape[-1]
    counts = keep.sum(axis=1)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    pos = [np.nonzero(keep[h])[0] for h in range(H)]
    kept_pos = np.concatenate(pos).astype(np.int32) if H else np.zeros(0, np.int32)
    K_out = np.concatenate([K[h][pos[h]] for h in range(H)])
    V_out = np.concatenate([V[h][pos[h]] for h in range(H)])
    per_row = 2 * d * elem_bytes  # one K row and one V row
    ragged = int(counts.sum()) * per_row
    L = H // heads_per_layer
    padded = int(sum(counts[l * heads_per_layer:(l + 1) * heads_per_layer].max() for l in range(L))) \
        * heads_per_layer * per_row
    full = H * n * per_row
    return dict(offsets=offsets, kept_pos=kept_pos, k_out=K_out, v_out=V_out,
                bytes_held=np.array([ragged, padded, full], np.int64))


# ----------------------------------------------------------------------------
# Candidate set, ES_pool and the pool-restricted balancing selector
# (Section 2.2, Definition 2.5; the appendix's enumeration protocol), and the
# per-row certificate statistics (Lemma 2.2; Section 2.3 "Dropped mass
# certificate"; the appendix's "Absolute forms")
# ----------------------------------------------------------------------------


def single_key_errors(p: np.ndarray, V: np.ndarray) -> np.ndarray:
    """p_j ||v_j - mu||: the error a key contributes on its own (Definition 2.5)."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    mu = dense_output(p, V)
    return p * np.linalg.norm(V - mu, axis=1)


def candidate_pool(z: np.ndarray, V: np.ndarray, s: int, extra: int) -> Tuple[np.ndarray, np.ndarray]:
    """The candidate set of Definition 2.5: the top-mass set A*_s plus the
    ``extra`` keys outside it of largest single-key error (ties to the lower
    index).  Returns (A*_s in rank order, the extra keys in error order)."""
    z = np.asarray(z, np.float64)
    p = weights(z)
    top = top_mass_set(z, s)
    e = single_key_errors(p, V)
    rest = np.setdiff1d(np.arange(z.size), top)
    order = np.lexsort((rest, -e[rest]))
    return top, rest[order[:extra]]


def pool_subset_errors(p: np.ndarray, V: np.ndarray, combos: np.ndarray, chunk: int = 1 << 15) -> np.ndarray:
    """es(A) from its definition for every row A of ``combos`` (key indices of
    the full row): the masses p_j and the dense output mu are the full row's,
    and m_A renormalises by p(A).  Only the keys that occur in ``combos`` enter
    the kept sums."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    mu = p @ V
    keys = np.unique(combos)
    col = np.searchsorted(keys, combos)
    pk = p[keys]
    pV = pk[:, None] * V[keys]
    out = np.empty(len(combos))
    for lo in range(0, len(combos), chunk):
        c = col[lo:lo + chunk]
        ind = np.zeros((len(c), keys.size))
        np.put_along_axis(ind, c, 1.0, axis=1)
        out[lo:lo + chunk] = np.linalg.norm((ind @ pV) / (ind @ pk)[:, None] - mu, axis=1)
    return out


def pool_best_subset(p: np.ndarray, V: np.ndarray, pool: Sequence[int], s: int) -> Tuple[np.ndarray, float]:
    """ES_pool(s): the exact minimum of es over the size-s subsets of the
    candidate set (Definition 2.5), by enumeration of the pool's keys in
    ascending order; the lexicographically smallest ascending tuple of key
    indices wins exact ties.  Returns (ascending key indices, ES_pool)."""
    keys = np.sort(np.asarray(pool, np.int64))
    combos = keys[combinations_table(keys.size, s)]
    es = pool_subset_errors(p, V, combos)
    best = combos[int(np.argmin(es))].copy()
    return best, forced_error(p, V, best)


def pool_swap(p: np.ndarray, V: np.ndarray, pool: Sequence[int], s: int, max_iters: int,
              start: Sequence[int]) -> Tuple[np.ndarray, np.ndarray, int]:
    """The balancing selector drawing from the candidate set: from ``start``
    (the top-mass set) take the swap of one kept key for one dropped key of
    the pool that most decreases es (ties to the smallest (out, in)), accept
    only a strict decrease, stop after ``max_iters`` swaps.  Returns
    (ascending set, trajectory padded with NaN, number of swaps)."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    pool = np.sort(np.asarray(pool, np.int64))
    S = np.sort(np.asarray(start, np.int64))
    traj = np.full(max_iters + 1, np.nan)
    cur = forced_error(p, V, S)
    traj[0] = cur
    it = 0
    while it < max_iters:
        out_keys = np.setdiff1d(pool, S)
        if out_keys.size == 0:
            break
        cands, pairs = [], []
        for i in S:
            for j in out_keys:
                cands.append(np.sort(np.concatenate([S[S != i], [j]])))
                pairs.append((int(i), int(j)))
        es = pool_subset_errors(p, V, np.array(cands, np.int64))
        t = int(np.argmin(es))
        if not es[t] < cur:
            break
        i, j = pairs[t]
        S = np.sort(np.concatenate([S[S != i], [j]]))
        it += 1
        cur = forced_error(p, V, S)
        traj[it] = cur
    return S, traj, it


# ----------------------------------------------------------------------------
# Free weights (Section 2.1, the definitions after Definition 2.1, and
# Proposition A.1; the appendix's "Penalty" subsection): ef(A) is the distance
# from mu to the convex hull of A's values, EF(s) its least value over size-s
# sets, EF_FW its Frank-Wolfe estimate over the candidate set
# ----------------------------------------------------------------------------


def hull_distance(V: np.ndarray, mu: np.ndarray, S: Sequence[int]) -> float:
    """ef(S) = dist(mu, conv{v_j : j in S}), exactly, by brute force over the
    faces.  The point of the hull nearest mu lies in the relative interior of
    some face and is a positive combination of affinely independent vertices F
    of that face, where it is also the point of aff F nearest mu.  So for every
    nonempty F subset of S take the point of aff F nearest mu (least squares
    with weights summing to one); it is in the hull when its weights are
    nonnegative, and the least distance among those points is ef(S).
    Exponential in |S|: small sets only."""
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
            if w.min() < -1e-12:
                continue
            best = min(best, float(np.linalg.norm(w @ V[list(F)] - mu)))
    return best


def exact_free_error(V: np.ndarray, mu: np.ndarray, keys: Sequence[int], s: int) -> float:
    """EF(s) restricted to ``keys``: the least ef(A) over the size-s subsets A
    of ``keys``.  A larger set only widens the hull, so this is the least
    distance from mu to the hull of at most s of the keys; brute force over
    those faces (small instances only)."""
    keys = [int(j) for j in keys]
    return min(hull_distance(V, mu, F) for F in itertools.combinations(keys, min(s, len(keys))))


def frank_wolfe(V: np.ndarray, mu: np.ndarray, keys: Sequence[int], s: int, max_iters: int) -> Dict[str, object]:
    """The Frank-Wolfe estimate EF_FW of EF(s) over the points v_j, j in
    ``keys``: minimise ||x - mu||^2 over x in their convex hull, holding x as
    weights w over the keys.  Start at the key nearest mu (ties to the lower
    key index).  Each step takes the vertex j minimising the linearised
    objective <v_j, x - mu> (ties to the lower key index) and the duality gap
    <x - mu, x - v_j>; it stops when that gap is not positive, when j would be
    an (s+1)-th key of the support, or after ``max_iters`` steps; otherwise it
    moves to x + eta (v_j - x) with the exact line search
    eta = min(1, gap / ||v_j - x||^2).  Returns ef = ||x - mu|| (an upper bound
    on EF(s) over ``keys``: x lies in the hull of at most s of them), the
    support (keys of positive weight, ascending), the weights and the number of
    steps taken."""
    V = np.asarray(V, np.float64)
    mu = np.asarray(mu, np.float64)
    keys = np.sort(np.asarray(keys, np.int64))
    P = V[keys]
    w = np.zeros(keys.size)
    w[int(np.argmin(np.linalg.norm(P - mu, axis=1)))] = 1.0
    steps = 0
    while steps < max_iters:
        x = w @ P
        r = x - mu
        j = int(np.argmin(P @ r))
        dvec = P[j] - x
        gap = -float(r @ dvec)
        if not gap > 0.0:
            break
        if w[j] == 0.0 and np.count_nonzero(w) >= s:
            break
        eta = min(1.0, gap / float(dvec @ dvec))
        w = (1.0 - eta) * w
        w[j] += eta
        steps += 1
    support = keys[w > 0.0]
    return dict(ef=float(np.linalg.norm(w @ P - mu)), support=support, weights=w[w > 0.0], steps=steps)


def geometric_set(support: Sequence[int], top: Sequence[int], s: int) -> np.ndarray:
    """A^geo_s: the Frank-Wolfe support padded to s keys with the top-mass
    keys it lacks, taken in rank order (appendix, "Penalty").  Ascending."""
    out = [int(j) for j in support]
    for j in top:
        if len(out) >= s:
            break
        if int(j) not in out:
            out.append(int(j))
    return np.sort(np.asarray(out, np.int64))


def certificate(p: np.ndarray, V: np.ndarray, S: Sequence[int]) -> Dict[str, float]:
    """Per-row statistics of a kept set S (the top-mass set in the paper):
    dropped mass pbar(S); Phi = ||g_S|| with g_S = sum_{j in S} p_j (v_j - mu)
    (Lemma 2.2); the radius D = max_j ||v_j - mu||; sigma with
    sigma^2 = sum_j p_j ||v_j - mu||^2; and the two absolute upper bounds on
    es(S): the diameter form 2 D pbar (Lemma 2.2, for the top-mass set) and
    the variance form sqrt(pbar / (1 - pbar)) sigma."""
    p = np.asarray(p, np.float64)
    V = np.asarray(V, np.float64)
    S = np.asarray(S, np.int64)
    mu = dense_output(p, V)
    dev = np.linalg.norm(V - mu, axis=1)
    g = (p[S][:, None] * (V[S] - mu)).sum(axis=0)
    drop = dropped_mass(p, S)
    sigma = float(math.sqrt(float(np.sum(p * dev ** 2))))
    D = float(dev.max())
    var_bound = math.sqrt(drop / (1.0 - drop)) * sigma if drop < 1.0 else math.inf
    return dict(dropped=drop, phi=float(np.linalg.norm(g)), diam=D, sigma=sigma,
                bound_diam=2.0 * D * drop, bound_var=var_bound)


def ratio(num: float, den: float) -> float:
    """num / den for the kappa statistics: 1 when both are 0, +inf when only
    the denominator is."""
    if den > 0.0:
        return num / den
    return 1.0 if num == 0.0 else math.inf


def row_pool(z: np.ndarray, V: np.ndarray, s: int, extra: int, max_iters: int,
             fw_iters: int = 64) -> Dict[str, object]:
    """Everything Definition 2.5 and the enumeration protocol report for one
    row: the candidate set, ES_pool and its argmin, the pool-restricted
    balancing set, kappa_hat = es(A*_s)/ES_pool, c_hat = 1 - ES_pool/es(A*_s),
    kappa_bal = es(A_bal)/ES_pool and the certificate statistics of A*_s;
    and, over the same candidate set, the Frank-Wolfe estimate EF_FW(s)
    (``fw_iters`` steps at most), the geometric set A^geo_s with its error and
    the penalty estimate pi_hat = ES_pool / EF_FW."""
    z = np.asarray(z, np.float64)
    p = weights(z)
    top, extras = candidate_pool(z, V, s, extra)
    pool = np.concatenate([top, extras])
    # every set's error through one evaluator on its ascending indices, so a
    # top-mass set that is also the pool optimum gives c_hat = 0 exactly
    es_top = forced_error(p, V, np.sort(top))
    best, es_pool = pool_best_subset(p, V, pool, s)
    bal, traj, n_swaps = pool_swap(p, V, pool, s, max_iters, top)
    es_bal = forced_error(p, V, bal)
    cert = certificate(p, V, top)
    fw = frank_wolfe(V, dense_output(p, V), pool, s, fw_iters)
    geo = geometric_set(fw["support"], top, s)
    return dict(top=top, extras=extras, best_idx=best, bal_idx=bal, es_top=es_top, es_pool=es_pool,
                es_bal=es_bal, kappa_hat=ratio(es_top, es_pool), c_hat=closed_fraction(es_top, es_pool),
                kappa_bal=ratio(es_bal, es_pool), n_swaps=n_swaps, traj=traj,
                ef_fw=fw["ef"], fw_support=fw["support"], fw_steps=fw["steps"], geo_idx=geo,
                es_geo=forced_error(p, V, geo), pi_hat=ratio(es_pool, fw["ef"]), **cert)


def cell_median(dropped: np.ndarray) -> float:
    """Median dropped mass over a cell's rows (a cell is flat when this, at
    s = 8, exceeds 0.25: Definition 2.5).  An even count averages the two
    middle values."""
    return float(np.median(np.asarray(dropped, np.float64)))


# ----------------------------------------------------------------------------
# Group vote (Section 2.1, the paragraph on deployment's one kept set per KV
# head): the s keys of largest mass summed over the group's rows, and what it
# costs each row against its own top-mass set
# ----------------------------------------------------------------------------


def group_vote(Z: np.ndarray, V: np.ndarray, s: int) -> Dict[str, object]:
    """Z [m][n] holds the logits of the m query rows that share one key/value
    head (the group), V [n][d] its values.  The vote keeps the s keys of
    largest mass summed over the group's rows (ties to the lower index); each
    row is then evaluated with the vote's set under its own forced weights.
    Returns the vote set in rank order and, per row, es(vote), es(A*_s) of the
    row's own top-mass set, their ratio (kappa conventions of ``ratio``) and
    the vote's dropped mass."""
    Z = np.asarray(Z, np.float64)
    P = weights(Z)
    score = P.sum(axis=0)
    vote = np.lexsort((np.arange(score.size), -score))[:s]
    vs = np.sort(vote)
    es_vote, es_top, drop = [], [], []
    for r in range(Z.shape[0]):
        es_vote.append(forced_error(P[r], V, vs))
        es_top.append(forced_error(P[r], V, np.sort(top_mass_set(Z[r], s))))
        drop.append(dropped_mass(P[r], vs))
    es_vote, es_top = np.array(es_vote), np.array(es_top)
    return dict(vote=vote, score=score, es_vote=es_vote, es_top=es_top,
                ratio=np.array([ratio(a, b) for a, b in zip(es_vote, es_top)]), dropped=np.array(drop))
