"""Oracle work for the GPU parity tests, run in worker processes (one BLAS
thread each, up to 16: the host's CPU share per GPU).  Each function takes one
picklable job and returns plain numbers; none touches the GPU."""
import os

import numpy as np
from threadpoolctl import threadpool_limits

from oracle import fw_oracle as O

# The swap kernels search and report in float32: a GPU gap matches an oracle
# value within these relative bounds (float32 sums with cancellation; the
# input dtype's spec tolerance for fp32 rows, tighter than it for bf16).
SWAP_REL = {"f32": 1e-5, "bf16": 1e-4}


def pool_map(fn, jobs, workers=None):
    """fn over jobs in spawned worker processes, results in job order."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor
    n = workers or max(1, min(16, len(os.sched_getaffinity(0)), len(jobs)))
    with ProcessPoolExecutor(max_workers=n, mp_context=mp.get_context("spawn")) as ex:
        return list(ex.map(fn, jobs))


def _bf16(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def classify_swap(job):
    """Replay the balancing selector beside the GPU's trajectory of one row.

    The oracle follows its own best swap at every step; the GPU's next gap
    must equal that swap's value within REL (the float32 search's precision,
    SWAP_REL) for as long as the two paths agree.  A step where two or more
    pairs lie within REL of the best is ambiguous: from there on the GPU may
    have taken another of the tied pairs, and a later mismatch of values, or a
    different final set, makes the row a tie case, whose own final set is
    then checked (its gap, and local optimality if it stopped early).  Without
    an ambiguous step any mismatch fails.  Where the GPU stops before
    max_iters, no swap may improve its gap by more than REL.  Returns
    (status, note) with status exact, tie or fail."""
    z, V, k, iters, gs, gt, gn, method, REL = job
    V = _bf16(V) if V.dtype == np.uint16 else np.asarray(V, np.float64)

    def tie_case(why):
        es_g = O.forced_error(p, V, gs)
        if abs(gt[gn] - es_g) > REL * es_g + 1e-12:
            return "fail", f"tie case ({why}): gpu final gap {gt[gn]} but its set has {es_g}"
        if gn < iters:
            vals, _, _ = O.swap_values(p, V, gs, method)
            if vals.min() < es_g * (1 - REL):
                return "fail", f"tie case ({why}): gpu's final set is not a local optimum ({vals.min()} < {es_g})"
        return "tie", f"{gn} swaps, {why}"

    with threadpool_limits(1):
        p = O.weights(z)
        S = np.sort(O.top_mass_set(z, k))
        cur = O.forced_error(p, V, S)
        if abs(gt[0] - cur) > REL * cur + 1e-12:
            return "fail", f"start gap gpu {gt[0]} oracle {cur}"
        ambiguous = False
        t = 0
        while True:
            if t == iters or t >= gn:
                if t < iters:  # the GPU stopped here: nothing may improve beyond REL
                    vals, _, _ = O.swap_values(p, V, S, method)
                    best = float(vals.min())
                    if best < cur * (1 - REL):
                        if ambiguous:
                            return tie_case(f"paths parted before step {t}")
                        return "fail", f"gpu stopped at step {t}, a swap improves {cur} -> {best}"
                    if best < cur:
                        return tie_case(f"sub-tolerance improvement left at step {t}")
                if np.array_equal(gs, S):
                    return "exact", f"{gn} swaps"
                if ambiguous:
                    return tie_case("same values, another tied set")
                return "fail", f"same trajectory values but a different final set after {t} steps"
            vals, Sin, Sout = O.swap_values(p, V, S, method)
            b = int(np.argmin(vals))
            best = float(vals.flat[b])
            g_next = float(gt[t + 1])
            if not best < cur:  # the oracle stops, the GPU took one more swap
                if g_next < cur * (1 - REL):
                    return "fail", f"oracle stops at step {t} at {cur}, gpu goes on to {g_next}"
                return tie_case(f"gpu took a sub-tolerance swap at step {t}")
            if abs(g_next - best) > REL * best + 1e-12:
                if ambiguous:
                    return tie_case(f"paths parted before step {t}")
                return "fail", f"step {t}: gpu {g_next}, oracle's best swap {best}"
            if int(np.count_nonzero(vals <= best * (1 + REL))) > 1:
                ambiguous = True
            i, j = divmod(b, Sout.size)
            S = np.sort(np.concatenate([Sin[Sin != Sin[i]], [Sout[j]]]))
            cur = O.forced_error(p, V, S)
            t += 1


def local_optimum_margin(job):
    """The float64 error of a final swap set and the least error over its full
    (kept, dropped) neighbourhood (Lemma 2.2's g-form, one sweep)."""
    z, Vb, S, gap_gpu = job
    V = _bf16(Vb) if np.asarray(Vb).dtype == np.uint16 else np.asarray(Vb, np.float64)
    with threadpool_limits(1):
        p = O.weights(z)
        S = np.sort(np.asarray(S, np.int64))
        es_g = O.forced_error(p, V, S)
        vals, _, _ = O.swap_values(p, V, S, "gform")
        return es_g, float(vals.min()), gap_gpu


def dense_topk_unit(job):
    """Worst relative errors and index tallies of one unit's rows against
    row_dense_topk (the rules of tests/parity.py).  Per row and budget, a GPU
    set equal to the oracle's is compared with the oracle's values; a GPU set
    that differs must differ only in keys whose float64 logits tie the
    oracle's within 1e-4 relative (a tie case), and its o_S, gap and dropped
    mass are then compared with the oracle's values for the GPU's own set.
    Returns (worst errors, (exact, tie, fail) rows, where the worst o_S is)."""
    unit, q, Kb, Vb, scale, bias, ks, o, o_s, gap, drop, idx = job
    K, V = _bf16(Kb), _bf16(Vb)
    with threadpool_limits(1):
        Z = O.logits(_bf16(q), K, scale, None if bias is None else np.asarray(bias, np.float64))
        worst = dict(o=0.0, o_s=0.0, gap=0.0, dropped=0.0)
        where = None
        exact = tie = fail = 0
        for g in range(Z.shape[0]):
            r = O.row_dense_topk(Z[g], V, ks)
            p = O.weights(Z[g])
            on = np.linalg.norm(r["o"])
            worst["o"] = max(worst["o"], float(np.linalg.norm(o[g] - r["o"]) / on))
            row_tie = row_fail = False
            for t, k in enumerate(ks):
                ref_os, ref_gap, ref_drop = r["o_s"][t], r["gap"][t], r["dropped"][t]
                if idx is not None:
                    gset, oset = idx[g, :k], r["topk_idx"][:k]
                    if not np.array_equal(np.sort(gset), np.sort(oset)):
                        a, b = np.setdiff1d(gset, oset), np.setdiff1d(oset, gset)
                        zk = Z[g][oset[-1]]
                        if a.size == b.size and np.all(np.abs(Z[g][np.concatenate([a, b])] - zk)
                                                       <= 1e-4 * max(1.0, abs(zk))):
                            row_tie = True
                        else:
                            row_fail = True
                        ref_os = O.forced_output(p, V, gset)
                        ref_gap = O.forced_error(p, V, gset)
                        ref_drop = O.dropped_mass(p, gset)
                e = float(np.linalg.norm(o_s[t, g] - ref_os) / np.linalg.norm(ref_os))
                if e > worst["o_s"]:
                    worst["o_s"], where = e, (unit, g, k, "fail" if row_fail else "tie" if row_tie else "exact")
                worst["gap"] = max(worst["gap"], float(abs(gap[t, g] - ref_gap) / max(ref_gap, 1e-6 * on)))
                worst["dropped"] = max(worst["dropped"], float(abs(drop[t, g] - ref_drop) / max(ref_drop, 1e-6)))
            if idx is not None:
                fail += row_fail
                tie += row_tie and not row_fail
                exact += not (row_tie or row_fail)
        return worst, (exact, tie, fail), where


def pool_row_ref(job):
    """The oracle's candidate-set search of one row (Definition 2.5, the
    balancing selector over the pool and the Frank-Wolfe estimate)."""
    z, Vb, s, extra, max_swaps, fw_iters = job
    V = _bf16(Vb) if np.asarray(Vb).dtype == np.uint16 else np.asarray(Vb, np.float64)
    with threadpool_limits(1):
        return O.row_pool(z, V, s, extra, max_swaps, fw_iters)


def best_subset_rows(job):
    """Exhaustive best subsets of a batch of rows (fp32 inputs) against the
    GPU's: (exact, tie, fail, worst relative error of best_gap, topk_gap,
    closed, dropped_topk)."""
    q, K, V, scale, k, best_idx, best_gap, topk_gap, closed, dtop = job
    with threadpool_limits(1):
        exact = tie = fail = 0
        worst = [0.0, 0.0, 0.0, 0.0]
        for r in range(q.shape[0]):
            z = O.logits(np.asarray(q[r], np.float64), np.asarray(K[r], np.float64), scale[r])
            Vr = np.asarray(V[r], np.float64)
            ref = O.row_best_subset(z, Vr, k)
            p = O.weights(z)
            if np.array_equal(best_idx[r], ref["best_idx"]):
                exact += 1
            elif O.forced_error(p, Vr, best_idx[r]) <= ref["best_gap"] * (1 + 1e-9) + 1e-15:
                tie += 1
            else:
                fail += 1
            floor = 1e-6 * np.linalg.norm(O.dense_output(p, Vr))
            for c, (gv, rv, fl) in enumerate(((best_gap[r], ref["best_gap"], floor), (topk_gap[r], ref["topk_gap"], floor),
                                              (closed[r], ref["closed"], 1.0), (dtop[r], ref["dropped_topk"], 1e-6))):
                worst[c] = max(worst[c], float(abs(gv - rv) / max(abs(rv), fl)))
        return exact, tie, fail, worst


def importance_cell(job):
    """The oracle's window importance (float64) of cell h of the
    curve-and-compaction workload, drawn here from its own seed stream."""
    from paper_2608_25230_amd import workloads as W
    wid, seed, h, G, n, d = job
    r = W.window_rows(wid, seed, 1, G, n, d, W.BF16, with_v=False, first=h)
    with threadpool_limits(1):
        return O.importance(r.as_f64("q")[0], r.as_f64("k")[0], float(r.scale[0]))
