// The lockstep revolving-door walk over every k-subset of an instance held
// in LDS (shared by the exhaustive best subset and the candidate-set search).
//
// By Lemma 2.2, es(A)^2 = ||g_A||^2 / p(A)^2 with g_A = sum_{j in A} u_j and
// u_j = p_j (v_j - mu), so ||g_A||^2 = sum_{i,j in A} Gm_ij: a subset is
// scored from Gram entries.  With O the lane's own part and W the walked
// part, against the wave's best ratio beta the test
//     f = S(A) - beta p(A)^2 <= 0
// is linear in the walk:
//     S(A) - beta p(A)^2 = K1 + sum_{x in W} e[x] + S_W - beta p(W)^2,
//     K1 = S_O - beta p(O)^2,   e[x] = 2 sum_{a in O} Gm_xa - 2 beta p(O) p_x,
// so one step is two register reads of e (indexed by the uniform keys), two
// adds, one multiply-add and a compare.  Subsets that pass are scored exactly
// (S / p^2 from the Gram, ties to the lexicographically smaller set), lower
// beta for the wave and rescale e.  Work items (h, a run of up to 64 owned
// parts) are taken by the waves of the workgroup from a shared counter.
//
// With `cpl` the plan enumerates the dropped sets D (k = n - s keys) and the
// scored set is the complement A = U \ D.  With c_x = sum_y Gm_xy and
// D = O + W:
//     S(A) = S_U - 2 c(D) + S(D),   p(A) = p_U - p(D),
// so the test keeps the same linear form in the walked keys:
//     S(A) - beta p(A)^2 = K1 + sum_{x in W} e[x] + S_W - beta p(W)^2,
//     K1 = S_U - 2 c(O) + S_O - beta (p_U - p_O)^2,
//     e[x] = 2 sum_{a in O} Gm_xa - 2 c_x + 2 beta (p_U - p_O) p_x,
// and the walk itself is unchanged: pools that drop a few keys of many walk
// small dropped sets instead of owning large kept parts.
//
// With HT (when the LDS has room), each wave keeps its own copy of the walk
// table's step values at its current beta, T[t] = S_W - beta p(W)^2, rebuilt
// when beta drops, so that a step is one add and a compare.
//
// The test runs at half scale: e, the step values, the base terms and the
// slack are all halved (the walk tables hold S_W / 2 and p(W)^2 / 2), which
// moves no comparison (halving is exact) and saves the doubling of e in
// every lane's set-up.
#pragma once

#include "enum_plan.hpp"

namespace fw {

// Whole workgroup (a multiple of 64 threads); every walked range of the plan
// holds at most WMAX keys.  Gm [n][pl.gp] and ps [n] (LDS,
// float64) hold the instance; seed_mask (block-uniform) is scored first, so
// the answer is never worse than it.  ent [nent] (double2), PLt [nent],
// redd [NT] (double), redm [NT] (uint64) and ctr[1] are LDS scratch.
// Returns the best mask, block-uniform.
// wtab (HT): nent doubles per wave of the workgroup (LDS).
// RD = false: the plan walks no part of more than kColexMax keys (no
// revolving-door walk is compiled).
template <int WMAX, bool HT = false, bool RD = true>
__device__ __forceinline__ uint64_t enum_best_body(const EnumPlan &pl, const double *Gm, const double *ps, uint64_t seed_mask,
                                     const uint2 *__restrict__ g_io, const uint64_t *__restrict__ g_wmk,
                                     const EnumJob *__restrict__ g_jobs, const uint64_t *__restrict__ g_omk,
                                     double2 *ent, double *PLt, double *redd, uint64_t *redm, int *ctr,
                                     bool cpl = false, double *cv = nullptr, double *wtab = nullptr) {
    const int NT = blockDim.x;
    const int gp = pl.gp;
    const int tid = threadIdx.x, lane = tid & 63;
    const uint64_t top_mask = seed_mask;
    const uint64_t allm = pl.n == 64 ? ~0ull : (1ull << pl.n) - 1ull;
    if (cpl)  // Gram row sums c_x (LDS; written before the barrier below)
        for (int x = tid; x < pl.n; x += NT) {
            double c = 0.0;
            for (int y = 0; y < pl.n; ++y) c += Gm[x * gp + y];
            cv[x] = c;
        }
    // per-row walk tables
    for (int t = tid; t < pl.nent; t += NT) {
        const uint64_t lm = g_wmk[t];
        if (lm == kPadMask) {  // neutral step
            ent[t] = make_double2(INFINITY, 0.0);
            PLt[t] = 0.0;
            continue;
        }
        double P = 0.0, S = 0.0;
        for (uint64_t a = lm; a; a &= a - 1) {
            const int x = __ffsll((unsigned long long)a) - 1;
            P += ps[x];
            for (uint64_t b2 = lm; b2; b2 &= b2 - 1) S += Gm[x * gp + (__ffsll((unsigned long long)b2) - 1)];
        }
        ent[t] = make_double2(0.5 * S, 0.5 * (P * P));
        PLt[t] = P;
    }
    if (tid == 0) ctr[0] = 0;
    __syncthreads();
    double SU = 0.0, PU = 0.0;  // S and p of every key (complement walks)
    if (cpl)
        for (int x = 0; x < pl.n; ++x) {
            SU += cv[x];
            PU += ps[x];
        }

    // seed: the top-k set, scored from the Gram
    double S_top = 0.0, P_top = 0.0;
    for (uint64_t a = top_mask; a; a &= a - 1) {
        const int x = __ffsll((unsigned long long)a) - 1;
        P_top += ps[x];
        for (uint64_t b2 = top_mask; b2; b2 &= b2 - 1) S_top += Gm[x * gp + (__ffsll((unsigned long long)b2) - 1)];
    }
    double best_val = S_top / (P_top * P_top);
    uint64_t best_mask = top_mask;
    double beta = best_val;  // wave-uniform
    // HT: the wave's step values at its beta (padding steps stay +inf)
    double *Tw = HT ? wtab + (size_t)(tid >> 6) * pl.nent : nullptr;
    auto build_tw = [&]() __attribute__((always_inline)) {
        if (HT)
            for (int t = lane; t < pl.nent; t += 64) {
                const double2 c = ent[t];
                Tw[t] = fma(-beta, c.y, c.x);
            }
    };
    build_tw();
    // Each wave takes its next work item, and loads that item's descriptor
    // and owned parts, while it walks the current one, so that the global
    // loads of a job start are not waited for between jobs.
    auto take_job = [&]() {
        int j = 0;
        if (lane == 0) j = atomicAdd(ctr, 1);
        return __builtin_amdgcn_readfirstlane(__shfl(j, 0));
    };
    int jn_next = take_job();
    EnumJob jb_next{};
    uint64_t om_next = 0, ok_next = 0;
    const uint64_t *g_okx = g_omk + (size_t)pl.njobs * 64;   // the owned parts' key lists
    if (jn_next < pl.njobs) {
        jb_next = g_jobs[jn_next];
        om_next = g_omk[(size_t)jn_next * 64 + lane];
        ok_next = g_okx[(size_t)jn_next * 64 + lane];
    }
    for (;;) {
        const int jn = jn_next;
        if (jn >= pl.njobs) break;
        const EnumJob jb = jb_next;
        const uint64_t Om = om_next, Ok = ok_next;
        jn_next = take_job();
        if (jn_next < pl.njobs) {
            jb_next = g_jobs[jn_next];
            om_next = g_omk[(size_t)jn_next * 64 + lane];
            ok_next = g_okx[(size_t)jn_next * 64 + lane];
        }
        const EnumClass C = pl.cls[jb.cls];
        const int wb = C.wb, wn = C.wn, ws = C.ws, ls = owned_keys(C);
        const bool act = lane < jb.lanes;
        // owned part of this lane (precomputed key mask; 0 on idle lanes):
        // p(O), S(O) and E[x] = sum_{a in O} Gm_{a, wb + x} over the walked range
        double PO = 0.0, SO = 0.0, CO = 0.0;
        double e[WMAX];
#pragma unroll
        for (int x = 0; x < WMAX; ++x) e[x] = 0.0;
        if (kFastOwned > 1 && ls <= kFastOwned) {
            // the owned keys from the job's key list (a byte each), then
            // independent Gram reads (no loop-carried address chains); idle
            // lanes read key 0
            int kx[kFastOwned];
#pragma unroll
            for (int i = 0; i < kFastOwned; ++i) kx[i] = (int)((Ok >> (8 * i)) & 0xFFu);
#pragma unroll
            for (int i = 0; i < kFastOwned; ++i) {
                if (i < ls) {
                    // (the first key assigns: no adds of zero)
                    const double *ri = Gm + kx[i] * gp;
                    PO = i ? PO + ps[kx[i]] : ps[kx[i]];
                    if (cpl) CO = i ? CO + cv[kx[i]] : cv[kx[i]];
                    double sv = ri[kx[i]];
#pragma unroll
                    for (int j = 0; j < i; ++j) sv = fma(2.0, ri[kx[j]], sv);
                    SO = i ? SO + sv : sv;
                    if (ws > 0) {
                        // all WMAX positions, unguarded: those past the walked
                        // range read neighbouring LDS words and are never used
#pragma unroll
                        for (int x = 0; x < WMAX; ++x) e[x] = i ? e[x] + ri[wb + x] : ri[wb + x];
                    }
                }
            }
        } else {
            for (uint64_t a = Om; a; a &= a - 1) {
                const int x = __ffsll((unsigned long long)a) - 1;
                PO += ps[x];
                if (cpl) CO += cv[x];
                const double *row = Gm + x * gp;
                for (uint64_t b2 = Om; b2; b2 &= b2 - 1) SO += row[__ffsll((unsigned long long)b2) - 1];
                if (ws > 0) {
#pragma unroll
                    for (int y = 0; y < WMAX; ++y) e[y] += row[wb + y];
                }
            }
        }
        // the base (S, p) of the scored set before the walked keys, and the
        // sign of the walked keys' masses in p
        const double PB = cpl ? PU - PO : PO;
        const double SB = cpl ? SU - 2.0 * CO + SO : SO;
        const double sgn = cpl ? 1.0 : -1.0;
        if (ws > 0) {  // e at half scale
            const double bp = sgn * beta * PB;
            if (cpl) {
#pragma unroll
                for (int x = 0; x < WMAX; ++x) e[x] = fma(bp, ps[wb + x], e[x] - cv[wb + x]);
            } else {
#pragma unroll
                for (int x = 0; x < WMAX; ++x) e[x] = fma(bp, ps[wb + x], e[x]);
            }
        }
        const double2 *en = ent + C.toff;
        const double *tw = HT ? Tw + C.toff : nullptr;
        // the step value S_W - beta p(W)^2 of walk step t
        auto stepv = [&](int t) __attribute__((always_inline)) -> double {
            if (HT) return tw[t];
            const double2 c = en[t];
            return fma(-beta, c.y, c.x);
        };
        const double *plt = PLt + C.toff;
        const uint64_t *wmk = g_wmk + C.toff;
        double thr = 0.5e-12 * beta;  // the slack, at half scale
        // exact score of walk step t for this lane (a candidate)
        auto exact = [&](int t) __attribute__((always_inline)) {
            const uint64_t wm = wmk[t];
            double S = SB + 2.0 * en[t].x;
            for (uint64_t a = wm; a; a &= a - 1) {
                const int ax = __ffsll((unsigned long long)a) - 1;
                const double *row = Gm + ax * gp;
                double E = 0.0;
                for (uint64_t b2 = Om; b2; b2 &= b2 - 1) E += row[__ffsll((unsigned long long)b2) - 1];
                S += 2.0 * E;
                if (cpl) S -= 2.0 * cv[ax];
            }
            const double P = cpl ? PB - plt[t] : PO + plt[t];
            const double val = S / (P * P);
            const uint64_t mask = cpl ? (allm & ~(Om | wm)) : (Om | wm);
            if (val < best_val || (val == best_val && lex_less(mask, best_mask))) {
                best_val = val;
                best_mask = mask;
            }
        };
        // after exact scores: the wave's best ratio becomes the new beta;
        // returns the change (0 when none), by which the caller rescales e
        auto lower_beta = [&]() __attribute__((always_inline)) -> double {
            double wbst = best_val;
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) wbst = fmin(wbst, __shfl_xor(wbst, off));
            if (!(wbst < beta)) return 0.0;
            const double dB = wbst - beta;
            beta = wbst;
            thr = 0.5e-12 * beta;
            build_tw();
            return dB;
        };

        if (!RD || (kColexMax >= 0 && ws <= kColexMax)) {
            // Colex walk of the walked part W = {i < j < l}: the outer keys'
            // terms are summed once per run of the innermost key, and the
            // innermost key indexes e at a compile-time position, so a step is
            // one add, one fused multiply-add and a compare.  Consecutive
            // steps of a run differ by one key (i -> i + 1).
            auto run = [&](double base, int t0, int lim) __attribute__((always_inline)) {
                const double nb = thr - base;  // test: e[i] + S_W - beta p(W)^2 <= thr - base
                uint64_t any = 0;
                // chunks of four steps: one batch of table reads per chunk
                // (positions past WMAX are padding steps of the table: skipped)
#pragma unroll
                for (int i0 = 0; i0 < WMAX; i0 += 4) {
                    if (i0 < lim) {
                        double c[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u) c[u] = i0 + u < WMAX ? stepv(t0 + i0 + u) : 0.0;
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            if (i0 + u < WMAX) any |= __ballot(e[i0 + u] + c[u] <= nb);
                    }
                }
                if (any) {  // rare: the same tests again (steps of the run only), exact scores, new beta
                    uint32_t cm = 0;
#pragma unroll
                    for (int i = 0; i < WMAX; ++i) {
                        if (i < lim) {
                            if (e[i] + stepv(t0 + i) <= nb) cm |= 1u << i;
                        }
                    }
                    for (; cm; cm &= cm - 1) exact(t0 + __ffs(cm) - 1);
                    const double dB = lower_beta();
#pragma unroll
                    for (int x = 0; x < WMAX; ++x)
                        e[x] += sgn * dB * PB * ps[wb + x];
                }
            };
            if (ws == 0) {
                const double YO = act ? 0.5 * (SB - beta * PB * PB) : INFINITY;
                if (__ballot(YO <= thr)) {
                    if (YO <= thr) exact(0);
                    lower_beta();  // nothing is walked: e is unused
                }
            } else if (ws == 1) {
                run(act ? 0.5 * (SB - beta * PB * PB) : INFINITY, 0, wn);
            } else {
                // Walked pairs {i < j} below a limit L, after an outer base B
                // (walked triples {i < j < l}: one block per l with
                // B = K1 + e[l], L = l).  Both pair keys index e at
                // compile-time positions.  e at the wave-uniform l comes from
                // selects written out here (a helper taking e by reference
                // would be folded into an indexed load, keeping e out of
                // registers).
                for (int l = ws == 2 ? wn : 2; l < wn || (ws == 2 && l == wn); ++l) {
                    double el = 0.0;
                    if (ws == 3) {
#pragma unroll
                        for (int x = 2; x < WMAX; ++x) el = l == x ? e[x] : el;
                    }
                    const double B = act ? 0.5 * (SB - beta * PB * PB) + el : INFINITY;
                    const int tl = ws == 3 ? l * (l - 1) * (l - 2) / 6 : 0;
                    uint64_t any = 0;
#pragma unroll
                    for (int j = 1; j < WMAX; ++j) {
                        if (j < l) {
                            const double nb = thr - (B + e[j]);
                            const int tj = tl + j * (j - 1) / 2;
#pragma unroll
                            for (int i = 0; i < j; ++i) any |= __ballot(e[i] + stepv(tj + i) <= nb);
                        }
                    }
                    if (any) {  // rare: the same tests again, exact scores, new beta
                        for (int j = 1; j < l; ++j) {
                            double ej = e[1];
#pragma unroll
                            for (int x = 2; x < WMAX; ++x) ej = j == x ? e[x] : ej;
                            const double nb = thr - (B + ej);
                            const int tj = tl + j * (j - 1) / 2;
                            uint32_t cm = 0;
#pragma unroll
                            for (int i = 0; i < WMAX; ++i) {
                                if (i < j) {
                                    if (e[i] + stepv(tj + i) <= nb) cm |= 1u << i;
                                }
                            }
                            for (; cm; cm &= cm - 1) exact(tj + __ffs(cm) - 1);
                        }
                        const double dB = lower_beta();
#pragma unroll
                        for (int x = 0; x < WMAX; ++x)
                            e[x] += sgn * dB * PB * ps[wb + x];
                    }
                }
            }
            continue;
        }
        if constexpr (RD) {
        // Revolving-door walk (walked parts of more than kColexMax keys): one
        // key leaves and one enters per step, both wave-uniform, so e is read
        // at uniform register positions (its own copy: only indexed here).
        double er[WMAX];
#pragma unroll
        for (int x = 0; x < WMAX; ++x) er[x] = e[x];
        double Y = 0.5 * (SB - beta * PB * PB);
#pragma unroll
        for (int x = 0; x < WMAX; ++x)
            if (x < ws) Y += er[x];
        if (!act) Y = INFINITY;
        const uint2 *io = g_io + C.toff;
        const int steps = jb.steps;  // a multiple of 4 (padded with neutral steps)
        // four steps per round: the step tables are loaded together and the
        // rare candidates handled after the four tests (a beta lowered within
        // the round only widens the filter of the remaining steps)
        for (int t0 = 0; t0 < steps; t0 += 4) {
            uint2 w[4];
            double c[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                w[u] = io[t0 + u];
                c[u] = stepv(t0 + u);
            }
            bool cand[4];
            uint64_t any = 0;
            double y = Y;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                y += er[w[u].x] - er[w[u].y];
                const double f = y + c[u];
                cand[u] = f <= thr;
                any |= __ballot(cand[u]);  // wave masks: or-ed on the scalar unit
            }
            Y = y;
            if (any) {  // rare: exact scores, then the wave's new beta
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (cand[u]) exact(t0 + u);
                const double dB = lower_beta();
                if (dB != 0.0) {
#pragma unroll
                    for (int x = 0; x < WMAX; ++x)
                        er[x] += sgn * dB * PB * ps[wb + x];
                    // Y for the round's last real step from the rescaled e
                    int tl = t0 + 3;
                    while (wmk[tl] == kPadMask) --tl;
                    double yy = 0.5 * (SB - beta * PB * PB);
                    for (uint64_t a = wmk[tl]; a; a &= a - 1) yy += er[__ffsll((unsigned long long)a) - 1 - wb];
                    Y = act ? yy : INFINITY;
                }
            }
        }
        }  // RD
    }
    // workgroup argmin with the lexicographic tie rule: within each wave by
    // shuffles, then over the waves
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const double ov = __shfl_xor(best_val, off);
        const uint64_t om = __shfl_xor(best_mask, off);
        if (ov < best_val || (ov == best_val && lex_less(om, best_mask))) {
            best_val = ov;
            best_mask = om;
        }
    }
    if (lane == 0) {
        redd[tid >> 6] = best_val;
        redm[tid >> 6] = best_mask;
    }
    __syncthreads();
    if (tid == 0) {
        for (int i = 1; i < NT / 64; ++i) {
            if (redd[i] < redd[0] || (redd[i] == redd[0] && lex_less(redm[i], redm[0]))) {
                redd[0] = redd[i];
                redm[0] = redm[i];
            }
        }
    }
    __syncthreads();
    const uint64_t best = redm[0];
    __syncthreads();
    return best;
}

}  // namespace fw
