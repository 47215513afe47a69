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
#pragma once

#include "enum_plan.hpp"

namespace fw {

// Whole workgroup (a multiple of 64 threads).  Gm [n][n] and ps [n] (LDS,
// float64) hold the instance; seed_mask (block-uniform) is scored first, so
// the answer is never worse than it.  ent [nent] (double2), PLt [nent],
// redd [NT] (double), redm [NT] (uint64) and ctr[1] are LDS scratch.
// Returns the best mask, block-uniform.
__device__ __forceinline__ uint64_t enum_best_body(const EnumPlan &pl, const double *Gm, const double *ps, uint64_t seed_mask,
                                     const uint2 *__restrict__ g_io, const uint64_t *__restrict__ g_wmk,
                                     const EnumJob *__restrict__ g_jobs, const uint64_t *__restrict__ g_omk,
                                     double2 *ent, double *PLt, double *redd, uint64_t *redm, int *ctr) {
    const int NT = blockDim.x;
    const int n = pl.n;
    const int tid = threadIdx.x, lane = tid & 63;
    const uint64_t top_mask = seed_mask;
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
            for (uint64_t b2 = lm; b2; b2 &= b2 - 1) S += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
        }
        ent[t] = make_double2(S, P * P);
        PLt[t] = P;
    }
    if (tid == 0) ctr[0] = 0;
    __syncthreads();

    // seed: the top-k set, scored from the Gram
    double S_top = 0.0, P_top = 0.0;
    for (uint64_t a = top_mask; a; a &= a - 1) {
        const int x = __ffsll((unsigned long long)a) - 1;
        P_top += ps[x];
        for (uint64_t b2 = top_mask; b2; b2 &= b2 - 1) S_top += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
    }
    double best_val = S_top / (P_top * P_top);
    uint64_t best_mask = top_mask;
    double beta = best_val;  // wave-uniform
    for (;;) {
        int jn = 0;
        if (lane == 0) jn = atomicAdd(ctr, 1);
        jn = __builtin_amdgcn_readfirstlane(__shfl(jn, 0));
        if (jn >= pl.njobs) break;
        const EnumJob jb = g_jobs[jn];
        const EnumClass C = pl.cls[jb.cls];
        const int wb = C.wb, wn = C.wn;
        const bool act = lane < jb.lanes;
        // owned part of this lane (precomputed key mask; 0 on idle lanes)
        const uint64_t Om = g_omk[(size_t)jn * 64 + lane];
        double PO = 0.0, SO = 0.0;
        for (uint64_t a = Om; a; a &= a - 1) {
            const int x = __ffsll((unsigned long long)a) - 1;
            PO += ps[x];
            const double *row = Gm + x * n;
            for (uint64_t b2 = Om; b2; b2 &= b2 - 1) SO += row[__ffsll((unsigned long long)b2) - 1];
        }
        // e[x] over the walked range, from contiguous Gram rows
        double e[kMaxWalk];
#pragma unroll
        for (int x = 0; x < kMaxWalk; ++x) e[x] = 0.0;
        if (C.ws > 0) {
            for (uint64_t a = Om; a; a &= a - 1) {
                const double *row = Gm + (__ffsll((unsigned long long)a) - 1) * n + wb;
#pragma unroll
                for (int x = 0; x < kMaxWalk; ++x)
                    if (x < wn) e[x] += row[x];
            }
#pragma unroll
            for (int x = 0; x < kMaxWalk; ++x)
                if (x < wn) e[x] = 2.0 * e[x] - 2.0 * beta * PO * ps[wb + x];
        }
        double Y = SO - beta * PO * PO;
#pragma unroll
        for (int x = 0; x < kMaxWalk; ++x)
            if (x < C.ws) Y += e[x];
        if (!act) Y = INFINITY;
        const uint2 *io = g_io + C.toff;
        const uint64_t *wmk = g_wmk + C.toff;
        const double2 *en = ent + C.toff;
        const double *plt = PLt + C.toff;
        const int steps = jb.steps;  // a multiple of 4 (padded with neutral steps)
        double thr = 1e-12 * beta;
        // exact score of walk step t for this lane (a candidate)
        auto exact = [&](int t) {
            const uint64_t wm = wmk[t];
            double S = SO + en[t].x;
            for (uint64_t a = wm; a; a &= a - 1) {
                const double *row = Gm + (__ffsll((unsigned long long)a) - 1) * n;
                double E = 0.0;
                for (uint64_t b2 = Om; b2; b2 &= b2 - 1) E += row[__ffsll((unsigned long long)b2) - 1];
                S += 2.0 * E;
            }
            const double P = PO + plt[t];
            const double val = S / (P * P);
            const uint64_t mask = Om | wm;
            if (val < best_val || (val == best_val && lex_less(mask, best_mask))) {
                best_val = val;
                best_mask = mask;
            }
        };
        // four steps per round: the step tables are loaded together and the
        // rare candidates handled after the four tests (a beta lowered within
        // the round only widens the filter of the remaining steps)
        for (int t0 = 0; t0 < steps; t0 += 4) {
            uint2 w[4];
            double2 c[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                w[u] = io[t0 + u];
                c[u] = en[t0 + u];
            }
            bool cand[4];
            uint64_t any = 0;
            double y = Y;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                y += e[w[u].x] - e[w[u].y];
                const double f = y + fma(-beta, c[u].y, c[u].x);
                cand[u] = f <= thr;
                any |= __ballot(cand[u]);  // wave masks: or-ed on the scalar unit
            }
            Y = y;
            if (any) {  // rare: exact scores, then the wave's new beta
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (cand[u]) exact(t0 + u);
                double wbst = best_val;
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) wbst = fmin(wbst, __shfl_xor(wbst, off));
                if (wbst < beta) {
                    const double dB = wbst - beta;
#pragma unroll
                    for (int x = 0; x < kMaxWalk; ++x)
                        if (x < wn) e[x] -= 2.0 * dB * PO * ps[wb + x];
                    beta = wbst;
                    thr = 1e-12 * beta;
                    // Y for the round's last real step from the rescaled e
                    int tl = t0 + 3;
                    while (wmk[tl] == kPadMask) --tl;
                    double yy = SO - beta * PO * PO;
                    for (uint64_t a = wmk[tl]; a; a &= a - 1) yy += e[__ffsll((unsigned long long)a) - 1 - wb];
                    Y = act ? yy : INFINITY;
                }
            }
        }
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

// The same walk, inlined or called at the compiler's choice (the candidate-set
// kernel, whose row phase already holds many registers); the exhaustive
// kernel calls the body inlined, which keeps it at four waves per SIMD.
__device__ inline uint64_t enum_best(const EnumPlan &pl, const double *Gm, const double *ps, uint64_t seed_mask,
                                     const uint2 *__restrict__ g_io, const uint64_t *__restrict__ g_wmk,
                                     const EnumJob *__restrict__ g_jobs, const uint64_t *__restrict__ g_omk,
                                     double2 *ent, double *PLt, double *redd, uint64_t *redm, int *ctr) {
    return enum_best_body(pl, Gm, ps, seed_mask, g_io, g_wmk, g_jobs, g_omk, ent, PLt, redd, redm, ctr);
}

}  // namespace fw
