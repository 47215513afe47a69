// Candidate-set search over long attention rows (Section 2.2, Definition 2.5,
// and the appendix's enumeration protocol), float64 throughout.
//
// One workgroup per row:
//   1. the whole row: logits z_j, weights p = softmax(z), dense output mu,
//      deviations ||v_j - mu||, single-key errors p_j ||v_j - mu||, the
//      radius D = max_j ||v_j - mu|| and sigma^2 = sum_j p_j ||v_j - mu||^2
//      (groups of lanes per key, whole key rows per load);
//   2. the candidate set: the top-mass set A*_s (logit desc, index asc) and
//      the `extra` keys outside it of largest single-key error (error desc,
//      index asc), each by s (extra) rounds of a workgroup argmax;
//   3. the pool instance in LDS: masses, values and the Gram matrix of
//      u_i = p_i (v_i - mu) over the pool's keys in ascending key order, with
//      the full row's p and mu (es is the full row's error);
//   4. ES_pool: every s-subset of the pool by the lockstep revolving-door walk
//      shared with the exhaustive best subset, seeded by A*_s -- in a kernel
//      of its own (pool_enum_kernel, four workgroups per CU), to which the
//      row kernel hands each pool's instance through the workspace; pools
//      that drop fewer than four keys are enumerated in the row kernel;
//   5. the balancing selector drawing from the pool: every (kept, dropped)
//      pair of the pool scored from the Gram each round, ties to the smallest
//      (out, in) key pair, accepted only on a strict decrease;
//   6. the reported errors of A*_s, the ES_pool argmin and the balancing set
//      from d-dimensional residual sums, and the certificate statistics;
//   7. beside the balancing (another wave), the Frank-Wolfe estimate of the
//      free-weight error EF(s) over the pool's values (Section 2.1's ef and
//      EF; the appendix's penalty estimate), run on the Gram matrix of the
//      deviations v_i - mu and reported from a d-dimensional sum, with the
//      geometric set (its support padded with top-mass keys in rank order).
// The enumeration kernel also takes the ES_pool set's reported error and the
// statistics that depend on it.  A last kernel takes each cell's median
// dropped mass over its rows.
#include "fw_internal.hpp"
#include "instance64.hpp"
#include "enum_walk.hpp"
#include "rowpass.hpp"

namespace fw {

namespace {

constexpr int PT = 256;       // threads per row workgroup
constexpr int kPoolMax = 64;  // pool keys (one 64-bit mask)

constexpr int kMaxBudgets = FW_POOL_MAX_BUDGETS;

struct PoolLds {
    size_t xq, mu, red, ctr, rank, eord, tmp, plist, pps, sc, seed;  // persistent
    size_t zz, ee, rk;                                   // row phase
    size_t gm, vs, cv, yd, wf;                           // pool phase (overlays the row phase)
    size_t total;
};

// The pool phase is sized for the largest pool (Pmax keys) of the call's
// budgets (the walks, with their tables, run in the enumeration kernel).
__host__ __device__ inline PoolLds pool_lds(int64_t N, int d, int Pmax) {
    PoolLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.xq = take((size_t)d * 8);
    L.mu = take((size_t)d * 8);
    L.red = take((size_t)PT * 16);
    L.ctr = take(16);
    L.rank = take((size_t)kPoolMax * 4);                // top keys in rank order
    L.eord = take((size_t)kPoolMax * 4);                // keys of largest single-key error, in order
    L.tmp = take((size_t)kPoolMax * 4);                 // a pool in output order
    L.plist = take((size_t)kMaxBudgets * kPoolMax * 4);  // each pool, ascending keys
    L.pps = take((size_t)kMaxBudgets * kPoolMax * 8);    // their masses
    L.sc = take((size_t)(kMaxBudgets + 2) * 8);
    L.seed = take((size_t)kMaxBudgets * 8);        // each A*_s as a pool mask
    const size_t base = o;
    L.zz = base;
    L.ee = align_up(L.zz + (size_t)N * 8, 16);
    L.rk = align_up(L.ee + (size_t)N * 8, 16);
    const size_t row_end = L.rk + (size_t)N;
    L.gm = base;
    L.vs = align_up(L.gm + (size_t)Pmax * Pmax * 8, 16);
    L.cv = align_up(L.vs + (size_t)Pmax * (d + 1) * 4, 16);
    L.yd = align_up(L.cv + (size_t)Pmax * 8, 16);      // Gram matrix of v_i - mu
    L.wf = align_up(L.yd + (size_t)Pmax * Pmax * 8, 16);  // Frank-Wolfe weights
    const size_t pool_end = L.wf + (size_t)Pmax * 8;
    L.total = align_up(row_end > pool_end ? row_end : pool_end, 16);
    return L;
}

// Pools that drop fewer than kWalkDrop keys are enumerated through the
// dropped set in the row kernel (enum_complement): a walk's owned parts would
// hold nearly every key.  Pools dropping kWalkDrop or more are walked by the
// enumeration kernel; those dropping at most kDirectDrop keys fall back to
// the dropped-set enumeration when no walk plan exists.  (Measured: the
// paper's (32, 4) pool through the enumeration kernel's dropped-set walk cut
// the four budgets from 9.54 to 8.91 ms.)
constexpr int kDirectDrop = 4;
constexpr int kWalkDrop = 4;

// Every s-subset A of the pool as the complement of a dropped set D of
// q = P - s keys: with c_i = sum_j Gm_ij over the pool, S_U = sum_i c_i and
// p_U = p(pool), ||g_A||^2 = S_U - 2 sum_{i in D} c_i + sum_{i,j in D} Gm_ij
// and p(A) = p_U - p(D).  The colex ranks of D are split into one run per
// thread, each stepping to the next mask of the same size; ties go to the
// lexicographically smallest A.  Returns A's mask, block-uniform.
__device__ inline uint64_t enum_complement(const double *Gm, const double *ps, int P, int q, double *cv,
                                           double *redd, uint64_t *redm) {
    const int tid = threadIdx.x, NT = blockDim.x, lane = tid & 63, w = tid >> 6;
    const uint64_t all = P == 64 ? ~0ull : ((1ull << P) - 1ull);
    if (q == 0) return all;
    for (int x = tid; x < P; x += NT) {
        double c = 0.0;
        for (int y = 0; y < P; ++y) c += Gm[x * P + y];
        cv[x] = c;
    }
    __syncthreads();
    double SU = 0.0, pU = 0.0;
    for (int x = 0; x < P; ++x) {
        SU += cv[x];
        pU += ps[x];
    }
    const uint64_t total = binom(P, q);
    const uint64_t lo = total * (uint64_t)tid / (uint64_t)NT, hi = total * (uint64_t)(tid + 1) / (uint64_t)NT;
    double best = INFINITY;
    uint64_t bestA = 0;
    if (lo < hi) {
        // unrank lo (combinatorial number system, colex)
        uint64_t D = 0, rr = lo;
        int c = P - 1;
        for (int sz = q; sz >= 1; --sz) {
            while (binom(c, sz) > rr) --c;
            D |= 1ull << c;
            rr -= binom(c, sz);
            --c;
        }
        // the keys of D in registers, every term from independent reads;
        // against the thread's best ratio beta the test S - beta p(A)^2 <= 0
        // is one fused multiply-add, and only passing sets take the division
        double beta = INFINITY;
        for (uint64_t r = lo; r < hi; ++r) {
            int kd[kDirectDrop];
            uint64_t m = D;
#pragma unroll
            for (int x = 0; x < kDirectDrop; ++x) {
                kd[x] = m ? __ffsll((unsigned long long)m) - 1 : 0;
                m &= m - 1;
            }
            double S = SU, pD = 0.0;
#pragma unroll
            for (int x = 0; x < kDirectDrop; ++x) {
                if (x < q) {
                    const double *rx = Gm + kd[x] * P;
                    pD += ps[kd[x]];
                    double t = rx[kd[x]] - 2.0 * cv[kd[x]];
#pragma unroll
                    for (int y = 0; y < x; ++y) t = fma(2.0, rx[kd[y]], t);
                    S += t;
                }
            }
            const double PA = pU - pD;
            if (!(fma(-beta, PA * PA, fmax(S, 0.0)) <= 1e-12 * beta) && beta < INFINITY) {
                const uint64_t u = D & (~D + 1ull), v = D + u;
                D = v | (((v ^ D) >> 2) >> (__ffsll((unsigned long long)D) - 1));
                continue;
            }
            const double val = fmax(S, 0.0) / (PA * PA);
            const uint64_t A = all & ~D;
            if (val < best || (val == best && lex_less(A, bestA))) {
                best = val;
                bestA = A;
                beta = val;
            }
            // next mask of the same size (colex successor)
            const uint64_t u = D & (~D + 1ull), v = D + u;
            D = v | (((v ^ D) >> 2) >> (__ffsll((unsigned long long)D) - 1));
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        const double ov = __shfl_xor(best, off);
        const uint64_t om = __shfl_xor(bestA, off);
        if (ov < best || (ov == best && om != 0 && (bestA == 0 || lex_less(om, bestA)))) {
            best = ov;
            bestA = om;
        }
    }
    __syncthreads();
    if (lane == 0) {
        redd[w] = best;
        redm[w] = bestA;
    }
    __syncthreads();
    best = redd[0];
    bestA = redm[0];
    for (int i = 1; i < NT / 64; ++i)
        if (redd[i] < best || (redd[i] == best && redm[i] != 0 && (bestA == 0 || lex_less(redm[i], bestA)))) {
            best = redd[i];
            bestA = redm[i];
        }
    __syncthreads();
    return bestA;
}

// One budget of a call: s kept keys, `extra` keys beyond A*_s, offsets of the
// row's index lists, and how its pool is enumerated.
struct PoolBudget {
    int s, extra, P, pool_off, set_off;
    int direct;  // through the dropped set (enum_complement), else the walk
    int cpl;     // the walk enumerates the dropped sets (its plan: P keys, P - s of them)
    size_t tab_off;  // the walk tables' offset in the workspace
    size_t inst_off, inst_stride;  // walked budgets: the rows' instances in the workspace
    EnumPlan pl;
    EnumTables tab;
};

// A walked budget's row instance, handed from the row kernel to the
// enumeration kernel: the pool's Gram matrix (P x P, row pitch P, float64),
// masses (P), the reported errors of A*_s and of the balancing set and EF_FW
// (float64), the seed mask A*_s and the pool's keys (ascending, int32).
struct PoolInst {
    size_t gm, ps, es, seed, keys, bytes;
};
__host__ __device__ inline PoolInst pool_inst(int P) {
    PoolInst I{};
    size_t o = 0;
    I.gm = o;
    o += (size_t)P * P * 8;
    I.ps = o;
    o += (size_t)P * 8;
    I.es = o;
    o += 3 * 8;
    I.seed = o;
    o += 8;
    I.keys = o;
    o += (size_t)P * 4;
    I.bytes = align_up(o, 16);
    return I;
}

struct PoolArgs {
    const void *q, *k, *v;
    const float *scale, *bias;
    int64_t H, G, N;
    int d, nb, max_swaps, fw_iters, Smax, Ptot, Stot, Pmax;
    PoolBudget b[kMaxBudgets];
    int32_t *pool_idx, *best_idx, *bal_idx, *geo_idx, *n_swaps;
    float *stats;
    char *ws;       // the workspace (walked budgets' instances, the rows' mu)
    size_t mu_off;  // [R][d] float64
};

}  // namespace

template <typename T>
__global__ void __launch_bounds__(PT) pool_row_kernel(PoolArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, NT = blockDim.x;
    const int64_t N = a.N;
    const int d = a.d, nb = a.nb;
    const int64_t R = a.H * a.G;
    const PoolLds L = pool_lds(N, d, a.Pmax);
    double *xq = (double *)(smem + L.xq);
    double *mu = (double *)(smem + L.mu);
    double *redd = (double *)(smem + L.red);
    uint64_t *redm = (uint64_t *)(redd + NT);
    int64_t *redi = (int64_t *)(redd + NT);
    int *ctr = (int *)(smem + L.ctr);
    int *rank = (int *)(smem + L.rank);
    int *eord = (int *)(smem + L.eord);
    int *tmp = (int *)(smem + L.tmp);
    int *plist = (int *)(smem + L.plist);
    double *pps = (double *)(smem + L.pps);
    double *sc = (double *)(smem + L.sc);  // [0, nb): dropped masses; nb: sigma^2; nb + 1: D
    double *zz = (double *)(smem + L.zz);
    double *ee = (double *)(smem + L.ee);
    unsigned char *rk = smem + L.rk;  // rank among the top keys, 255 beyond them
    uint64_t *seeds = (uint64_t *)(smem + L.seed);

    const int64_t r = xcd_order(blockIdx.x, gridDim.x);  // a unit's rows on one XCD
    const int64_t h = r / a.G;
    const T *qr = (const T *)a.q + r * d;
    const T *kh = (const T *)a.k + h * N * d;
    const T *vh = (const T *)a.v + h * N * d;
    const double scale = a.scale ? (double)a.scale[h] : (double)default_scale(d);

    // ---- 1. the row, once for every budget -------------------------------------
    for (int c = tid; c < d; c += NT) xq[c] = (double)Elem<T>::load(qr, c);
    for (int64_t j = tid; j < N; j += NT) rk[j] = 255;
    __syncthreads();
    double xr[8];  // this lane's columns of the query (then of mu), in registers
#pragma unroll
    for (int i = 0; i < 8; ++i) xr[i] = 0.0;
    lane_columns<T>(d, [&](int c, int slot) { xr[slot] = xq[c]; });
    for_key_sums(
        kh, N, d, [&](int, int slot, float x, double acc) { return fma(xr[slot], (double)x, acc); },
        [&](int64_t j, double acc) { zz[j] = scale * acc + (a.bias ? (double)a.bias[j] : 0.0); });
    __syncthreads();
    double zmax = -INFINITY;
    for (int64_t j = tid; j < N; j += NT) zmax = fmax(zmax, zz[j]);
    zmax = block_reduce(zmax, redd, OpMax());

    // top keys in rank order (z desc, j asc); every budget's A*_s is a prefix
    wave_top(zz, N, a.Smax, rank, redd, redi);
    for (int t = tid; t < a.Smax; t += NT) rk[rank[t]] = (unsigned char)t;
    // weights in place of the logits; each budget's dropped mass summed over
    // its dropped keys themselves
    double lsum = 0.0;
    for (int64_t j = tid; j < N; j += NT) lsum += exp(zz[j] - zmax);
    lsum = block_sum(lsum, redd);
    double drop[kMaxBudgets];
#pragma unroll
    for (int b = 0; b < kMaxBudgets; ++b) drop[b] = 0.0;
    for (int64_t j = tid; j < N; j += NT) {
        const double p = exp(zz[j] - zmax) / lsum;
        zz[j] = p;
        const int rj = rk[j];
#pragma unroll
        for (int b = 0; b < kMaxBudgets; ++b)
            if (b < nb && rj >= a.b[b].s) drop[b] += p;
    }
#pragma unroll
    for (int b = 0; b < kMaxBudgets; ++b)
        if (b < nb) drop[b] = block_sum(drop[b], redd);  // barriers: zz holds p

    // dense output: each lane accumulates its columns over the keys it visits
    {
        constexpr int VEC = RowVec<T>::VEC;
        double part[8];  // the lane's columns: VEC of one chunk, or up to 4 single ones
#pragma unroll
        for (int i = 0; i < 8; ++i) part[i] = 0.0;
        const bool vec = d % VEC == 0;
        const int GL = vec ? group_lanes(d, VEC) : 64;
        for_keys(vh, N, d, [&](int64_t j, int, int, auto &&walk) {
            if (j < 0) return;
            const double p = zz[j];
            walk([&](int, int slot, float x) { part[slot] = fma(p, (double)x, part[slot]); });
        });
        // combine: the (wave, group) partial sums through LDS, one group per round
        for (int c = tid; c < d; c += NT) mu[c] = 0.0;
        __syncthreads();
        const int lane = tid & 63, gi = vec ? lane % GL : lane;
        for (int rnd = 0; rnd < NT / 64 * (64 / GL); ++rnd) {
            const int me = (tid >> 6) * (64 / GL) + lane / GL;
            if (me == rnd) {
                if (vec) {
#pragma unroll
                    for (int i = 0; i < VEC; ++i) {
                        const int c = gi * VEC + i;
                        if (c < d) mu[c] += part[i];
                    }
                } else {
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const int c = gi + 64 * t;
                        if (c < d) mu[c] += part[t];
                    }
                }
            }
            __syncthreads();
        }
    }

    // the row's mu for the enumeration kernel's reported errors
    if (a.ws)
        for (int c = tid; c < d; c += NT) ((double *)(a.ws + a.mu_off))[r * d + c] = mu[c];

    // deviations: single-key errors, sigma^2 and D
    double s2 = 0.0, dmax = 0.0;
    lane_columns<T>(d, [&](int c, int slot) { xr[slot] = mu[c]; });
    for_key_sums(
        vh, N, d,
        [&](int, int slot, float x, double acc) {
            const double t = (double)x - xr[slot];
            return fma(t, t, acc);
        },
        [&](int64_t j, double acc) {
            const double p = zz[j];
            ee[j] = p * sqrt(acc);
            s2 = fma(p, acc, s2);
            dmax = fmax(dmax, acc);
        });
    s2 = block_sum(s2, redd);
    dmax = block_reduce(dmax, redd, OpMax());

    // ---- 2. each budget's candidate set ------------------------------------------
    // keys outside the smallest budget's A*_s in order of single-key error
    // (e desc, j asc): the first extra + s - smin hold a budget's extra keys
    // (at most s - smin of them are in its A*_s)
    int smin = a.b[0].s, me = 0;
    for (int b = 1; b < nb; ++b) smin = a.b[b].s < smin ? a.b[b].s : smin;
    for (int b = 0; b < nb; ++b) me = a.b[b].extra + a.b[b].s - smin > me ? a.b[b].extra + a.b[b].s - smin : me;
    wave_top(ee, N, me, eord, redd, redi, rk, smin);
    for (int b = 0; b < nb; ++b) {
        const PoolBudget &B = a.b[b];
        const int s = B.s, P = B.P;
        // the extra keys: largest single-key errors outside A*_s
        if (tid == 0) {
            int t = 0;
            for (int u = 0; u < me && t < B.extra; ++u) {
                const int j = eord[u];
                if (rk[j] >= s) tmp[s + t++] = j;
            }
        }
        if (tid < s) tmp[tid] = rank[tid];
        __syncthreads();
        // output order, then ascending keys with their masses
        if (tid < P) {
            const int key = tmp[tid];
            int pos = 0;
            for (int u = 0; u < P; ++u) pos += tmp[u] < key;
            plist[b * kPoolMax + pos] = key;
            pps[b * kPoolMax + pos] = zz[key];
            if (a.pool_idx) a.pool_idx[r * a.Ptot + B.pool_off + tid] = key;
        }
        __syncthreads();
        if (tid == 0) {
            uint64_t seed = 0;
            for (int i = 0; i < P; ++i)
                if (rk[plist[b * kPoolMax + i]] < s) seed |= 1ull << i;
            seeds[b] = seed;
        }
        __syncthreads();  // tmp is reused by the next budget
    }
    if (tid == 0) {
        for (int b = 0; b < nb; ++b) sc[b] = drop[b];
        sc[nb] = s2;
        sc[nb + 1] = sqrt(dmax);
    }
    __syncthreads();  // the row arrays are dead from here

    // ---- 3.-6. each budget's pool: instance, ES_pool, balancing, statistics -----
    double *Gm = (double *)(smem + L.gm);
    float *Vs = (float *)(smem + L.vs);
    double *cv = (double *)(smem + L.cv);
    double *Yd = (double *)(smem + L.yd);
    double *wf = (double *)(smem + L.wf);
    const int pitch = d + 1;
    for (int b = 0; b < nb; ++b) {
        const PoolBudget &B = a.b[b];
        const int s = B.s, P = B.P;
        const int *pid = plist + b * kPoolMax;
        const double *ps = pps + b * kPoolMax;
        const uint64_t seed = seeds[b];
        // the pool instance
        for (int e = tid; e < P * d; e += NT) {
            const int i = e / d, c = e % d;
            Vs[i * pitch + c] = Elem<T>::load(vh, (int64_t)pid[i] * d + c);
        }
        __syncthreads();
        // the Gram matrices of u_i = p_i (v_i - mu) and of v_i - mu (blocked,
        // as for the exhaustive search's rows)
        gram_matrix(P, d, pitch, Vs, ps, mu, Gm, P, Yd);
        __syncthreads();

        // ES_pool: pools dropping a few keys here; the walked ones hand their
        // instance to the enumeration kernel
        char *inst = B.direct ? nullptr : a.ws + B.inst_off + r * B.inst_stride;
        const PoolInst I = pool_inst(P);
        if (inst) {
            for (int e = tid; e < P * P; e += NT) ((double *)(inst + I.gm))[e] = Gm[e];
            for (int e = tid; e < P; e += NT) {
                ((double *)(inst + I.ps))[e] = ps[e];
                ((int32_t *)(inst + I.keys))[e] = pid[e];
            }
            if (tid == 0) *(uint64_t *)(inst + I.seed) = seed;
        }
        const uint64_t best = B.direct ? enum_complement(Gm, ps, P, P - s, cv, redd, redm) : 0ull;

        // Balancing within the pool on wave 0 alone (P <= 64 keys, one per
        // lane, no workgroup barrier), while waves 1 and 2 take the reported
        // errors of A*_s and the ES_pool set.
        const int lane = tid & 63, w = tid >> 6;
        // es(M) = ||sum_{i in M} p_i (v_i - mu)|| / p(M), within one wave
        auto wave_es = [&](uint64_t M) {
            if ((int64_t)__popcll(M) == N) return 0.0;
            double g2 = 0.0;
            for (int c = lane; c < d; c += 64) {
                double g = 0.0;
                for (uint64_t m = M; m; m &= m - 1) {
                    const int i = __ffsll((unsigned long long)m) - 1;
                    g = fma(ps[i], (double)Vs[i * pitch + c] - mu[c], g);
                }
                g2 = fma(g, g, g2);
            }
            g2 = wave_sum(g2);
            double pm = 0.0;
            for (uint64_t m = M; m; m &= m - 1) pm += ps[__ffsll((unsigned long long)m) - 1];
            return sqrt(g2) / pm;
        };
        uint64_t A = seed;
        int swaps = 0;
        double es_bal = 0.0;
        if (w == 0) {
            if (s < P) {
                const int x = lane;
                const bool inP = x < P;
                const double px = inP ? ps[x] : 0.0, gxx = inP ? Gm[x * P + x] : 0.0;
                const int nout = P - s;
                while (swaps < a.max_swaps) {
                    // c_x = sum_{y in A} Gm_xy, and the set's Gram value S and
                    // mass, recomputed from the Gram matrix every round
                    double cx = 0.0;
                    if (inP)
                        for (uint64_t m = A; m; m &= m - 1) cx += Gm[(__ffsll((unsigned long long)m) - 1) * P + x];
                    const bool mem = inP && ((A >> x) & 1ull);
                    const double S = wave_sum(mem ? cx : 0.0), PA = wave_sum(mem ? px : 0.0);
                    const double cur = S / (PA * PA);
                    // lane j (a non-member) against every member i, ascending;
                    // pair t = (member rank) nout + (non-member rank)
                    const bool out = inP && !mem;
                    double bv = 0.0;
                    int bii = -1, ii = 0;
                    for (uint64_t m = A; m; m &= m - 1, ++ii) {
                        const int i = __ffsll((unsigned long long)m) - 1;
                        const double ci = lane_value(cx, i), gii = lane_value(gxx, i), pi = lane_value(px, i);
                        if (out) {
                            const double Sn = S - 2.0 * ci + gii + 2.0 * (cx - Gm[i * P + x]) + gxx;
                            const double Pn = PA - pi + px;
                            const double val = fmax(Sn, 0.0) / (Pn * Pn);
                            if (bii < 0 || -val > bv) {
                                bv = -val;
                                bii = ii;
                            }
                        }
                    }
                    // argmax of -val over the wave; ties to the smallest t
                    int bt = bii < 0 ? -1 : bii * nout + (x - __popcll(A & ((1ull << x) - 1ull)));
#pragma unroll
                    for (int off = 32; off > 0; off >>= 1) {
                        const double ov = __shfl_xor(bv, off);
                        const int ot = __shfl_xor(bt, off);
                        if (ot >= 0 && (bt < 0 || ov > bv || (ov == bv && ot < bt))) {
                            bv = ov;
                            bt = ot;
                        }
                    }
                    if (bt < 0 || !(-bv < cur)) break;
                    const int i = nth_bit(A, bt / nout);
                    const int j = nth_bit(~A & (P == 64 ? ~0ull : (1ull << P) - 1ull), bt % nout);
                    A = (A & ~(1ull << i)) | (1ull << j);
                    ++swaps;
                }
            }
            es_bal = wave_es(A);
        } else if (w == 1 || (w == 2 && B.direct)) {
            const double e = wave_es(w == 1 ? seed : best);
            if (lane == 0) redd[w] = e;
        } else if (w == 3) {
            // Frank-Wolfe over the pool's values, one lane per pool key: with
            // y_x = v_x - mu and the iterate's residual r = sum_i w_i y_i, lane
            // x holds w_x and t_x = <y_x, r>; the vertex is the least t_x
            // (ties to the lower key), the duality gap |r|^2 - t_j, and the
            // exact line search eta = min(1, gap / |y_j - r|^2)
            const int x = lane;
            const bool inP = x < P;
            const uint64_t lanes = P == 64 ? ~0ull : (1ull << P) - 1ull;
            auto wave_argmin = [&](double v, int &at) {
                int j = inP ? x : 64;
                v = inP ? v : INFINITY;
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const double ov = __shfl_xor(v, off);
                    const int oj = __shfl_xor(j, off);
                    if (ov < v || (ov == v && oj < j)) {
                        v = ov;
                        j = oj;
                    }
                }
                at = j;
                return v;
            };
            int j0;
            wave_argmin(inP ? Yd[x * P + x] : 0.0, j0);  // the key nearest mu
            double wx = x == j0 ? 1.0 : 0.0;
            double tx = inP ? Yd[j0 * P + x] : 0.0;
            uint64_t sup = 1ull << j0;
            int steps = 0;
            while (steps < a.fw_iters) {
                int j;
                const double tj = wave_argmin(tx, j);
                const double q = wave_sum(wx * tx);
                const double gap = q - tj;
                if (!(gap > 0.0)) break;
                if (!((sup >> j) & 1ull) && __popcll(sup) >= s) break;
                const double nrm = Yd[j * P + j] - 2.0 * tj + q;
                if (!(nrm > 0.0)) break;
                const double eta = fmin(1.0, gap / nrm);
                wx *= 1.0 - eta;
                if (x == j) wx += eta;
                tx = inP ? fma(eta, Yd[j * P + x], (1.0 - eta) * tx) : 0.0;
                sup = __ballot(wx > 0.0) & lanes;
                ++steps;
            }
            if (inP) wf[x] = wx;
            // ||sum_i w_i (v_i - mu)|| over the support, columns across lanes
            double e2 = 0.0;
            for (int c = lane; c < d; c += 64) {
                double g = 0.0;
                for (uint64_t m = sup; m; m &= m - 1) {
                    const int i = __ffsll((unsigned long long)m) - 1;
                    g = fma(wf[i], (double)Vs[i * pitch + c] - mu[c], g);
                }
                e2 = fma(g, g, e2);
            }
            e2 = wave_sum(e2);
            // the geometric set: the support, then top-mass keys in rank order
            uint64_t geo = sup;
            for (int t = 0; t < s && __popcll(geo) < s; ++t) {
                const int key = rank[t];
                geo |= __ballot(inP && pid[x] == key) & lanes;
            }
            const double eg = wave_es(geo);
            if (lane == 0) {
                redd[3] = sqrt(e2);
                redd[4] = eg;
                redd[5] = (double)steps;
                redm[3] = geo;
            }
        }
        __syncthreads();
        const double es_top = redd[1], es_pool = redd[2];
        const double ef_fw = redd[3], es_geo = redd[4], fw_steps = redd[5];
        const uint64_t geo = redm[3];
        if (tid == 0) {
            int t = 0, u = 0, v = 0;
            for (int i = 0; i < P; ++i) {
                if (B.direct && ((best >> i) & 1ull) && t < s) a.best_idx[r * a.Stot + B.set_off + t++] = pid[i];
                if (a.bal_idx && ((A >> i) & 1ull) && u < s) a.bal_idx[r * a.Stot + B.set_off + u++] = pid[i];
                if (a.geo_idx && ((geo >> i) & 1ull) && v < s) a.geo_idx[r * a.Stot + B.set_off + v++] = pid[i];
            }
            if (a.n_swaps) a.n_swaps[b * R + r] = swaps;
            const double m = sc[b], sigma = sqrt(sc[nb]), D = sc[nb + 1];
            double ptop = 0.0;
            for (int i = 0; i < P; ++i)
                if ((seed >> i) & 1ull) ptop += ps[i];
            auto ratio = [](double num, double den) {
                return den > 0.0 ? num / den : (num == 0.0 ? 1.0 : (double)INFINITY);
            };
            float *o = a.stats + (b * R + r) * FW_POOL_NSTATS;
            o[0] = (float)es_top;
            o[2] = (float)es_bal;
            if (B.direct) {
                o[1] = (float)es_pool;
                o[3] = (float)ratio(es_top, es_pool);
                o[4] = (float)(es_top > 0.0 ? 1.0 - es_pool / es_top : 0.0);
                o[5] = (float)ratio(es_bal, es_pool);
                o[14] = (float)ratio(es_pool, ef_fw);
            } else {  // the enumeration kernel forms the ES_pool columns
                double *ev = (double *)(inst + I.es);
                ev[0] = es_top;
                ev[1] = es_bal;
                ev[2] = ef_fw;
            }
            o[6] = (float)m;
            o[7] = (float)(es_top * ptop);
            o[8] = (float)D;
            o[9] = (float)sigma;
            o[10] = (float)(2.0 * D * m);
            o[11] = (float)(m < 1.0 ? sqrt(m / (1.0 - m)) * sigma : (double)INFINITY);
            o[12] = (float)ef_fw;
            o[13] = (float)es_geo;
            o[15] = (float)fw_steps;
        }
        __syncthreads();  // the next budget overwrites the pool arrays
    }
}

// ---------------------------------------------------------------------------
// ES_pool of a walked budget: one workgroup per row takes the row's pool
// instance from the workspace, runs the walk shared with the exhaustive best
// subset (seeded by A*_s), and forms the ES_pool set's reported error from
// d-dimensional sums over the pool's values (the same sums, in the same
// order, as the row kernel's other reported errors) and the statistics that
// depend on it.
namespace {
struct PoolEnumArgs {
    const void *v;
    int64_t G, N, R;
    int d, P, s, cpl, Stot, set_off, b;
    EnumPlan pl;
    EnumTables tab;
    const char *inst;
    size_t inst_stride;
    const double *mu;
    int32_t *best_idx;
    float *stats;
};

struct PoolEnumLds {
    size_t gm, ps, cv, keys, ent, pl, red, ctr, wt, total;
};
// ht: each wave also keeps the walk's step values at its own beta
__host__ __device__ inline PoolEnumLds pool_enum_lds(int P, int nent, int nt, bool ht) {
    PoolEnumLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.gm = take((size_t)P * P * 8);
    L.ps = take((size_t)P * 8);
    L.cv = take((size_t)P * 8);
    L.keys = take((size_t)P * 4);
    L.ent = take((size_t)nent * 16);
    L.pl = take((size_t)nent * 8);
    L.red = take((size_t)(nt / 64) * 3 * 8);
    L.ctr = take(16);
    L.wt = take(ht ? (size_t)(nt / 64) * nent * 8 : 0);
    L.total = o;
    return L;
}
constexpr size_t kPoolEnumLdsHT = 40 * 1024;  // per-wave step values within four workgroups per CU
}  // namespace

template <typename T, int WMAX, bool HT>
__global__ void __launch_bounds__(PT, 4) pool_enum_kernel(PoolEnumArgs e) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, NT = blockDim.x, lane = tid & 63;
    const int P = e.P, d = e.d;
    const PoolEnumLds L = pool_enum_lds(P, e.pl.nent, NT, HT);
    double *Gm = (double *)(smem + L.gm);
    double *ps = (double *)(smem + L.ps);
    double *cv = (double *)(smem + L.cv);
    int32_t *pid = (int32_t *)(smem + L.keys);
    double *redd = (double *)(smem + L.red);
    uint64_t *redm = (uint64_t *)(redd + 2 * (NT >> 6));
    const int64_t r = blockIdx.x;
    const char *rec = e.inst + r * e.inst_stride;
    const PoolInst I = pool_inst(P);
    for (int x = tid; x < P * P; x += NT) Gm[x] = ((const double *)(rec + I.gm))[x];
    for (int x = tid; x < P; x += NT) {
        ps[x] = ((const double *)(rec + I.ps))[x];
        pid[x] = ((const int32_t *)(rec + I.keys))[x];
    }
    const uint64_t seed = *(const uint64_t *)(rec + I.seed);
    __syncthreads();
    const uint64_t best = enum_best_body<WMAX, HT>(e.pl, Gm, ps, seed, e.tab.io, e.tab.wmk, e.tab.jobs, e.tab.omk,
                                                   (double2 *)(smem + L.ent), (double *)(smem + L.pl), redd, redm,
                                                   (int *)(smem + L.ctr), e.cpl != 0, cv, (double *)(smem + L.wt));
    if (tid >= 64) return;
    // es(best) = ||sum_{i in best} p_i (v_i - mu)|| / p(best), columns across
    // the lanes of wave 0
    const T *vh = (const T *)e.v + (r / e.G) * e.N * d;
    const double *mu = e.mu + r * d;
    double es_pool = 0.0;
    if ((int64_t)__popcll(best) != e.N) {
        double g2 = 0.0;
        for (int c = lane; c < d; c += 64) {
            double g = 0.0;
            for (uint64_t m = best; m; m &= m - 1) {
                const int i = __ffsll((unsigned long long)m) - 1;
                g = fma(ps[i], (double)(float)Elem<T>::load(vh, (int64_t)pid[i] * d + c) - mu[c], g);
            }
            g2 = fma(g, g, g2);
        }
        g2 = wave_sum(g2);
        double pm = 0.0;
        for (uint64_t m = best; m; m &= m - 1) pm += ps[__ffsll((unsigned long long)m) - 1];
        es_pool = sqrt(g2) / pm;
    }
    if (lane == 0) {
        int t = 0;
        for (int i = 0; i < P; ++i)
            if (((best >> i) & 1ull) && t < e.s) e.best_idx[r * e.Stot + e.set_off + t++] = pid[i];
        const double *ev = (const double *)(rec + I.es);
        const double es_top = ev[0], es_bal = ev[1], ef_fw = ev[2];
        auto ratio = [](double num, double den) {
            return den > 0.0 ? num / den : (num == 0.0 ? 1.0 : (double)INFINITY);
        };
        float *o = e.stats + (e.b * e.R + r) * FW_POOL_NSTATS;
        o[1] = (float)es_pool;
        o[3] = (float)ratio(es_top, es_pool);
        o[4] = (float)(es_top > 0.0 ? 1.0 - es_pool / es_top : 0.0);
        o[5] = (float)ratio(es_bal, es_pool);
        o[14] = (float)ratio(es_pool, ef_fw);
    }
}

// Per cell and budget: the median of the dropped mass over the cell's G rows
// (the mean of the two middle values for even G), and the flat label
// median > threshold.  Grid: (H, budgets).
__global__ void __launch_bounds__(256) pool_cell_kernel(const float *stats, int64_t H, int64_t G, float threshold,
                                                        float *cell_median, uint8_t *cell_flat) {
    __shared__ float lo_hi[2];
    const int64_t h = blockIdx.x, b = blockIdx.y;
    const float *st = stats + (b * H * G + h * G) * FW_POOL_NSTATS + FW_POOL_DROPPED;
    const int64_t lo = (G - 1) / 2, hi = G / 2;
    for (int64_t g = threadIdx.x; g < G; g += blockDim.x) {
        const float x = st[g * FW_POOL_NSTATS];
        int64_t rank = 0;
        for (int64_t u = 0; u < G; ++u) {
            const float y = st[u * FW_POOL_NSTATS];
            rank += (y < x) || (y == x && u < g);
        }
        if (rank == lo) lo_hi[0] = x;
        if (rank == hi) lo_hi[1] = x;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const float med = (float)(0.5 * ((double)lo_hi[0] + (double)lo_hi[1]));
        if (cell_median) cell_median[b * H + h] = med;
        if (cell_flat) cell_flat[b * H + h] = med > threshold ? 1 : 0;
    }
}

// ---------------------------------------------------------------------------
// Host: plans of every budget, launch configuration.
namespace {
struct PoolPlan {
    int nb, Smax, Ptot, Stot, Pmax;
    PoolBudget b[kMaxBudgets];
    size_t lds, ws, mu_off;
    bool walked;  // some budget is enumerated by the enumeration kernel
};

// R rows: the workspace holds every walked budget's row instances.
bool make_pool_plan(int64_t N, int d, int nb, const int32_t *s, const int32_t *extra, int64_t R, PoolPlan *out) {
    if (nb < 1 || nb > kMaxBudgets) return false;
    PoolPlan pp{};
    pp.nb = nb;
    size_t ws = 0;
    for (int b = 0; b < nb; ++b) {
        const int sb = s[b], eb = extra[b], P = sb + eb;
        if (sb < 1 || eb < 0 || P > kPoolMax || P > N) return false;
        PoolBudget &B = pp.b[b];
        B.s = sb;
        B.extra = eb;
        B.P = P;
        B.pool_off = pp.Ptot;
        B.set_off = pp.Stot;
        pp.Ptot += P;
        pp.Stot += sb;
        pp.Smax = sb > pp.Smax ? sb : pp.Smax;
        pp.Pmax = P > pp.Pmax ? P : pp.Pmax;
        B.direct = eb < kWalkDrop;
        if (!B.direct) {
            if (binom(P, sb) >= (1ull << 31)) return false;
            // walk the kept sets or the dropped sets, whichever plan costs less
            EnumPlan pk, pd;
            double ck = 0.0, cd = 0.0;
            const bool okk = choose_plan(P, sb, &pk, &ck), okd = choose_plan(P, eb, &pd, &cd);
            if (!okk && !okd) {
                if (eb > kDirectDrop) return false;
                B.direct = 1;
                continue;
            }
            B.cpl = okd && (!okk || cd < ck);
            B.pl = B.cpl ? pd : pk;
            B.pl.d = d;
            B.pl.G = 1;
            ws = align_up(ws, 256);
            B.tab_off = ws;
            ws += enum_tables(B.pl, nullptr).bytes;
            if (pool_enum_lds(P, B.pl.nent, PT, false).total > 160 * 1024) return false;
            pp.walked = true;
        }
    }
    if (pp.walked) {
        ws = align_up(ws, 256);
        pp.mu_off = ws;
        ws += (size_t)R * d * 8;
        for (int b = 0; b < nb; ++b) {
            PoolBudget &B = pp.b[b];
            if (B.direct) continue;
            ws = align_up(ws, 256);
            B.inst_off = ws;
            B.inst_stride = pool_inst(B.P).bytes;
            ws += (size_t)R * B.inst_stride;
        }
    }
    // the row kernel holds no walk tables: the walks run in the enumeration kernel
    pp.lds = pool_lds(N, d, pp.Pmax).total;
    if (pp.lds > 160 * 1024) return false;
    // 0 is the size query's answer for invalid arguments: a call whose pools
    // are all enumerated directly asks for a token 256 bytes it does not use
    pp.ws = ws ? align_up(ws, 256) : 256;
    *out = pp;
    return true;
}
}  // namespace

bool pool_plannable(int64_t N, int d, int nb, const int32_t *s, const int32_t *extra) {
    PoolPlan pp;
    return make_pool_plan(N, d, nb, s, extra, 1, &pp);
}

size_t pool_ws_bytes(const fw_rows &rows, int nb, const int32_t *s, const int32_t *extra) {
    PoolPlan pp;
    if (!make_pool_plan(rows.n, (int)rows.d, nb, s, extra, rows.H * rows.G, &pp)) return 0;
    return pp.ws;
}

hipError_t launch_pool(const fw_rows &rows, int nb, const int32_t *s, const int32_t *extra, int max_swaps,
                       int fw_iters, int32_t *pool_idx, int32_t *best_idx, int32_t *bal_idx, int32_t *geo_idx,
                       int32_t *n_swaps, float *stats,
                       float flat_threshold, float *cell_median, uint8_t *cell_flat, void *ws, hipStream_t st) {
    PoolPlan pp;
    if (!make_pool_plan(rows.n, (int)rows.d, nb, s, extra, rows.H * rows.G, &pp))
        return hipErrorInvalidConfiguration;
    PoolArgs a{};
    hipError_t e = hipSuccess;
    for (int b = 0; b < nb; ++b) {
        a.b[b] = pp.b[b];
        if (!a.b[b].direct) {
            a.b[b].tab = enum_tables(a.b[b].pl, (char *)ws + a.b[b].tab_off);
            if ((e = launch_enum_tables(a.b[b].pl, a.b[b].tab, st)) != hipSuccess) return e;
        }
    }
    a.q = rows.q;
    a.k = rows.k;
    a.v = rows.v;
    a.scale = rows.scale;
    a.bias = rows.bias;
    a.H = rows.H;
    a.G = rows.G;
    a.N = rows.n;
    a.d = (int)rows.d;
    a.nb = nb;
    a.max_swaps = max_swaps;
    a.fw_iters = fw_iters;
    a.Smax = pp.Smax;
    a.Ptot = pp.Ptot;
    a.Stot = pp.Stot;
    a.Pmax = pp.Pmax;
    a.pool_idx = pool_idx;
    a.best_idx = best_idx;
    a.bal_idx = bal_idx;
    a.geo_idx = geo_idx;
    a.n_swaps = n_swaps;
    a.stats = stats;
    a.ws = pp.walked ? (char *)ws : nullptr;
    a.mu_off = pp.mu_off;
    const unsigned R = (unsigned)(rows.H * rows.G);
    if (rows.dtype == FW_BF16)
        hipLaunchKernelGGL(pool_row_kernel<uint16_t>, dim3(R), dim3(PT), pp.lds, st, a);
    else
        hipLaunchKernelGGL(pool_row_kernel<float>, dim3(R), dim3(PT), pp.lds, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    for (int b = 0; b < nb; ++b) {
        const PoolBudget &B = a.b[b];
        if (B.direct) continue;
        PoolEnumArgs g{};
        g.v = rows.v;
        g.G = rows.G;
        g.N = rows.n;
        g.R = (int64_t)R;
        g.d = (int)rows.d;
        g.P = B.P;
        g.s = B.s;
        g.cpl = B.cpl;
        g.Stot = pp.Stot;
        g.set_off = B.set_off;
        g.b = b;
        g.pl = B.pl;
        g.tab = B.tab;
        g.inst = (const char *)ws + B.inst_off;
        g.inst_stride = B.inst_stride;
        g.mu = (const double *)((const char *)ws + pp.mu_off);
        g.best_idx = best_idx;
        g.stats = stats;
        int wmax = 0;
        for (int q = 0; q < B.pl.ncls; ++q) wmax = B.pl.cls[q].wn > wmax ? B.pl.cls[q].wn : wmax;
        const PoolEnumLds Lh = pool_enum_lds(B.P, B.pl.nent, PT, true);
        const bool ht = Lh.total <= kPoolEnumLdsHT;
        const size_t lds = ht ? Lh.total : pool_enum_lds(B.P, B.pl.nent, PT, false).total;
        auto go = [&](auto kern) { hipLaunchKernelGGL(kern, dim3(R), dim3(PT), lds, st, g); };
        auto pick = [&](auto tag) {
            using T = decltype(tag);
            if (wmax <= 12) {
                if (ht) go(pool_enum_kernel<T, 12, true>);
                else go(pool_enum_kernel<T, 12, false>);
            } else if (wmax <= 14) {
                if (ht) go(pool_enum_kernel<T, 14, true>);
                else go(pool_enum_kernel<T, 14, false>);
            } else {
                if (ht) go(pool_enum_kernel<T, kMaxWalk, true>);
                else go(pool_enum_kernel<T, kMaxWalk, false>);
            }
        };
        if (rows.dtype == FW_BF16) pick(uint16_t{});
        else pick(float{});
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (cell_median || cell_flat)
        hipLaunchKernelGGL(pool_cell_kernel, dim3((unsigned)rows.H, (unsigned)nb), dim3(256), 0, st, stats, rows.H,
                           rows.G, flat_threshold, cell_median, cell_flat);
    return hipGetLastError();
}

}  // namespace fw
