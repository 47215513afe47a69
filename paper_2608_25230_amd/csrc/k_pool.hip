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
//      shared with the exhaustive best subset, seeded by A*_s;
//   5. the balancing selector drawing from the pool: every (kept, dropped)
//      pair of the pool scored from the Gram each round, ties to the smallest
//      (out, in) key pair, accepted only on a strict decrease;
//   6. the reported errors of A*_s, the ES_pool argmin and the balancing set
//      from d-dimensional residual sums, and the certificate statistics.
// A second kernel takes each cell's median dropped mass over its rows.
#include "fw_internal.hpp"
#include "instance64.hpp"
#include "enum_walk.hpp"

namespace fw {

namespace {

constexpr int PT = 256;       // threads per row workgroup
constexpr int kPoolMax = 64;  // pool keys (one 64-bit mask)

struct PoolLds {
    size_t xq, mu, red, ctr, pid, ps, sc;  // persistent
    size_t zz, ee, bits;                   // row phase
    size_t gm, vs, ent, pl, cv;            // pool phase (overlays the row phase)
    size_t total;
};

__host__ __device__ inline PoolLds pool_lds(int64_t N, int d, int P, int nent) {
    PoolLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.xq = take((size_t)d * 8);
    L.mu = take((size_t)d * 8);
    L.red = take((size_t)PT * 16);
    L.ctr = take(16);
    L.pid = take((size_t)kPoolMax * 4 * 2);  // pool keys ascending, then in output order
    L.ps = take((size_t)kPoolMax * 8);
    L.sc = take((size_t)16 * 8);
    const size_t base = o;
    L.zz = base;
    L.ee = align_up(L.zz + (size_t)N * 8, 16);
    L.bits = align_up(L.ee + (size_t)N * 8, 16);
    const size_t row_end = L.bits + (size_t)((N + 63) / 64) * 8;
    L.gm = base;
    L.vs = align_up(L.gm + (size_t)P * P * 8, 16);
    L.cv = align_up(L.vs + (size_t)P * (d + 1) * 4, 16);
    L.ent = align_up(L.cv + (size_t)P * 8, 16);
    L.pl = L.ent + (size_t)nent * 16;
    const size_t pool_end = L.pl + (size_t)nent * 8;
    L.total = align_up(row_end > pool_end ? row_end : pool_end, 16);
    return L;
}

// Key rows are read by groups of lanes: a group of GL lanes covers one key,
// each lane VEC consecutive columns per load (whole rows per instruction).
template <typename T> struct RowVec;
template <> struct RowVec<uint16_t> {
    static constexpr int VEC = 8;
    __device__ static void load(const uint16_t *row, int c0, float (&x)[8]) {
        const uint4 w = *(const uint4 *)(row + c0);
        const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] = __uint_as_float(u[i] << 16);
            x[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
        }
    }
};
template <> struct RowVec<float> {
    static constexpr int VEC = 4;
    __device__ static void load(const float *row, int c0, float (&x)[4]) {
        const float4 w = *(const float4 *)(row + c0);
        x[0] = w.x; x[1] = w.y; x[2] = w.z; x[3] = w.w;
    }
};

// lanes per key for rows of d elements: a power of two covering d / VEC chunks
__host__ __device__ inline int group_lanes(int d, int vec) {
    const int chunks = (d + vec - 1) / vec;
    int g = 1;
    while (g < chunks && g < 64) g <<= 1;
    return g;
}

// Sum over the GL lanes of a group (GL a power of two <= 64).
__device__ __forceinline__ double group_sum(double v, int GL) {
    for (int off = 1; off < GL; off <<= 1) v += __shfl_xor(v, off);
    return v;
}

// For every key j of M [N][d]: f(j, lane_in_group, GL, walk), where
// walk(g) calls g(c, slot, x) for the lane's elements x = M[j][c]; slot
// (< 32) numbers them within the lane, the same for every key.  The GL lanes
// of a group share a key (j = -1 on lanes past the end, which still take part
// in the group's shuffles).  VEC-wide loads when d is a multiple of VEC, else
// one element per lane.  d <= 256: at most four chunks (elements) per lane.
template <typename T, typename F>
__device__ void for_keys(const T *M, int64_t N, int d, F &&f) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, NW = blockDim.x >> 6;
    constexpr int VEC = RowVec<T>::VEC;
    if (d % VEC == 0) {
        const int GL = group_lanes(d, VEC), KPW = 64 / GL;  // keys per wave step
        const int gi = lane % GL, gk = lane / GL;
        const int chunks = d / VEC;
        for (int64_t j0 = (int64_t)w * KPW; j0 < N; j0 += (int64_t)NW * KPW) {
            const int64_t j = j0 + gk;
            const bool ok = j < N;
            f(ok ? j : -1, gi, GL, [&](auto &&g) {
                if (!ok) return;
                const T *row = M + j * d;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int ch = gi + GL * t;
                    if (ch < chunks) {
                        float x[VEC];
                        RowVec<T>::load(row, ch * VEC, x);
#pragma unroll
                        for (int i = 0; i < VEC; ++i) g(ch * VEC + i, t * VEC + i, x[i]);
                    }
                }
            });
        }
    } else {
        for (int64_t j = w; j < N; j += NW) {
            f(j, lane, 64, [&](auto &&g) {
                const T *row = M + j * d;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int c = lane + 64 * t;
                    if (c < d) g(c, t, Elem<T>::load(row, c));
                }
            });
        }
    }
}

// Workgroup argmax of (key desc, index asc) over per-thread candidates
// (idx < 0: none).  Returns the winner on every thread.
__device__ inline void block_argmax(double &val, int64_t &idx, double *redv, int64_t *redi) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, NW = blockDim.x >> 6;
    auto better = [](double v1, int64_t i1, double v2, int64_t i2) {
        if (i1 < 0) return false;
        if (i2 < 0) return true;
        return v1 > v2 || (v1 == v2 && i1 < i2);
    };
    for (int off = 32; off > 0; off >>= 1) {
        const double ov = __shfl_xor(val, off);
        const int64_t oi = __shfl_xor(idx, off);
        if (better(ov, oi, val, idx)) { val = ov; idx = oi; }
    }
    __syncthreads();
    if (lane == 0) { redv[w] = val; redi[w] = idx; }
    __syncthreads();
    val = redv[0];
    idx = redi[0];
    for (int i = 1; i < NW; ++i)
        if (better(redv[i], redi[i], val, idx)) { val = redv[i]; idx = redi[i]; }
    __syncthreads();
}

__device__ inline double block_sum(double v, double *red) { return block_reduce(v, red, OpSum()); }

struct PoolArgs {
    const void *q, *k, *v;
    const float *scale, *bias;
    int64_t H, G, N;
    int d, s, extra, max_swaps;
    EnumPlan pl;
    EnumTables tab;
    int32_t *pool_idx, *best_idx, *bal_idx, *n_swaps;
    float *stats;
};

}  // namespace

template <typename T>
__global__ void __launch_bounds__(PT) pool_row_kernel(PoolArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, NT = blockDim.x;
    const int64_t N = a.N;
    const int d = a.d, s = a.s, P = a.s + a.extra;
    const PoolLds L = pool_lds(N, d, P, a.pl.nent);
    double *xq = (double *)(smem + L.xq);
    double *mu = (double *)(smem + L.mu);
    double *redd = (double *)(smem + L.red);
    uint64_t *redm = (uint64_t *)(redd + NT);
    int64_t *redi = (int64_t *)(redd + NT);
    int *ctr = (int *)(smem + L.ctr);
    int *pid = (int *)(smem + L.pid);  // [0, P): ascending keys; [64, 64 + P): output order
    double *ps = (double *)(smem + L.ps);
    double *sc = (double *)(smem + L.sc);
    double *zz = (double *)(smem + L.zz);
    double *ee = (double *)(smem + L.ee);
    uint64_t *bits = (uint64_t *)(smem + L.bits);

    const int64_t r = blockIdx.x;
    const int64_t h = r / a.G;
    const T *qr = (const T *)a.q + r * d;
    const T *kh = (const T *)a.k + h * N * d;
    const T *vh = (const T *)a.v + h * N * d;
    const double scale = a.scale ? (double)a.scale[h] : (double)default_scale(d);

    // ---- 1. the row ---------------------------------------------------------
    for (int c = tid; c < d; c += NT) xq[c] = (double)Elem<T>::load(qr, c);
    for (int64_t e = tid; e < (N + 63) / 64; e += NT) bits[e] = 0ull;
    __syncthreads();
    for_keys(kh, N, d, [&](int64_t j, int gi, int GL, auto &&walk) {
        double acc = 0.0;
        walk([&](int c, int, float x) { acc = fma(xq[c], (double)x, acc); });
        acc = group_sum(acc, GL);
        if (j >= 0 && gi == 0) zz[j] = scale * acc + (a.bias ? (double)a.bias[j] : 0.0);
    });
    __syncthreads();
    double zmax = -INFINITY;
    for (int64_t j = tid; j < N; j += NT) zmax = fmax(zmax, zz[j]);
    zmax = block_reduce(zmax, redd, OpMax());

    // ---- 2a. top-mass set: s rounds, each the next key in (z desc, j asc) ---
    {
        double pv = INFINITY;
        int64_t pi = -1;
        for (int t = 0; t < s; ++t) {
            double bv = 0.0;
            int64_t bi = -1;
            for (int64_t j = tid; j < N; j += NT) {
                const double z = zz[j];
                const bool after = z < pv || (z == pv && j > pi);
                if (after && (bi < 0 || z > bv || (z == bv && j < bi))) { bv = z; bi = j; }
            }
            block_argmax(bv, bi, redd, redi);
            if (tid == 0 && bi >= 0) {  // s <= n: a key is always found
                pid[64 + t] = (int)bi;
                bits[bi >> 6] |= 1ull << (bi & 63);
            }
            pv = bv;
            pi = bi;
        }
    }
    // weights in place of the logits; the dropped mass of A*_s summed over the
    // dropped keys themselves
    double lsum = 0.0;
    for (int64_t j = tid; j < N; j += NT) lsum += exp(zz[j] - zmax);
    lsum = block_sum(lsum, redd);
    double drop = 0.0;
    for (int64_t j = tid; j < N; j += NT) {
        const double p = exp(zz[j] - zmax) / lsum;
        zz[j] = p;
        if (!((bits[j >> 6] >> (j & 63)) & 1ull)) drop += p;
    }
    drop = block_sum(drop, redd);  // ends with a barrier: zz holds p

    // dense output: each lane accumulates its columns over the keys it visits
    {
        constexpr int VEC = RowVec<T>::VEC;
        double part[8 * 4];  // up to 4 chunks of VEC columns per lane (d <= 256)
#pragma unroll
        for (int i = 0; i < 32; ++i) part[i] = 0.0;
        const bool vec = d % VEC == 0;
        const int GL = vec ? group_lanes(d, VEC) : 64;
        for_keys(vh, N, d, [&](int64_t j, int gi, int, auto &&walk) {
            if (j < 0) return;
            const double p = zz[j];
            walk([&](int, int slot, float x) { part[slot] = fma(p, (double)x, part[slot]); });
        });
        // combine: partial sums per column through LDS, one column per thread
        for (int c = tid; c < d; c += NT) mu[c] = 0.0;
        __syncthreads();
        const int lane = tid & 63, gi = vec ? lane % GL : lane;
        for (int rnd = 0; rnd < NT / 64 * (64 / GL); ++rnd) {
            // round rnd: the lanes whose (wave, group) index is rnd add their partials
            const int me = (tid >> 6) * (64 / GL) + lane / GL;
            if (me == rnd) {
                if (vec) {
#pragma unroll
                    for (int t = 0; t < 4; ++t)
#pragma unroll
                        for (int i = 0; i < VEC; ++i) {
                            const int c = (gi + GL * t) * VEC + i;
                            if (c < d) mu[c] += part[t * VEC + i];
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

    // deviations: single-key errors, sigma^2 and D
    double s2 = 0.0, dmax = 0.0;
    for_keys(vh, N, d, [&](int64_t j, int gi, int GL, auto &&walk) {
        double acc = 0.0;
        walk([&](int c, int, float x) {
            const double t = (double)x - mu[c];
            acc = fma(t, t, acc);
        });
        acc = group_sum(acc, GL);
        if (j >= 0 && gi == 0) {
            const double p = zz[j];
            ee[j] = p * sqrt(acc);
            s2 = fma(p, acc, s2);
            dmax = fmax(dmax, acc);
        }
    });
    s2 = block_sum(s2, redd);
    dmax = block_reduce(dmax, redd, OpMax());

    // ---- 2b. extras: the largest single-key errors outside A*_s ------------
    {
        double pv = INFINITY;
        int64_t pi = -1;
        for (int t = 0; t < a.extra; ++t) {
            double bv = 0.0;
            int64_t bi = -1;
            for (int64_t j = tid; j < N; j += NT) {
                if ((bits[j >> 6] >> (j & 63)) & 1ull) continue;
                const double e = ee[j];
                const bool after = e < pv || (e == pv && j > pi);
                if (after && (bi < 0 || e > bv || (e == bv && j < bi))) { bv = e; bi = j; }
            }
            block_argmax(bv, bi, redd, redi);
            if (tid == 0) pid[64 + s + t] = bi >= 0 ? (int)bi : 0;  // s + extra <= n
            pv = bv;
            pi = bi;
        }
    }
    // pool keys ascending, their masses; the seed (A*_s) as a pool-position mask
    if (tid < P) {
        const int key = pid[64 + tid];
        int rank = 0;
        for (int u = 0; u < P; ++u) rank += pid[64 + u] < key;
        pid[rank] = key;
        ps[rank] = zz[key];
        if (a.pool_idx) a.pool_idx[r * P + tid] = key;
    }
    if (tid == 0) {
        sc[0] = drop;
        sc[1] = s2;
        sc[2] = sqrt(dmax);
    }
    __syncthreads();  // the row arrays are dead from here
    uint64_t seed = 0;
    for (int i = 0; i < P; ++i)
        if ((bits[pid[i] >> 6] >> (pid[i] & 63)) & 1ull) seed |= 1ull << i;
    __syncthreads();

    // ---- 3. the pool instance -------------------------------------------------
    double *Gm = (double *)(smem + L.gm);
    float *Vs = (float *)(smem + L.vs);
    double *cv = (double *)(smem + L.cv);
    double2 *ent = (double2 *)(smem + L.ent);
    double *PLt = (double *)(smem + L.pl);
    const int pitch = d + 1;
    for (int e = tid; e < P * d; e += NT) {
        const int i = e / d, c = e % d;
        Vs[i * pitch + c] = Elem<T>::load(vh, (int64_t)pid[i] * d + c);
    }
    __syncthreads();
    for (int e = tid; e < P * (P + 1) / 2; e += NT) {
        int i = 0, rem = e;
        while (rem >= P - i) { rem -= P - i; ++i; }
        const int j = i + rem;
        double acc = 0.0;
        for (int c = 0; c < d; ++c) acc = fma((double)Vs[i * pitch + c] - mu[c], (double)Vs[j * pitch + c] - mu[c], acc);
        const double g = ps[i] * ps[j] * acc;
        Gm[i * P + j] = g;
        Gm[j * P + i] = g;
    }
    if (tid == 0) ctr[0] = 0;
    __syncthreads();

    // ---- 4. ES_pool --------------------------------------------------------------
    const uint64_t best = enum_best(a.pl, Gm, ps, seed, a.tab.io, a.tab.wmk, a.tab.jobs, a.tab.omk, ent, PLt,
                                    redd, redm, ctr);

    // ---- 5. balancing within the pool --------------------------------------------
    const uint64_t all = P == 64 ? ~0ull : ((1ull << P) - 1ull);
    uint64_t A = seed;
    int swaps = 0;
    if (s < P) {
        // Gram value of the current set, recomputed exactly after every swap
        auto gram_of = [&](uint64_t M, double &S, double &PA) {
            double v = 0.0, pm = 0.0;
            for (int e = tid; e < P * P; e += NT) {
                const int i = e / P, j = e % P;
                if (((M >> i) & 1ull) && ((M >> j) & 1ull)) v += Gm[e];
            }
            for (int i = tid; i < P; i += NT)
                if ((M >> i) & 1ull) pm += ps[i];
            S = block_sum(v, redd);
            PA = block_sum(pm, redd);
        };
        double S, PA;
        gram_of(A, S, PA);
        double cur = S / (PA * PA);
        const int nout = P - s;
        while (swaps < a.max_swaps) {
            for (int x = tid; x < P; x += NT) {
                double c = 0.0;
                for (int y = 0; y < P; ++y)
                    if ((A >> y) & 1ull) c += Gm[x * P + y];
                cv[x] = c;
            }
            __syncthreads();
            double bv = 0.0;
            int64_t bi = -1;
            for (int t = tid; t < s * nout; t += NT) {
                const int ii = t / nout, jj = t % nout;
                // ii-th member and jj-th non-member of A, ascending
                int i = -1, j = -1;
                {
                    int ci = 0, cj = 0;
                    for (int x = 0; x < P; ++x) {
                        if ((A >> x) & 1ull) { if (ci++ == ii) i = x; }
                        else if (cj++ == jj) j = x;
                    }
                }
                if (i < 0 || j < 0) continue;  // A always holds s of the P keys
                const double Sn = S - 2.0 * cv[i] + Gm[i * P + i] + 2.0 * (cv[j] - Gm[i * P + j]) + Gm[j * P + j];
                const double Pn = PA - ps[i] + ps[j];
                const double val = fmax(Sn, 0.0) / (Pn * Pn);
                // argmax of -val; ties to the smallest (out, in) = smallest t
                if (bi < 0 || -val > bv) { bv = -val; bi = t; }
            }
            block_argmax(bv, bi, redd, redi);
            if (bi < 0 || !(-bv < cur)) break;
            const int ii = (int)(bi / nout), jj = (int)(bi % nout);
            int i = -1, j = -1;
            {
                int ci = 0, cj = 0;
                for (int x = 0; x < P; ++x) {
                    if ((A >> x) & 1ull) { if (ci++ == ii) i = x; }
                    else if (cj++ == jj) j = x;
                }
            }
            if (i < 0 || j < 0) break;
            A = (A & ~(1ull << i)) | (1ull << j);
            ++swaps;
            gram_of(A, S, PA);
            cur = S / (PA * PA);
        }
        (void)all;
    }

    // ---- 6. reported errors and statistics -------------------------------------
    // es(M) = ||sum_{i in M} p_i (v_i - mu)|| / p(M) over the pool's staged rows
    auto es_of = [&](uint64_t M) {
        if ((int64_t)__popcll(M) == N) return 0.0;
        double g2 = 0.0;
        for (int c = tid; c < d; c += NT) {
            double g = 0.0;
            for (uint64_t m = M; m; m &= m - 1) {
                const int i = __ffsll((unsigned long long)m) - 1;
                g = fma(ps[i], (double)Vs[i * pitch + c] - mu[c], g);
            }
            g2 = fma(g, g, g2);
        }
        g2 = block_sum(g2, redd);
        double pm = 0.0;
        for (uint64_t m = M; m; m &= m - 1) pm += ps[__ffsll((unsigned long long)m) - 1];
        return sqrt(g2) / pm;
    };
    const double es_top = es_of(seed);
    const double es_pool = es_of(best);
    const double es_bal = es_of(A);
    if (tid == 0) {
        int t = 0, u = 0;
        for (int i = 0; i < P; ++i) {
            if (((best >> i) & 1ull) && t < s) a.best_idx[r * s + t++] = pid[i];
            if (a.bal_idx && ((A >> i) & 1ull) && u < s) a.bal_idx[r * s + u++] = pid[i];
        }
        if (a.n_swaps) a.n_swaps[r] = swaps;
        const double m = sc[0], sigma = sqrt(sc[1]), D = sc[2];
        double ptop = 0.0;
        for (int i = 0; i < P; ++i)
            if ((seed >> i) & 1ull) ptop += ps[i];
        auto ratio = [](double num, double den) {
            return den > 0.0 ? num / den : (num == 0.0 ? 1.0 : (double)INFINITY);
        };
        float *o = a.stats + r * FW_POOL_NSTATS;
        o[0] = (float)es_top;
        o[1] = (float)es_pool;
        o[2] = (float)es_bal;
        o[3] = (float)ratio(es_top, es_pool);
        o[4] = (float)(es_top > 0.0 ? 1.0 - es_pool / es_top : 0.0);
        o[5] = (float)ratio(es_bal, es_pool);
        o[6] = (float)m;
        o[7] = (float)(es_top * ptop);
        o[8] = (float)D;
        o[9] = (float)sigma;
        o[10] = (float)(2.0 * D * m);
        o[11] = (float)(m < 1.0 ? sqrt(m / (1.0 - m)) * sigma : (double)INFINITY);
    }
}

// Per cell: the median of the dropped mass over its G rows (the mean of the
// two middle values for even G), and the flat label median > threshold.
__global__ void __launch_bounds__(256) pool_cell_kernel(const float *stats, int64_t G, float threshold,
                                                        float *cell_median, uint8_t *cell_flat) {
    __shared__ float lo_hi[2];
    const int64_t h = blockIdx.x;
    const int64_t lo = (G - 1) / 2, hi = G / 2;
    for (int64_t g = threadIdx.x; g < G; g += blockDim.x) {
        const float x = stats[(h * G + g) * FW_POOL_NSTATS + 6];
        int64_t rank = 0;
        for (int64_t u = 0; u < G; ++u) {
            const float y = stats[(h * G + u) * FW_POOL_NSTATS + 6];
            rank += (y < x) || (y == x && u < g);
        }
        if (rank == lo) lo_hi[0] = x;
        if (rank == hi) lo_hi[1] = x;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const float med = (float)(0.5 * ((double)lo_hi[0] + (double)lo_hi[1]));
        if (cell_median) cell_median[h] = med;
        if (cell_flat) cell_flat[h] = med > threshold ? 1 : 0;
    }
}

// ---------------------------------------------------------------------------
bool pool_plan(int64_t N, int d, int s, int extra, EnumPlan *pl, size_t *lds) {
    const int P = s + extra;
    if (P > kPoolMax || P > N || s < 1) return false;
    if (binom(P, s) >= (1ull << 31)) return false;
    EnumPlan p;
    if (!choose_plan(P, s, &p)) return false;
    p.d = d;
    p.G = 1;
    const size_t L = pool_lds(N, d, P, p.nent).total;
    if (L > 160 * 1024) return false;
    if (pl) *pl = p;
    if (lds) *lds = L;
    return true;
}

size_t pool_ws_bytes(const fw_rows &rows, int s, int extra) {
    EnumPlan p;
    if (!pool_plan(rows.n, (int)rows.d, s, extra, &p, nullptr)) return 0;
    return enum_tables(p, nullptr).bytes;
}

hipError_t launch_pool(const fw_rows &rows, int s, int extra, int max_swaps, int32_t *pool_idx,
                       int32_t *best_idx, int32_t *bal_idx, int32_t *n_swaps, float *stats,
                       float flat_threshold, float *cell_median, uint8_t *cell_flat, void *ws,
                       hipStream_t st) {
    PoolArgs a{};
    size_t lds = 0;
    if (!pool_plan(rows.n, (int)rows.d, s, extra, &a.pl, &lds)) return hipErrorInvalidConfiguration;
    a.tab = enum_tables(a.pl, ws);
    hipError_t e = launch_enum_tables(a.pl, a.tab, st);
    if (e != hipSuccess) return e;
    a.q = rows.q;
    a.k = rows.k;
    a.v = rows.v;
    a.scale = rows.scale;
    a.bias = rows.bias;
    a.H = rows.H;
    a.G = rows.G;
    a.N = rows.n;
    a.d = (int)rows.d;
    a.s = s;
    a.extra = extra;
    a.max_swaps = max_swaps;
    a.pool_idx = pool_idx;
    a.best_idx = best_idx;
    a.bal_idx = bal_idx;
    a.n_swaps = n_swaps;
    a.stats = stats;
    const unsigned R = (unsigned)(rows.H * rows.G);
    if (rows.dtype == FW_BF16)
        hipLaunchKernelGGL(pool_row_kernel<uint16_t>, dim3(R), dim3(PT), lds, st, a);
    else
        hipLaunchKernelGGL(pool_row_kernel<float>, dim3(R), dim3(PT), lds, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (cell_median || cell_flat)
        hipLaunchKernelGGL(pool_cell_kernel, dim3((unsigned)rows.H), dim3(256), 0, st, stats, rows.G,
                           flat_threshold, cell_median, cell_flat);
    return hipGetLastError();
}

}  // namespace fw
