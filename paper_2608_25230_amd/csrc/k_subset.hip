// Exhaustive best kept set of size k (Section 2.2, Definition 2.5 with every
// key of the row as the candidate set), float64 throughout.
//
// Per row the kernel builds the instance of Definition 2.1 (weights p, dense
// output mu) and the Gram matrix Gm_ij = u_i . u_j of the residuals
// u_j = p_j (v_j - mu).  By Lemma 2.2, es(A)^2 = ||g_A||^2 / p(A)^2 with
// g_A = sum_{j in A} u_j, so ||g_A||^2 = sum_{i,j in A} Gm_ij: a subset is
// scored from Gram entries, not from d-dimensional sums.
//
// Enumeration.  The keys split into a low range [0, m) and a high range
// [m, n); every k-subset is a high part H (|H| = h) plus a low part L
// (|L| = k - h).  A lane owns one H; the lanes of a wave, all with the same h,
// walk every L in the same revolving-door order over [0, m), so each step's
// entering and leaving keys are wave-uniform and the shared per-step values
// (S_L = sum_{x,y in L} Gm_xy and p(L)^2) come from per-row tables.  Against
// the wave's best ratio beta the test
//     f = S(A) - beta p(A)^2 <= 0
// is linear in the walk:
//     S(A) - beta p(A)^2 = K1 + sum_{x in L} e[x] + S_L - beta p(L)^2,
//     K1 = S_H - beta p(H)^2,   e[x] = 2 sum_{a in H} Gm_xa - 2 beta p(H) p_x,
// so one step is two register reads of e (indexed by the uniform keys), two
// adds, one multiply-add and a compare.  Subsets that pass are scored exactly
// (S / p^2 from the Gram, ties to the lexicographically smaller set), lower
// beta for the wave and rescale e.  The top-k set seeds every lane, so the
// answer is never worse than top-k.  Work items (h, a run of up to 64 high
// parts) are taken by the waves of the row's workgroup from a shared counter,
// longest walks first.  Reported gaps are recomputed from the d-dimensional
// residual sums of the chosen sets.
#include "fw_internal.hpp"
#include "instance64.hpp"
#include "revdoor.hpp"

namespace fw {

namespace {

constexpr int kSubsetThreads = 256;
constexpr int kMaxLow = 16;       // low range size (per-lane e[] in registers)
constexpr int kMaxEntries = 2048; // walk-table entries per row (LDS)

// Enumeration plan shared by host (sizes) and device (tables, jobs).
struct EnumPlan {
    int n, k, d, G;
    int m;             // low range [0, m)
    int hlo, hhi;      // high part sizes with work
    int nent;          // walk-table entries: sum over used walk sizes of C(m, kw)
    int njobs;
    int toff[kMaxLow + 1];  // first entry of the walk of size kw (-1 if unused)
};

__host__ __device__ inline int ceil64(uint64_t x) { return (int)((x + 63) / 64); }

__host__ __device__ inline bool plan_for(int n, int k, int m, EnumPlan *P) {
    EnumPlan p{};
    p.n = n;
    p.k = k;
    p.m = m;
    p.hlo = k - m > 0 ? k - m : 0;
    p.hhi = k < n - m ? k : n - m;
    if (p.hlo > p.hhi) return false;
    for (int kw = 0; kw <= kMaxLow; ++kw) p.toff[kw] = -1;
    uint64_t nent = 0, njobs = 0;
    for (int h = p.hlo; h <= p.hhi; ++h) {
        const int kw = k - h;
        p.toff[kw] = (int)nent;
        nent += binom(m, kw);
        njobs += (uint64_t)ceil64(binom(n - m, h));
    }
    if (nent > (uint64_t)kMaxEntries || njobs > (1u << 22)) return false;
    p.nent = (int)nent;
    p.njobs = (int)njobs;
    *P = p;
    return true;
}

// Estimated cost in wave-steps: walk steps of every job plus the per-lane
// set-up of its high part (about one step per nine instructions).
__host__ inline double plan_cost(const EnumPlan &p) {
    double c = 0.0;
    for (int h = p.hlo; h <= p.hhi; ++h) {
        const double jobs = (double)ceil64(binom(p.n - p.m, h));
        const double steps = (double)binom(p.m, p.k - h);
        const double setup = (double)(p.m * h + h * h + 3 * (p.n - p.m)) / 9.0;
        c += jobs * (steps + setup);
    }
    return c;
}

__host__ inline bool choose_plan(int64_t n, int k, EnumPlan *out) {
    bool found = false;
    double best = 0.0;
    const int mmax = n < kMaxLow ? (int)n : kMaxLow;
    for (int m = 1; m <= mmax; ++m) {
        EnumPlan p;
        if (!plan_for((int)n, k, m, &p)) continue;
        const double c = plan_cost(p);
        if (!found || c < best) {
            best = c;
            *out = p;
            found = true;
        }
    }
    return found;
}

// Job descriptor: h, kw, first high-part rank, lanes, steps, table offset.
struct EnumJob {
    int32_t h, kw, start, lanes, steps, toff;
};

struct SubsetLds {
    size_t gm, pz, mu, ent, pl, vs, pas, red, ctr, total;
};

__host__ __device__ inline SubsetLds subset_lds(int n, int d, int k, int nent, int nt) {
    SubsetLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.gm = take((size_t)n * n * 8);
    L.pz = take((size_t)n * 8 * 2);
    L.mu = take((size_t)d * 8);
    // walk tables overlay the values staged for the instance (dead by then)
    const size_t tab = (size_t)nent * 16 + (size_t)nent * 8;
    const size_t vsb = (size_t)n * d * 4;
    const size_t region = take(tab > vsb ? tab : vsb);
    L.ent = region;
    L.pl = region + (size_t)nent * 16;
    L.vs = region;
    L.pas = take((size_t)(n + 1) * (k + 1) * 4);
    L.red = take((size_t)nt * 16);
    L.ctr = take(16);
    L.total = o;
    return L;
}

}  // namespace

// Walk tables (row independent): for every used walk size kw the
// revolving-door sequence over [0, m) -- entry t holds the keys entering and
// leaving at step t (in | out << 8) and the mask of L_t -- and the job list,
// longest walks first.
__global__ void enum_plan_kernel(EnumPlan p, uint32_t *io, uint32_t *lmk, EnumJob *jobs) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int c[kMaxLow + 2];
    for (int h = p.hlo; h <= p.hhi; ++h) {
        const int kw = p.k - h;
        int t = p.toff[kw];
        uint32_t mask = kw == 0 ? 0u : ((kw >= 32) ? 0xFFFFFFFFu : ((1u << kw) - 1u));
        io[t] = 0;
        lmk[t] = mask;
        if (kw > 0 && kw < p.m) {
            revdoor_init(c, kw, p.m);
            int in, out;
            while (revdoor_next(c, kw, &in, &out)) {
                ++t;
                mask ^= (1u << in) ^ (1u << out);
                io[t] = (uint32_t)in | ((uint32_t)out << 8);
                lmk[t] = mask;
            }
        }
    }
    // jobs, grouped by h in order of decreasing walk length
    int nj = 0;
    bool done[kMaxLow + 48];
    for (int h = 0; h <= p.hhi; ++h) done[h] = h < p.hlo;
    for (int round = p.hlo; round <= p.hhi; ++round) {
        int hb = -1;
        uint64_t best = 0;
        for (int h = p.hlo; h <= p.hhi; ++h)
            if (!done[h] && (hb < 0 || binom(p.m, p.k - h) > best)) { hb = h; best = binom(p.m, p.k - hb); }
        done[hb] = true;
        const uint64_t tot = binom(p.n - p.m, hb);
        for (uint64_t s = 0; s < tot; s += 64) {
            EnumJob j;
            j.h = hb;
            j.kw = p.k - hb;
            j.start = (int32_t)s;
            j.lanes = (int32_t)((tot - s) < 64 ? (tot - s) : 64);
            j.steps = (int32_t)binom(p.m, p.k - hb);
            j.toff = p.toff[p.k - hb];
            jobs[nj++] = j;
        }
    }
}

template <typename T>
__global__ void __launch_bounds__(kSubsetThreads)
best_subset_kernel(const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
                   const float *__restrict__ scale, const float *__restrict__ bias, EnumPlan pl,
                   const uint32_t *__restrict__ g_io, const uint32_t *__restrict__ g_lmk,
                   const EnumJob *__restrict__ g_jobs, int32_t *best_idx, float *best_gap,
                   float *topk_gap, float *closed, float *dropped_topk, int32_t *topk_idx) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int NT = blockDim.x;
    const int n = pl.n, d = pl.d, kk = pl.k, m = pl.m;
    const SubsetLds L = subset_lds(n, d, kk, pl.nent, NT);
    double *Gm = (double *)(smem + L.gm);
    double *ps = (double *)(smem + L.pz);
    double *zs = ps + n;
    double *mu = (double *)(smem + L.mu);
    double2 *ent = (double2 *)(smem + L.ent);  // (S_L, p(L)^2)
    double *PLt = (double *)(smem + L.pl);     // p(L)
    float *Vs = (float *)(smem + L.vs);
    uint32_t *pas = (uint32_t *)(smem + L.pas);  // C(c, s), c <= n, s <= k (saturated)
    double *redd = (double *)(smem + L.red);
    uint64_t *redm = (uint64_t *)(redd + NT);
    int *ctr = (int *)(smem + L.ctr);

    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t r = blockIdx.x;
    const int64_t hh = r / pl.G;
    const T *qr = q + r * d;
    const T *kh = k + hh * (int64_t)n * d;
    const T *vh = v + hh * (int64_t)n * d;

    instance64(qr, kh, vh, scale ? scale[hh] : default_scale(d), bias, n, d, Vs, zs, ps, mu, Gm);
    // top-k set: rank by (z desc, index asc)
    const uint64_t top_mask = topk_mask64(zs, n, kk, topk_idx ? topk_idx + r * kk : nullptr, redm);
    // per-row walk tables (Vs is dead: instance64 ends with a barrier)
    for (int t = tid; t < pl.nent; t += NT) {
        const uint32_t lm = g_lmk[t];
        double P = 0.0, S = 0.0;
        for (uint32_t a = lm; a; a &= a - 1) {
            const int x = __ffs(a) - 1;
            P += ps[x];
            for (uint32_t b2 = lm; b2; b2 &= b2 - 1) S += Gm[x * n + (__ffs(b2) - 1)];
        }
        ent[t] = make_double2(S, P * P);
        PLt[t] = P;
    }
    for (int e = tid; e < (n + 1) * (kk + 1); e += NT) {
        const uint64_t b = binom(e / (kk + 1), e % (kk + 1));
        pas[e] = b > 0x7FFFFFFFull ? 0x7FFFFFFFu : (uint32_t)b;
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
    const int N = n - m;

    for (;;) {
        int jn = 0;
        if (lane == 0) jn = atomicAdd(ctr, 1);
        jn = __builtin_amdgcn_readfirstlane(__shfl(jn, 0));
        if (jn >= pl.njobs) break;
        const EnumJob jb = g_jobs[jn];
        const int h = jb.h, kw = jb.kw;
        const bool act = lane < jb.lanes;
        // high part of this lane: colex rank start + lane among h-subsets of [m, n)
        uint64_t Hm = 0;
        if (act) {
            uint32_t rr = (uint32_t)(jb.start + lane);
            int c = N - 1;
            for (int s = h; s >= 1; --s) {
                while (pas[c * (kk + 1) + s] > rr) --c;
                Hm |= 1ull << (m + c);
                rr -= pas[c * (kk + 1) + s];
                --c;
            }
        }
        double PH = 0.0, SH = 0.0;
        for (uint64_t a = Hm; a; a &= a - 1) {
            const int x = __ffsll((unsigned long long)a) - 1;
            PH += ps[x];
            for (uint64_t b2 = Hm; b2; b2 &= b2 - 1) SH += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
        }
        double e[kMaxLow];
#pragma unroll
        for (int x = 0; x < kMaxLow; ++x) {
            double E = 0.0;
            if (x < m)
                for (uint64_t a = Hm; a; a &= a - 1) E += Gm[x * n + (__ffsll((unsigned long long)a) - 1)];
            e[x] = (x < m) ? 2.0 * E - 2.0 * beta * PH * ps[x] : 0.0;
        }
        double K1 = SH - beta * PH * PH;
        double Y = K1;
        for (int x = 0; x < kw; ++x) Y += e[x];
        if (!act) Y = INFINITY;
        const uint32_t *io = g_io + jb.toff;
        const uint32_t *lmk = g_lmk + jb.toff;
        const double2 *en = ent + jb.toff;
        const double *plt = PLt + jb.toff;
        const int steps = jb.steps;
        double thr = 1e-12 * beta;
        // exact score of walk step t for this lane (a candidate)
        auto exact = [&](int t) {
            const uint32_t lm = lmk[t];
            double S = SH + en[t].x;
            for (uint32_t a = lm; a; a &= a - 1) {
                const int x = __ffs(a) - 1;
                double E = 0.0;
                for (uint64_t b2 = Hm; b2; b2 &= b2 - 1) E += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
                S += 2.0 * E;
            }
            const double P = PH + plt[t];
            const double val = S / (P * P);
            const uint64_t mask = Hm | (uint64_t)lm;
            if (val < best_val || (val == best_val && lex_less(mask, best_mask))) {
                best_val = val;
                best_mask = mask;
            }
        };
        // four steps per round: the step tables are loaded together and the
        // rare candidates handled after the four tests (a beta lowered within
        // the round only widens the filter of the remaining steps)
        for (int t0 = 0; t0 < steps; t0 += 4) {
            uint32_t w[4];
            double2 c[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int t = t0 + u;
                w[u] = (t > 0 && t < steps) ? io[t] : 0u;
                c[u] = (t < steps) ? en[t] : make_double2(INFINITY, 0.0);
            }
            bool cand[4];
            bool any = false;
            double y = Y;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                y += e[w[u] & 255u] - e[(w[u] >> 8) & 255u];
                const double f = y + fma(-beta, c[u].y, c[u].x);
                cand[u] = f <= thr;
                any |= cand[u];
            }
            Y = y;
            if (__ballot(any)) {  // rare: exact scores, then the wave's new beta
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (cand[u]) exact(t0 + u);
                double wb = best_val;
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) wb = fmin(wb, __shfl_xor(wb, off));
                if (wb < beta) {
                    const double dB = wb - beta;
#pragma unroll
                    for (int x = 0; x < kMaxLow; ++x)
                        if (x < m) e[x] -= 2.0 * dB * PH * ps[x];
                    beta = wb;
                    thr = 1e-12 * beta;
                    K1 = SH - beta * PH * PH;
                    // Y for the round's last step from the rescaled e
                    const int tl = (t0 + 3 < steps) ? t0 + 3 : steps - 1;
                    double yy = K1;
                    for (uint32_t a = lmk[tl]; a; a &= a - 1) yy += e[__ffs(a) - 1];
                    Y = act ? yy : INFINITY;
                }
            }
        }
    }
    // workgroup argmin with the lexicographic tie rule
    redd[tid] = best_val;
    redm[tid] = best_mask;
    __syncthreads();
    if (tid == 0) {
        for (int i = 1; i < NT; ++i) {
            if (redd[i] < redd[0] || (redd[i] == redd[0] && lex_less(redm[i], redm[0]))) {
                redd[0] = redd[i];
                redm[0] = redm[i];
            }
        }
    }
    __syncthreads();
    const uint64_t best = redm[0];
    __syncthreads();
    if (tid == 0) {
        int i = 0;
        for (uint64_t a = best; a; a &= a - 1) best_idx[r * kk + i++] = __ffsll((unsigned long long)a) - 1;
        if (dropped_topk) {
            double dm = 0.0;
            for (int j = 0; j < n; ++j)
                if (!((top_mask >> j) & 1ull)) dm += ps[j];
            dropped_topk[r] = (float)dm;
        }
    }
    const double es_best = exact_gap(best, n, vh, ps, mu, d, redd);
    const double es_top = exact_gap(top_mask, n, vh, ps, mu, d, redd);
    if (tid == 0) {
        best_gap[r] = (float)es_best;
        if (topk_gap) topk_gap[r] = (float)es_top;
        if (closed) {
            double c = (es_top > 0.0) ? 1.0 - es_best / es_top : 0.0;
            closed[r] = (float)(c < 0.0 ? 0.0 : (c > 1.0 ? 1.0 : c));
        }
    }
}

namespace {
struct SubsetWs {
    uint32_t *io, *lmk;
    EnumJob *jobs;
    size_t bytes;
};

SubsetWs subset_ws(const EnumPlan &p, void *ws) {
    SubsetWs W{};
    size_t off = 0;
    char *base = (char *)ws;
    auto take = [&](size_t bytes) -> void * {
        off = align_up(off, 256);
        void *ptr = base ? base + off : nullptr;
        off += bytes;
        return ptr;
    };
    W.io = (uint32_t *)take((size_t)p.nent * 4);
    W.lmk = (uint32_t *)take((size_t)p.nent * 4);
    W.jobs = (EnumJob *)take((size_t)p.njobs * sizeof(EnumJob));
    W.bytes = align_up(off, 256);
    return W;
}
}  // namespace

size_t best_subset_ws_bytes(int64_t n, int k) {
    EnumPlan p;
    if (!choose_plan(n, k, &p)) return 0;
    return subset_ws(p, nullptr).bytes;
}

bool best_subset_plannable(int64_t n, int k) {
    EnumPlan p;
    return choose_plan(n, k, &p);
}

hipError_t launch_best_subset(const fw_rows &rows, int k, int32_t *best_idx, float *best_gap,
                              float *topk_gap, float *closed, float *dropped_topk,
                              int32_t *topk_idx, void *ws, hipStream_t st) {
    EnumPlan p;
    if (!choose_plan(rows.n, k, &p)) return hipErrorInvalidConfiguration;
    p.d = (int)rows.d;
    p.G = (int)rows.G;
    const SubsetWs W = subset_ws(p, ws);
    hipLaunchKernelGGL(enum_plan_kernel, dim3(1), dim3(64), 0, st, p, W.io, W.lmk, W.jobs);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int nt = kSubsetThreads;
    const SubsetLds L = subset_lds(p.n, p.d, k, p.nent, nt);
    if (L.total > 160 * 1024) return hipErrorInvalidConfiguration;
    const unsigned R = (unsigned)(rows.H * rows.G);
    if (rows.dtype == FW_BF16)
        hipLaunchKernelGGL(best_subset_kernel<uint16_t>, dim3(R), dim3(nt), L.total, st,
                           (const uint16_t *)rows.q, (const uint16_t *)rows.k, (const uint16_t *)rows.v,
                           rows.scale, rows.bias, p, W.io, W.lmk, W.jobs, best_idx, best_gap, topk_gap,
                           closed, dropped_topk, topk_idx);
    else
        hipLaunchKernelGGL(best_subset_kernel<float>, dim3(R), dim3(nt), L.total, st,
                           (const float *)rows.q, (const float *)rows.k, (const float *)rows.v,
                           rows.scale, rows.bias, p, W.io, W.lmk, W.jobs, best_idx, best_gap, topk_gap,
                           closed, dropped_topk, topk_idx);
    return hipGetLastError();
}

}  // namespace fw
