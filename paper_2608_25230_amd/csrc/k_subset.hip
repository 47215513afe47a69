// Exhaustive best kept set of size k (Section 2.2, Definition 2.5 with every
// key of the row as the candidate set), float64 throughout.
//
// Per row the kernel builds the instance of Definition 2.1 (weights p, dense
// output mu) and the Gram matrix Gm_ij = u_i . u_j of the residuals
// u_j = p_j (v_j - mu).  By Lemma 2.2, es(A)^2 = ||g_A||^2 / p(A)^2 with
// g_A = sum_{j in A} u_j, so ||g_A||^2 = sum_{i,j in A} Gm_ij: a subset is
// scored from Gram entries, not from d-dimensional sums.
//
// Enumeration.  Every k-subset A splits into its top kt = k - kw elements T
// and its kw smallest elements L, all below b = min T.  A lane takes one T
// and walks every L in revolving-door order over {0..b-1}; all lanes of a
// wave step through the same (in, out) sequence, so the per-step values
// shared by the wave (the Gram sum S_L and mass P_L of L) come from per-row
// tables.  Against the lane's best ratio beta the test
//     f = S(A) - beta * P(A)^2 <= 0
// is linear in the walk: S(A) - beta P(A)^2 = K1 + sum_{x in L} e[x]
//     + S_L - beta P_L^2, with K1 = S_T - beta P_T^2 and
//     e[x] = 2 sum_{a in T} Gm_xa - 2 beta P_T p_x,
// so each step costs two reads of e and a few adds.  Subsets that pass are
// scored exactly (S / P^2, ties to the lexicographically smaller set) and
// lower beta.  The top-k set seeds every lane, so the answer is never worse
// than top-k.  Reported gaps are recomputed from the d-dimensional residual
// sums of the chosen sets.
#include "fw_internal.hpp"
#include "instance64.hpp"
#include "revdoor.hpp"

namespace fw {

namespace {

constexpr int kSubsetThreads = 256;  // upper bound; the launch may use 128 or 64

struct SubsetPlan {
    int n, k, d;
    int kw;      // walk size
    int kt;      // lane-owned top part size
    int B;       // largest walk range
    int nsteps;  // C(B, kw)
    int ntasks;  // number of T sets
    int G;
};

SubsetPlan make_plan(int64_t n, int k, int64_t d, int64_t G, int max_steps = 2048) {
    SubsetPlan p{};
    p.n = (int)n;
    p.k = k;
    p.d = (int)d;
    p.G = (int)G;
    int kw = k < 3 ? k : 3;
    for (;;) {
        int kt = k - kw;
        int B = (kt == 0) ? (int)n : (int)n - kt;
        uint64_t steps = binom(B, kw);
        if (steps <= (uint64_t)max_steps || kw == 1) {
            p.kw = kw;
            p.kt = kt;
            p.B = B;
            p.nsteps = (int)steps;
            break;
        }
        --kw;
    }
    // tasks: T = {b} + (kt-1)-subset of (b, n), b from n-kt down to kw
    if (p.kt == 0) {
        p.ntasks = 1;
    } else {
        uint64_t tot = 0;
        for (int b = p.n - p.kt; b >= p.kw; --b) tot += binom(p.n - 1 - b, p.kt - 1);
        p.ntasks = (int)tot;
    }
    return p;
}

struct SubsetLds {
    size_t gm, pz, mu, tab, lm, r0, io, cnt, red, total;
};

__host__ __device__ inline SubsetLds subset_lds(const SubsetPlan &p, int nt) {
    SubsetLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.gm = take((size_t)p.n * p.n * 8);
    L.pz = take((size_t)p.n * 8 * 2);
    L.mu = take((size_t)p.d * 8);
    L.tab = take((size_t)p.nsteps * 8 * 3);
    L.lm = take((size_t)p.nsteps * 8);
    size_t r0a = (size_t)p.n * p.d * 4, r0b = (size_t)p.B * nt * 8;
    L.r0 = take(r0a > r0b ? r0a : r0b);
    L.io = take((size_t)p.nsteps * 2);
    L.cnt = take(66 * 4);
    L.red = take((size_t)nt * 16);
    L.total = o;
    return L;
}

}  // namespace

__global__ void revdoor_table_kernel(int B, int kw, uint8_t *inout, uint64_t *lmask) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int c[68];
    revdoor_init(c, kw, B);
    uint64_t m = 0;
    for (int j = 0; j < kw; ++j) m |= 1ull << j;
    lmask[0] = m;
    inout[0] = inout[1] = 0;
    int t = 1, in, out;
    while (revdoor_next(c, kw, &in, &out)) {
        m ^= (1ull << in) ^ (1ull << out);
        inout[2 * t] = (uint8_t)in;
        inout[2 * t + 1] = (uint8_t)out;
        lmask[t] = m;
        ++t;
    }
}

template <typename T>
__global__ void __launch_bounds__(kSubsetThreads)
best_subset_kernel(const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
                   const float *__restrict__ scale, const float *__restrict__ bias, SubsetPlan pl,
                   const uint8_t *__restrict__ g_inout, const uint64_t *__restrict__ g_lmask,
                   int32_t *best_idx, float *best_gap, float *topk_gap, float *closed,
                   float *dropped_topk, int32_t *topk_idx) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int NT = blockDim.x;
    const SubsetLds L = subset_lds(pl, NT);
    double *Gm = (double *)(smem + L.gm);
    double *ps = (double *)(smem + L.pz);
    double *zs = ps + pl.n;
    double *mu = (double *)(smem + L.mu);
    double *SL = (double *)(smem + L.tab);
    double *PL = SL + pl.nsteps;
    double *PL2 = PL + pl.nsteps;
    uint64_t *lm = (uint64_t *)(smem + L.lm);
    float *Vs = (float *)(smem + L.r0);
    double *et = (double *)(smem + L.r0);
    uint8_t *io = (uint8_t *)(smem + L.io);
    int *cnt = (int *)(smem + L.cnt);
    double *redd = (double *)(smem + L.red);
    uint64_t *redm = (uint64_t *)(redd + NT);

    const int n = pl.n, d = pl.d, kk = pl.k;
    const int tid = threadIdx.x;
    const int64_t r = blockIdx.x;
    const int64_t h = r / pl.G;
    const T *qr = q + r * d;
    const T *kh = k + h * (int64_t)n * d;
    const T *vh = v + h * (int64_t)n * d;

    for (int e = tid; e < pl.nsteps * 2; e += NT) io[e] = g_inout[e];
    for (int e = tid; e < pl.nsteps; e += NT) lm[e] = g_lmask[e];
    instance64(qr, kh, vh, scale ? scale[h] : default_scale(d), bias, n, d, Vs, zs, ps, mu, Gm);
    // top-k set: rank by (z desc, index asc)
    const uint64_t top_mask = topk_mask64(zs, n, kk, topk_idx ? topk_idx + r * kk : nullptr, redm);
    // per-row walk tables, and the task offsets per b
    for (int t = tid; t < pl.nsteps; t += NT) {
        uint64_t m = lm[t];
        double P = 0.0, S = 0.0;
        for (uint64_t a = m; a; a &= a - 1) {
            int x = __ffsll((unsigned long long)a) - 1;
            P += ps[x];
            for (uint64_t b2 = m; b2; b2 &= b2 - 1) S += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
        }
        SL[t] = S;
        PL[t] = P;
        PL2[t] = P * P;
    }
    if (tid == 0) {
        int acc = 0, i = 0;
        if (pl.kt > 0)
            for (int b = n - pl.kt; b >= pl.kw; --b, ++i) {
                cnt[i] = acc;
                acc += (int)binom(n - 1 - b, pl.kt - 1);
            }
        cnt[i] = acc;
    }
    __syncthreads();  // Vs is dead from here: its space holds the lane arrays

    // seed: the top-k set, scored from the Gram
    double S_top = 0.0, P_top = 0.0;
    for (uint64_t a = top_mask; a; a &= a - 1) {
        int x = __ffsll((unsigned long long)a) - 1;
        P_top += ps[x];
        for (uint64_t b2 = top_mask; b2; b2 &= b2 - 1) S_top += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
    }
    double best_val = S_top / (P_top * P_top);
    uint64_t best_mask = top_mask;
    double beta = best_val;

    for (int task = tid; task < pl.ntasks; task += NT) {
        // decode T and b
        int b;
        uint64_t Tm = 0;
        if (pl.kt == 0) {
            b = n;
        } else {
            int i = 0;
            b = n - pl.kt;
            while (task >= cnt[i + 1]) { ++i; --b; }
            int rr = task - cnt[i];
            Tm = 1ull << b;
            // colex unrank of rr among (kt-1)-subsets of {0..n-2-b}, shifted by b+1
            for (int s = pl.kt - 1; s >= 1; --s) {
                int c = s - 1;
                while ((int)binom(c + 1, s) <= rr) ++c;
                rr -= (int)binom(c, s);
                Tm |= 1ull << (b + 1 + c);
            }
        }
        double PT = 0.0, ST = 0.0;
        for (uint64_t a = Tm; a; a &= a - 1) {
            int x = __ffsll((unsigned long long)a) - 1;
            PT += ps[x];
            for (uint64_t b2 = Tm; b2; b2 &= b2 - 1) ST += Gm[x * n + (__ffsll((unsigned long long)b2) - 1)];
        }
        for (int x = 0; x < b; ++x) {
            double Ex = 0.0;
            for (uint64_t a = Tm; a; a &= a - 1) Ex += Gm[x * n + (__ffsll((unsigned long long)a) - 1)];
            et[x * NT + tid] = 2.0 * Ex - 2.0 * beta * PT * ps[x];
        }
        double K1 = ST - beta * PT * PT;
        double X = 0.0;
        for (int x = 0; x < pl.kw; ++x) X += et[x * NT + tid];
        const int nst = (int)binom(b, pl.kw);
        for (int t = 0; t < nst; ++t) {
            if (t > 0) {
                const int in = io[2 * t], out = io[2 * t + 1];
                X += et[in * NT + tid] - et[out * NT + tid];
            }
            const double f = X + K1 + SL[t] - beta * PL2[t];
            if (f <= 1e-12 * beta) {
                const uint64_t Lm = lm[t];
                const uint64_t mask = Tm | Lm;
                double S = ST + SL[t];
                for (uint64_t a = Lm; a; a &= a - 1) {
                    int x = __ffsll((unsigned long long)a) - 1;
                    double Ex = 0.0;
                    for (uint64_t c2 = Tm; c2; c2 &= c2 - 1) Ex += Gm[x * n + (__ffsll((unsigned long long)c2) - 1)];
                    S += 2.0 * Ex;
                }
                const double P = PT + PL[t];
                const double val = S / (P * P);
                if (val < best_val || (val == best_val && lex_less(mask, best_mask))) {
                    const double dB = val - beta;
                    for (int x = 0; x < b; ++x) et[x * NT + tid] -= 2.0 * dB * PT * ps[x];
                    best_val = val;
                    best_mask = mask;
                    beta = val;
                    K1 = ST - beta * PT * PT;
                    X = 0.0;
                    for (uint64_t a = Lm; a; a &= a - 1)
                        X += et[(__ffsll((unsigned long long)a) - 1) * NT + tid];
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

// Largest walk cap and thread count whose LDS fits in 160 KiB.
static bool choose_plan(int64_t n, int k, int64_t d, int64_t G, SubsetPlan *plan, int *nt) {
    for (int cap = 2048; cap >= 64; cap >>= 1) {
        for (int t = 256; t >= 64; t >>= 1) {
            SubsetPlan p = make_plan(n, k, d, G, cap);
            if (subset_lds(p, t).total <= 160 * 1024) {
                *plan = p;
                *nt = t;
                return true;
            }
        }
    }
    return false;
}

size_t best_subset_ws_bytes(int64_t n, int k) {
    SubsetPlan p = make_plan(n, k, 1, 1);  // the largest walk any launch uses
    return align_up((size_t)p.nsteps * 2, 256) + (size_t)p.nsteps * 8;
}

hipError_t launch_best_subset(const fw_rows &rows, int k, int32_t *best_idx, float *best_gap,
                              float *topk_gap, float *closed, float *dropped_topk,
                              int32_t *topk_idx, void *ws, hipStream_t st) {
    SubsetPlan p;
    int nt;
    if (!choose_plan(rows.n, k, rows.d, rows.G, &p, &nt)) return hipErrorInvalidConfiguration;
    uint8_t *inout = (uint8_t *)ws;
    uint64_t *lmask = (uint64_t *)((char *)ws + align_up((size_t)p.nsteps * 2, 256));
    hipLaunchKernelGGL(revdoor_table_kernel, dim3(1), dim3(64), 0, st, p.B, p.kw, inout, lmask);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const SubsetLds L = subset_lds(p, nt);
    const unsigned R = (unsigned)(rows.H * rows.G);
    if (rows.dtype == FW_BF16)
        hipLaunchKernelGGL(best_subset_kernel<uint16_t>, dim3(R), dim3(nt), L.total, st,
                           (const uint16_t *)rows.q, (const uint16_t *)rows.k, (const uint16_t *)rows.v,
                           rows.scale, rows.bias, p, inout, lmask, best_idx, best_gap, topk_gap,
                           closed, dropped_topk, topk_idx);
    else
        hipLaunchKernelGGL(best_subset_kernel<float>, dim3(R), dim3(nt), L.total, st,
                           (const float *)rows.q, (const float *)rows.k, (const float *)rows.v,
                           rows.scale, rows.bias, p, inout, lmask, best_idx, best_gap, topk_gap,
                           closed, dropped_topk, topk_idx);
    return hipGetLastError();
}

}  // namespace fw
