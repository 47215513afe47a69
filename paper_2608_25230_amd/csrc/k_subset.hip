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
// (|L| = k - h).  For each h one of the two parts is owned by a lane and the
// other is walked: the lanes of a wave, all with the same h, walk every
// walked part in the same revolving-door order over its range (at most 16
// keys), so each step's entering and leaving keys are wave-uniform and the
// shared per-step values (S_W = sum_{x,y in W} Gm_xy and p(W)^2 of the walked
// part W) come from per-row tables.  With O the lane's own part, against the
// wave's best ratio beta the test
//     f = S(A) - beta p(A)^2 <= 0
// is linear in the walk:
//     S(A) - beta p(A)^2 = K1 + sum_{x in W} e[x] + S_W - beta p(W)^2,
//     K1 = S_O - beta p(O)^2,   e[x] = 2 sum_{a in O} Gm_xa - 2 beta p(O) p_x,
// so one step is two register reads of e (indexed by the uniform keys), two
// adds, one multiply-add and a compare.  Subsets that pass are scored exactly
// (S / p^2 from the Gram, ties to the lexicographically smaller set), lower
// beta for the wave and rescale e.  The top-k set seeds every lane, so the
// answer is never worse than top-k.  The plan picks m and, per h, which part
// the lanes own, to minimise walk steps plus per-lane set-up.  Work items
// (h, a run of up to 64 owned parts) are taken by the waves of the row's
// workgroup from a shared counter, longest first.  Reported gaps are
// recomputed from the d-dimensional residual sums of the chosen sets.
#include <type_traits>

#include "fw_internal.hpp"
#include "instance64.hpp"
#include "revdoor.hpp"
#include "enum_walk.hpp"

namespace fw {

namespace {

constexpr int kSubsetThreads = 256;

// Gram row pitch: odd, so that lanes reading different rows at one column
// fall on different LDS banks.
__host__ __device__ inline int gram_pitch(int n) { return n | 1; }

constexpr size_t kSubsetLdsKeep = 32 * 1024;  // five workgroups per CU

struct SubsetLds {
    size_t gm, pz, mu, ent, pl, vs, red, ctr, wt, total;
    bool keep_vs;
};

// ht: each wave also keeps the walk's step values at its own beta (nent
// doubles per wave)
__host__ __device__ inline SubsetLds subset_lds(int n, int d, int k, int nent, int nt, bool ht) {
    SubsetLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.gm = take((size_t)n * gram_pitch(n) * 8);
    L.pz = take((size_t)n * 8 * 2);
    L.mu = take((size_t)d * 8);
    const size_t tab = (size_t)nent * 16 + (size_t)nent * 8;
    const size_t vsb = (size_t)n * instance_pitch(d) * 4;
    L.red = take((size_t)(nt / 64) * 3 * 8);   // two doubles and one mask per wave
    L.ctr = take(16);
    L.wt = take(ht ? (size_t)(nt / 64) * nent * 8 : 0);
    // the values stay staged through the walk when that keeps five
    // workgroups per CU; otherwise the walk tables overlay them and they
    // are staged again for the reported errors
    L.keep_vs = o + tab + vsb + 32 <= kSubsetLdsKeep;
    const size_t region = take(L.keep_vs ? tab : (tab > vsb ? tab : vsb));
    L.ent = region;
    L.pl = region + (size_t)nent * 16;
    L.vs = L.keep_vs ? take(vsb) : region;
    L.total = o;
    return L;
}

}  // namespace

// Row-independent tables of a plan, one launch: blocks [0, 16 ncls) build
// the walk tables, block row y = b / 16 class y's table (unless an earlier
// class shares it), one entry per thread, each entry unranked on its own:
// colex order (parts of at most kColexMax keys) by the combinatorial number
// system, else the revolving-door order by revdoor_unrank, with the keys
// entering and leaving at step t (relative to the range) taken from the bits
// in which entry t differs from entry t - 1; masks hold absolute key
// positions.  The remaining blocks hold one job per wave: jobs run through
// the classes in plan order (the host orders them by decreasing job cost),
// ceil(count / 64) jobs per class, and lane l of job j holds the owned part
// of colex rank start + l (a key mask, and its first eight keys, ascending,
// one byte each).
__global__ void __launch_bounds__(256) enum_tables_kernel(EnumPlan p, uint2 *io, uint64_t *wmk, EnumJob *jobs,
                                                          uint64_t *omk) {
    const int ntab = 16 * p.ncls;
    if ((int)blockIdx.x < ntab) {
        const int y = blockIdx.x / 16, x = blockIdx.x % 16;
        const EnumClass &C = p.cls[y];
        for (int q2 = 0; q2 < y; ++q2)
            if (p.cls[q2].toff == C.toff) return;  // built by class q2
        const uint64_t cnt = binom(C.wn, C.ws), end = pad4(cnt);
        const bool colex = C.ws <= kColexMax;
        auto colex_mask = [&](uint64_t rr) {
            uint64_t m = 0;
            int c = C.wn - 1;
            for (int sz = C.ws; sz >= 1; --sz) {
                while (binom(c, sz) > rr) --c;
                m |= 1ull << c;
                rr -= binom(c, sz);
                --c;
            }
            return m;
        };
        for (uint64_t t = (uint64_t)x * blockDim.x + threadIdx.x; t < end; t += 16ull * blockDim.x) {
            const size_t at = (size_t)C.toff + t;
            if (t >= cnt) {  // neutral steps: no key moves, never a candidate
                io[at] = make_uint2(0u, 0u);
                wmk[at] = kPadMask;
                continue;
            }
            const uint64_t rel = colex ? colex_mask(t) : revdoor_unrank(t, C.wn, C.ws);
            uint2 st = make_uint2(0u, 0u);
            if (!colex && t > 0) {
                const uint64_t prev = revdoor_unrank(t - 1, C.wn, C.ws);
                st = make_uint2((uint32_t)(__ffsll((unsigned long long)(rel & ~prev)) - 1),
                                (uint32_t)(__ffsll((unsigned long long)(prev & ~rel)) - 1));
            }
            io[at] = st;
            wmk[at] = rel << C.wb;
        }
        return;
    }
    __shared__ int jfirst[kMaxClass + 1], jsteps[kMaxClass];
    __shared__ uint64_t jcount[kMaxClass];
    const int tid = threadIdx.x, lane = tid & 63;
    if (tid < p.ncls) {
        const EnumClass &C = p.cls[tid];
        jcount[tid] = owned_count(C);
        jfirst[tid + 1] = ceil64(jcount[tid]);
        jsteps[tid] = (int)pad4(binom(C.wn, C.ws));
    }
    __syncthreads();
    if (tid == 0) {
        jfirst[0] = 0;
        for (int q = 0; q < p.ncls; ++q) jfirst[q + 1] += jfirst[q];
    }
    __syncthreads();
    const int j = (blockIdx.x - ntab) * 4 + (tid >> 6);
    if (j >= p.njobs) return;
    int q = 0;
    while (q + 1 < p.ncls && jfirst[q + 1] <= j) ++q;
    const EnumClass &C = p.cls[q];
    const uint64_t s0 = (uint64_t)(j - jfirst[q]) * 64;
    const int nl = (jcount[q] - s0) < 64 ? (int)(jcount[q] - s0) : 64;
    if (lane == 0) {
        EnumJob jb;
        jb.cls = q;
        jb.start = (int32_t)s0;
        jb.lanes = nl;
        jb.steps = jsteps[q];
        jobs[j] = jb;
    }
    // the colex rank of an ls-subset of [lb, lb + ln) as a key mask
    auto unrank = [](uint64_t rr, int lb, int ln, int ls) {
        uint64_t m = 0;
        int c = ln - 1;
        for (int sz = ls; sz >= 1; --sz) {
            while (binom(c, sz) > rr) --c;
            m |= 1ull << (lb + c);
            rr -= binom(c, sz);
            --c;
        }
        return m;
    };
    uint64_t m = 0;
    if (lane < nl) {
        // rank = first part's rank x (second part's count) + second part's rank
        const uint64_t rr = s0 + lane;
        const uint64_t n2 = C.ln2 ? binom(C.ln2, C.ls2) : 1ull;
        m = unrank(rr / n2, C.lb, C.ln, C.ls);
        if (C.ln2) m |= unrank(rr % n2, C.lb2, C.ln2, C.ls2);
    }
    omk[(size_t)j * 64 + lane] = m;
    uint64_t keys = 0;
    for (int i = 0; i < 8 && m; ++i, m &= m - 1) keys |= (uint64_t)(__ffsll((unsigned long long)m) - 1) << (8 * i);
    omk[(size_t)(p.njobs + j) * 64 + lane] = keys;
}

template <typename T, int WMAX, bool HT, bool RD>
__global__ void __launch_bounds__(kSubsetThreads, 5)
best_subset_kernel(const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
                   const float *__restrict__ scale, const float *__restrict__ bias, EnumPlan pl,
                   const uint2 *__restrict__ g_io, const uint64_t *__restrict__ g_wmk,
                   const EnumJob *__restrict__ g_jobs, const uint64_t *__restrict__ g_omk,
                   int32_t *best_idx, float *best_gap,
                   float *topk_gap, float *closed, float *dropped_topk, int32_t *topk_idx) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int NT = blockDim.x;
    const int n = pl.n, d = pl.d, kk = pl.k;
    const SubsetLds L = subset_lds(n, d, kk, pl.nent, NT, HT);
    double *Gm = (double *)(smem + L.gm);
    double *ps = (double *)(smem + L.pz);
    double *zs = ps + n;
    double *mu = (double *)(smem + L.mu);
    double2 *ent = (double2 *)(smem + L.ent);  // (S_L, p(L)^2)
    double *PLt = (double *)(smem + L.pl);     // p(L)
    float *Vs = (float *)(smem + L.vs);
    double *redd = (double *)(smem + L.red);
    uint64_t *redm = (uint64_t *)(redd + 2 * (NT >> 6));
    int *ctr = (int *)(smem + L.ctr);
    double *wtab = (double *)(smem + L.wt);

    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t r = blockIdx.x;
    const int64_t hh = r / pl.G;
    const T *qr = q + r * d;
    const T *kh = k + hh * (int64_t)n * d;
    const T *vh = v + hh * (int64_t)n * d;

    instance64(qr, kh, vh, scale ? scale[hh] : default_scale(d), bias, n, d, Vs, zs, ps, mu, Gm, pl.gp);
    // top-k set: rank by (z desc, index asc)
    const uint64_t top_mask = topk_mask64(zs, n, kk, topk_idx ? topk_idx + r * kk : nullptr);
    // (instance64 ends with a barrier: the walk tables may overlay Vs)
    const uint64_t best = enum_best_body<WMAX, HT, RD>(pl, Gm, ps, top_mask, g_io, g_wmk, g_jobs, g_omk, ent, PLt, redd,
                                                   redm, ctr, false, nullptr, wtab);
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
    if (!L.keep_vs) {  // the values again (the walk tables that overlaid them are dead)
        stage_rows(vh, n, d, Vs, instance_pitch(d));
        __syncthreads();
    }
    const double2 es = exact_gap2_lds(best, top_mask, n, Vs, instance_pitch(d), ps, mu, d, redd);
    const double es_best = es.x, es_top = es.y;
    if (tid == 0) {
        best_gap[r] = (float)es_best;
        if (topk_gap) topk_gap[r] = (float)es_top;
        if (closed) {
            double c = (es_top > 0.0) ? 1.0 - es_best / es_top : 0.0;
            closed[r] = (float)(c < 0.0 ? 0.0 : (c > 1.0 ? 1.0 : c));
        }
    }
}

hipError_t launch_enum_tables(const EnumPlan &p, const EnumTables &W, hipStream_t st) {
    // up to kMaxEntries entries per table over 16 blocks of 256 threads, then
    // four jobs per block
    const unsigned nb = 16u * (unsigned)p.ncls + (unsigned)((p.njobs + 3) / 4);
    hipLaunchKernelGGL(enum_tables_kernel, dim3(nb), dim3(256), 0, st, p, W.io, W.wmk, W.jobs, W.omk);
    return hipGetLastError();
}

size_t best_subset_ws_bytes(int64_t n, int k) {
    EnumPlan p;
    if (!choose_plan(n, k, &p)) return 0;
    return enum_tables(p, nullptr).bytes;
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
    p.gp = gram_pitch(p.n);
    const EnumTables W = enum_tables(p, ws);
    hipError_t e = launch_enum_tables(p, W, st);
    if (e != hipSuccess) return e;
    const int nt = kSubsetThreads;
    // a narrower walk register file when every walked range allows it
    int wmax = 0;
    bool rd = false;  // some walked part takes the revolving-door order
    for (int q = 0; q < p.ncls; ++q) {
        wmax = p.cls[q].wn > wmax ? p.cls[q].wn : wmax;
        rd = rd || p.cls[q].ws > kColexMax;
    }
    // per-wave step values when they fit beside the staged values within five
    // workgroups per CU (at n = 24, k = 6 neither does: five workgroups per CU
    // without them ran 7 % faster than four with both)
    const SubsetLds Lh = subset_lds(p.n, p.d, k, p.nent, nt, true);
    const bool ht = Lh.keep_vs && Lh.total <= kSubsetLdsKeep;
    const SubsetLds L = ht ? Lh : subset_lds(p.n, p.d, k, p.nent, nt, false);
    if (L.total > 160 * 1024) return hipErrorInvalidConfiguration;
    const unsigned R = (unsigned)(rows.H * rows.G);
    auto go = [&](auto kern, const auto *q, const auto *k, const auto *v) {
        hipLaunchKernelGGL(kern, dim3(R), dim3(nt), L.total, st, q, k, v, rows.scale, rows.bias, p, W.io, W.wmk,
                           W.jobs, W.omk, best_idx, best_gap, topk_gap, closed, dropped_topk, topk_idx);
    };
    auto pick = [&](const auto *q, const auto *k, const auto *v) {
        using T = std::remove_cv_t<std::remove_pointer_t<decltype(q)>>;
        if (wmax <= 12) {
            if (ht) go(best_subset_kernel<T, 12, true, true>, q, k, v);
            else if (rd) go(best_subset_kernel<T, 12, false, true>, q, k, v);
            else go(best_subset_kernel<T, 12, false, false>, q, k, v);  // colex walks only
        } else {
            if (ht) go(best_subset_kernel<T, kMaxWalk, true, true>, q, k, v);
            else go(best_subset_kernel<T, kMaxWalk, false, true>, q, k, v);
        }
    };
    if (rows.dtype == FW_BF16)
        pick((const uint16_t *)rows.q, (const uint16_t *)rows.k, (const uint16_t *)rows.v);
    else
        pick((const float *)rows.q, (const float *)rows.k, (const float *)rows.v);
    return hipGetLastError();
}

}  // namespace fw
