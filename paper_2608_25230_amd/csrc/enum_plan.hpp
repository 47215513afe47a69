// Enumeration plan of every k-subset of n <= 64 keys (shared by the
// exhaustive best subset and the candidate-set search): the keys split into
// two or three consecutive ranges, and every k-subset into its parts in
// them.  A class fixes how many keys each range holds; in a class one range's
// part is walked in revolving-door order over that range (at most 16 keys)
// by all lanes of a wave in lockstep, and the other parts together are owned
// by a lane.  The host picks the split and, per class, the walked range, to
// minimise walk steps plus per-lane set-up; the device builds the walk tables
// and the job list from the plan.  Three ranges pay off when two would leave
// many classes with a long owned part and a walk of a step or two (a pool
// dropping six of 38 keys); the split with the lower estimated cost wins.
#pragma once

#include "fw_common.hpp"

namespace fw {

constexpr int kMaxWalk = 16;      // walked range size (per-lane e[] in registers)
constexpr int kMaxEntries = 4096; // walk-table entries per row (LDS)
constexpr int kMaxClass = 32;     // classes with work (plans needing more are not taken)
constexpr int kColexMax = 3;      // walked parts of at most this many keys run in colex order
constexpr int kFastOwned = 8;     // owned parts of at most this many keys take the unrolled set-up

// One class: the walked part and the one or two owned parts (16-bit
// fields: four budgets' plans travel in one kernel argument block).
struct EnumClass {
    int16_t wb, wn, ws;     // walked part: range [wb, wb + wn), size ws
    int16_t lb, ln, ls;     // owned part: range [lb, lb + ln), size ls
    int16_t lb2, ln2, ls2;  // second owned part (ln2 = 0: none)
    int16_t toff;           // first walk-table entry (< kMaxEntries)
};
__host__ __device__ inline int owned_keys(const EnumClass &C) { return C.ls + C.ls2; }
__host__ __device__ inline uint64_t owned_count(const EnumClass &C) {
    return binom(C.ln, C.ls) * (C.ln2 ? binom(C.ln2, C.ls2) : 1ull);
}

// Enumeration plan shared by host (sizes) and device (tables, jobs).
struct EnumPlan {
    int n, k, d, G;
    int gp;  // Gram row pitch (doubles), >= n
    int m, m2;  // ranges [0, m), [m, m2), [m2, n) (two ranges: m2 = n)
    int ncls;
    EnumClass cls[kMaxClass];
    int nent;  // walk-table entries
    int njobs;
};

__host__ __device__ inline int ceil64(uint64_t x) { return (int)((x + 63) / 64); }
// walks run in rounds of four steps; tables are padded with neutral steps
__host__ __device__ inline uint64_t pad4(uint64_t x) { return (x + 3) & ~(uint64_t)3; }
constexpr uint64_t kPadMask = ~(uint64_t)0;  // walk-table mask of a padding step

// Estimated instructions of one wave job: set-up of the owned part plus the
// walk.
__host__ __device__ inline double job_cost(int wn, int ws, int ln, int ls) {
    const double steps = (double)binom(wn, ws);
    double setup = 40.0 + 6.0 * ls * ls;  // the owned part comes from a table
    (void)ln;
    if (ws > 0) setup += ls * (1.5 * wn + 8.0) + 3.0 * wn;
    return setup + 10.0 * steps;
}

__host__ __device__ inline bool plan_for(int n, int k, int m, EnumPlan *P, double *cost) {
    EnumPlan p{};
    p.n = n;
    p.k = k;
    p.gp = n;
    p.m = m;
    p.m2 = n;
    const int N = n - m;
    const int hlo = k - m > 0 ? k - m : 0, hhi = k < N ? k : N;
    if (hlo > hhi || hhi - hlo + 1 > kMaxClass) return false;
    double total = 0.0;
    uint64_t nent = 0, njobs = 0;
    int toffA[kMaxWalk + 1], toffB[kMaxWalk + 1];
    for (int q = 0; q <= kMaxWalk; ++q) toffA[q] = toffB[q] = -1;
    for (int h = hlo; h <= hhi; ++h) {
        const int kw = k - h;
        // A: lanes own the high part, walk the low range; B: the reverse
        const bool okA = m <= kMaxWalk, okB = N <= kMaxWalk;
        if (!okA && !okB) return false;
        const double cA = okA ? ceil64(binom(N, h)) * job_cost(m, kw, N, h) : 0.0;
        const double cB = okB ? ceil64(binom(m, kw)) * job_cost(N, h, m, kw) : 0.0;
        const bool useA = okA && (!okB || cA <= cB);
        EnumClass c{};
        if (useA) {
            c.wb = 0; c.wn = m; c.ws = kw; c.lb = m; c.ln = N; c.ls = h;
            if (toffA[kw] < 0) { toffA[kw] = (int)nent; nent += pad4(binom(m, kw)); }
            c.toff = toffA[kw];
        } else {
            c.wb = m; c.wn = N; c.ws = h; c.lb = 0; c.ln = m; c.ls = kw;
            if (toffB[h] < 0) { toffB[h] = (int)nent; nent += pad4(binom(N, h)); }
            c.toff = toffB[h];
        }
        total += useA ? cA : cB;
        njobs += (uint64_t)ceil64(owned_count(c));
        p.cls[p.ncls++] = c;
    }
    if (nent > (uint64_t)kMaxEntries || njobs > (1u << 17)) return false;
    p.nent = (int)nent;
    p.njobs = (int)njobs;
    *P = p;
    *cost = total;
    return true;
}

// Three ranges [0, m1), [m1, m2), [m2, n): every split of k into (h0, h1, h2)
// is a class; its walked range is the one (of at most kMaxWalk keys) with the
// least estimated cost, the lanes owning the other two parts.
__host__ inline bool plan_for3(int n, int k, int m1, int m2, EnumPlan *P, double *cost) {
    EnumPlan p{};
    p.n = n;
    p.k = k;
    p.gp = n;
    p.m = m1;
    p.m2 = m2;
    const int rb[3] = {0, m1, m2}, rn[3] = {m1, m2 - m1, n - m2};
    int toff[3][kMaxWalk + 1];
    for (int r = 0; r < 3; ++r)
        for (int q = 0; q <= kMaxWalk; ++q) toff[r][q] = -1;
    double total = 0.0;
    uint64_t nent = 0, njobs = 0;
    for (int h0 = 0; h0 <= rn[0] && h0 <= k; ++h0)
        for (int h1 = 0; h1 <= rn[1] && h0 + h1 <= k; ++h1) {
            const int h2 = k - h0 - h1;
            if (h2 > rn[2]) continue;
            const int h[3] = {h0, h1, h2};
            int bw = -1;
            double bc = 0.0;
            for (int r = 0; r < 3; ++r) {
                if (rn[r] > kMaxWalk) continue;
                const int a = (r + 1) % 3, b = (r + 2) % 3;
                const double c = ceil64(binom(rn[a], h[a]) * binom(rn[b], h[b])) *
                                 job_cost(rn[r], h[r], rn[a] + rn[b], h[a] + h[b]);
                if (bw < 0 || c < bc) { bw = r; bc = c; }
            }
            if (bw < 0 || p.ncls == kMaxClass) return false;
            const int a = bw == 0 ? 1 : 0, b = bw == 2 ? 1 : 2;   // owned ranges, ascending
            EnumClass c{};
            c.wb = rb[bw]; c.wn = rn[bw]; c.ws = h[bw];
            c.lb = rb[a]; c.ln = rn[a]; c.ls = h[a];
            c.lb2 = rb[b]; c.ln2 = rn[b]; c.ls2 = h[b];
            if (toff[bw][c.ws] < 0) { toff[bw][c.ws] = (int)nent; nent += pad4(binom(c.wn, c.ws)); }
            c.toff = toff[bw][c.ws];
            total += bc;
            njobs += (uint64_t)ceil64(owned_count(c));
            p.cls[p.ncls++] = c;
        }
    if (nent > (uint64_t)kMaxEntries || njobs > (1u << 17)) return false;
    p.nent = (int)nent;
    p.njobs = (int)njobs;
    *P = p;
    *cost = total;
    return true;
}

// Classes in order of decreasing job cost (stable): the job list follows the
// class order, so the longest jobs are taken first.
__host__ inline void order_classes(EnumPlan *p) {
    double c[kMaxClass];
    for (int q = 0; q < p->ncls; ++q) {
        const EnumClass &C = p->cls[q];
        c[q] = job_cost(C.wn, C.ws, C.ln + C.ln2, owned_keys(C));
    }
    for (int i = 1; i < p->ncls; ++i)
        for (int j = i; j > 0 && c[j] > c[j - 1]; --j) {
            const EnumClass t = p->cls[j];
            p->cls[j] = p->cls[j - 1];
            p->cls[j - 1] = t;
            const double tc = c[j];
            c[j] = c[j - 1];
            c[j - 1] = tc;
        }
}

__host__ inline bool choose_plan(int64_t n, int k, EnumPlan *out, double *cost_out = nullptr) {
    bool found = false;
    double best = 0.0;
    auto take = [&](const EnumPlan &p, double c) {
        if (!found || c < best) {
            best = c;
            *out = p;
            found = true;
        }
    };
    for (int m = 1; m <= (int)n; ++m) {
        EnumPlan p;
        double c;
        if (plan_for((int)n, k, m, &p, &c)) take(p, c);
    }
    // Three ranges, near an even split (a few dozen candidates), only when
    // the estimate is well below the best two-range plan's: three ranges walk
    // shorter ranges, more of them in revolving-door order (dearer steps
    // than the colex walks the estimate prices), and their longer walk tables
    // can leave no LDS for the per-wave step values.  Measured: n = 38, k = 6
    // at 0.55 of the two-range estimate ran 2.1 times faster; n = 24, k = 6 at
    // 0.83 ran 1.24 times slower.
    const int N = (int)n;
    const bool two = found;
    const double best2 = best;
    // (skipped when the two-range plan is already small: the search costs
    // host time on every call, which a small enumeration would not recover)
    if (two && best2 < 1e5) {
        order_classes(out);
        if (cost_out) *cost_out = best;
        return true;
    }
    EnumPlan p3{};
    double c3 = 0.0;
    bool f3 = false;
    for (int m1 = N / 3 - 3; m1 <= N / 3 + 3; ++m1)
        for (int m2 = 2 * N / 3 - 3; m2 <= 2 * N / 3 + 3; ++m2) {
            if (m1 < 1 || m2 <= m1 || m2 >= N) continue;
            EnumPlan p;
            double c;
            if (plan_for3(N, k, m1, m2, &p, &c) && (!f3 || c < c3)) {
                p3 = p;
                c3 = c;
                f3 = true;
            }
        }
    if (f3 && (!two || c3 < 0.7 * best2)) {
        *out = p3;
        best = c3;
        found = true;
    }
    if (found) order_classes(out);
    if (found && cost_out) *cost_out = best;
    return found;
}

// Job descriptor: the class and a run of owned parts (colex ranks).
struct EnumJob {
    int32_t cls, start, lanes, steps;
};


// Row-independent tables of a plan in the caller's workspace: walk steps
// (io, wmk), the job list and each job's owned parts (omk: njobs x 64 key
// masks, then njobs x 64 lists of the first eight owned keys, ascending, one
// byte each).
struct EnumTables {
    uint2 *io;
    uint64_t *wmk;
    EnumJob *jobs;
    uint64_t *omk;
    size_t bytes;
};

__host__ inline EnumTables enum_tables(const EnumPlan &p, void *ws) {
    EnumTables W{};
    size_t off = 0;
    char *base = (char *)ws;
    auto take = [&](size_t bytes) -> void * {
        off = align_up(off, 256);
        void *ptr = base ? base + off : nullptr;
        off += bytes;
        return ptr;
    };
    W.io = (uint2 *)take((size_t)p.nent * 8);
    W.wmk = (uint64_t *)take((size_t)p.nent * 8);
    W.jobs = (EnumJob *)take((size_t)p.njobs * sizeof(EnumJob));
    W.omk = (uint64_t *)take((size_t)p.njobs * 64 * 8 * 2);
    W.bytes = align_up(off, 256);
    return W;
}

// k_subset.hip: fills the tables of a plan (one small launch on `st`).
hipError_t launch_enum_tables(const EnumPlan &p, const EnumTables &W, hipStream_t st);

}  // namespace fw
