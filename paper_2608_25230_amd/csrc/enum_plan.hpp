// Enumeration plan of every k-subset of n <= 64 keys (shared by the
// exhaustive best subset and the candidate-set search): the keys split into
// a low range [0, m) and a high range [m, n); every k-subset is a high part H
// (|H| = h) plus a low part (|L| = k - h).  For each h one part is owned by a
// lane and the other is walked in revolving-door order over its range (at
// most 16 keys) by all lanes of a wave in lockstep.  The host picks m and,
// per h, which part the lanes own, to minimise walk steps plus per-lane
// set-up; the device builds the walk tables and the job list from the plan.
#pragma once

#include "fw_common.hpp"

namespace fw {

constexpr int kMaxWalk = 16;      // walked range size (per-lane e[] in registers)
constexpr int kMaxEntries = 4096; // walk-table entries per row (LDS)
constexpr int kMaxClass = 17;     // values of h with work (min(m, n - m) + 1)
constexpr int kColexMax = 3;      // walked parts of at most this many keys run in colex order
constexpr int kFastOwned = 8;     // owned parts of at most this many keys take the unrolled set-up

// One value of h: which part the lanes own and which is walked.
struct EnumClass {
    int h;
    int wb, wn, ws;  // walked part: range [wb, wb + wn), size ws
    int lb, ln, ls;  // owned part: range [lb, lb + ln), size ls
    int toff;        // first walk-table entry
};

// Enumeration plan shared by host (sizes) and device (tables, jobs).
struct EnumPlan {
    int n, k, d, G;
    int gp;  // Gram row pitch (doubles), >= n
    int m;
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
        EnumClass c;
        c.h = h;
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
        njobs += (uint64_t)ceil64(binom(c.ln, c.ls));
        p.cls[p.ncls++] = c;
    }
    if (nent > (uint64_t)kMaxEntries || njobs > (1u << 17)) return false;
    p.nent = (int)nent;
    p.njobs = (int)njobs;
    *P = p;
    *cost = total;
    return true;
}

__host__ inline bool choose_plan(int64_t n, int k, EnumPlan *out, double *cost_out = nullptr) {
    bool found = false;
    double best = 0.0;
    for (int m = 1; m <= (int)n; ++m) {
        EnumPlan p;
        double c;
        if (!plan_for((int)n, k, m, &p, &c)) continue;
        if (!found || c < best) {
            best = c;
            *out = p;
            found = true;
        }
    }
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

// k_subset.hip: fills the tables of a plan (two small launches on `st`).
hipError_t launch_enum_tables(const EnumPlan &p, const EnumTables &W, hipStream_t st);

}  // namespace fw
