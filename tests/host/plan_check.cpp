// Host check of the enumeration plans (enum_plan.hpp) and of the owned-part
// unranking the table kernel uses: for each (n, k), the classes of the chosen
// plan (in order of decreasing job cost), each an owned part (one or two
// ranges) times a walked part, cover every k-subset of {0..n-1} exactly once.
// Also the walk tables' entries as the table kernel forms them, each on its
// own (colex by the combinatorial number system, revolving door by unranking,
// a step's keys from the bits in which it differs from the step before),
// against the sequential walks (Gosper's successor, Algorithm R).  Prints
// "plans OK" on success.
#include <cstdio>
#include <cstdint>
#include <unordered_set>
#include <utility>
#include <vector>

#include "enum_plan.hpp"
#include "revdoor.hpp"

using namespace fw;

// the colex rank of an ls-subset of [lb, lb + ln) as a key mask (the job
// kernel's rule)
static uint64_t unrank(uint64_t rr, int lb, int ln, int ls) {
    uint64_t m = 0;
    int c = ln - 1;
    for (int sz = ls; sz >= 1; --sz) {
        while (binom(c, sz) > rr) --c;
        m |= 1ull << (lb + c);
        rr -= binom(c, sz);
        --c;
    }
    return m;
}

static bool check(int n, int k, bool enumerate) {
    EnumPlan p;
    double cost;
    if (!choose_plan(n, k, &p, &cost)) {
        printf("n=%d k=%d: no plan\n", n, k);
        return false;
    }
    printf("n=%d k=%d: ranges [0,%d) [%d,%d) [%d,%d), %d classes, %d jobs, %d table entries\n", n, k, p.m, p.m,
           p.m2, p.m2, n, p.ncls, p.njobs, p.nent);
    uint64_t total = 0;
    int jobs = 0;
    for (int q = 1; q < p.ncls; ++q) {  // longest jobs first
        const EnumClass &A = p.cls[q - 1], &B = p.cls[q];
        if (job_cost(A.wn, A.ws, A.ln + A.ln2, owned_keys(A)) < job_cost(B.wn, B.ws, B.ln + B.ln2, owned_keys(B))) {
            printf("  classes out of job-cost order\n");
            return false;
        }
    }
    std::unordered_set<uint64_t> seen;
    for (int q = 0; q < p.ncls; ++q) {
        const EnumClass &C = p.cls[q];
        if (C.wn > kMaxWalk || C.ws > C.wn || owned_keys(C) + C.ws != k) {
            printf("  class %d: malformed\n", q);
            return false;
        }
        const uint64_t own = owned_count(C), walk = binom(C.wn, C.ws);
        total += own * walk;
        jobs += ceil64(own);
        if (!enumerate) continue;
        std::vector<uint64_t> W;
        for (uint64_t r = 0; r < walk; ++r) W.push_back(unrank(r, C.wb, C.wn, C.ws));
        const uint64_t n2 = C.ln2 ? binom(C.ln2, C.ls2) : 1ull;
        for (uint64_t r = 0; r < own; ++r) {
            uint64_t m = unrank(r / n2, C.lb, C.ln, C.ls);
            if (C.ln2) m |= unrank(r % n2, C.lb2, C.ln2, C.ls2);
            for (uint64_t w : W) {
                const uint64_t all = n == 64 ? ~0ull : (1ull << n) - 1ull;
                if ((m & w) || __builtin_popcountll(m | w) != k || ((m | w) & ~all)) {
                    printf("  class %d: a malformed subset\n", q);
                    return false;
                }
                if (!seen.insert(m | w).second) {
                    printf("  subset listed twice\n");
                    return false;
                }
            }
        }
    }
    if (total != binom(n, k) || jobs != p.njobs) {
        printf("  %llu subsets of %llu, %d jobs of %d\n", (unsigned long long)total,
               (unsigned long long)binom(n, k), jobs, p.njobs);
        return false;
    }
    return !enumerate || seen.size() == binom(n, k);
}

static bool tables_match() {
    for (int wn = 1; wn <= kMaxWalk; ++wn)
        for (int ws = 0; ws <= wn; ++ws) {
            const uint64_t cnt = binom(wn, ws);
            std::vector<uint64_t> seq;
            std::vector<std::pair<int, int>> steps;
            uint32_t rel = ws == 0 ? 0u : ((1u << ws) - 1u);
            seq.push_back(rel);
            steps.push_back({0, 0});
            if (ws <= kColexMax) {
                for (uint64_t e = 1; e < cnt; ++e) {
                    const uint32_t low = rel & (~rel + 1u), r = rel + low;
                    rel = (((r ^ rel) >> 2) >> (__builtin_ffs(low) - 1)) | r;
                    seq.push_back(rel);
                    steps.push_back({0, 0});
                }
            } else if (ws > 0 && ws < wn) {
                int c[kMaxWalk + 2], in, out;
                revdoor_init(c, ws, wn);
                while (revdoor_next(c, ws, &in, &out)) {
                    rel ^= (1u << in) ^ (1u << out);
                    seq.push_back(rel);
                    steps.push_back({in, out});
                }
            }
            if (seq.size() != cnt) return false;
            for (uint64_t t = 0; t < cnt; ++t) {
                const uint64_t m = ws <= kColexMax ? unrank(t, 0, wn, ws) : revdoor_unrank(t, wn, ws);
                int in = 0, out = 0;
                if (ws > kColexMax && t > 0) {
                    const uint64_t pv = revdoor_unrank(t - 1, wn, ws);
                    in = __builtin_ffsll(m & ~pv) - 1;
                    out = __builtin_ffsll(pv & ~m) - 1;
                }
                if (m != seq[t] || in != steps[t].first || out != steps[t].second) {
                    printf("walk table (%d, %d) differs at step %llu\n", wn, ws, (unsigned long long)t);
                    return false;
                }
            }
        }
    return true;
}

int main() {
    // the benchmark's plans (n = 24, k = 6; the candidate sets' kept and
    // dropped plans, among them the widened cap's 5 and 6 of 37 and 38) and
    // edge shapes
    const int cases[][2] = {{24, 6}, {38, 6}, {37, 5}, {28, 4}, {20, 8}, {22, 6}, {36, 4}, {16, 4}, {12, 5},
                            {30, 3}, {40, 4}, {64, 2}, {26, 13}, {10, 10}, {9, 1}, {1, 1}, {33, 16}};
    bool ok = tables_match();
    for (const auto &c : cases) ok = check(c[0], c[1], binom(c[0], c[1]) <= 3000000) && ok;
    puts(ok ? "plans OK" : "plans FAILED");
    return ok ? 0 : 1;
}
