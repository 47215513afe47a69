// Passes over the key or value rows of one attention row, for kernels that
// run one workgroup per row (or per group of rows) in float64: vector loads
// of whole key rows by groups of lanes with many rows' loads in flight, and
// workgroup reductions.
#pragma once

#include "fw_common.hpp"

namespace fw {

// Key rows are read by groups of lanes: a group of GL lanes covers one key,
// each lane VEC consecutive columns per load (whole rows per instruction).
template <typename T> struct RowVec;
template <> struct RowVec<uint16_t> {
    static constexpr int VEC = 8;
    __device__ static uint4 raw(const uint16_t *row, int c0) { return *(const uint4 *)(row + c0); }
    __device__ static void unpack(const uint4 &w, float (&x)[8]) {
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
    __device__ static uint4 raw(const float *row, int c0) { return *(const uint4 *)(row + c0); }
    __device__ static void unpack(const uint4 &w, float (&x)[4]) {
        x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
        x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
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
// numbers them within the lane (< VEC), the same for every key.  The GL lanes
// of a group share a key (j = -1 on lanes past the end, which still take part
// in the group's shuffles).  With VEC-wide loads (d a multiple of VEC) a
// group covers a row with one 16-byte chunk per lane (d <= 256 gives at most
// 64 chunks); otherwise a wave takes one key with up to four elements per
// lane.  Every lane keeps U keys' loads in flight (raw 16-byte words) before
// it uses the first: the passes over a row are bound by load latency.
template <typename T, typename F>
__device__ void for_keys(const T *M, int64_t N, int d, F &&f) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, NW = blockDim.x >> 6;
    constexpr int VEC = RowVec<T>::VEC;
    if (d % VEC == 0) {
        constexpr int U = 16;
        const int GL = group_lanes(d, VEC), KPW = 64 / GL;  // keys per wave step
        const int gi = lane % GL, gk = lane / GL;
        const bool has = gi < d / VEC;  // GL >= d / VEC: one chunk per lane at most
        const int64_t stride = (int64_t)NW * KPW;
        for (int64_t j0 = (int64_t)w * KPW; j0 < N; j0 += stride * U) {
            uint4 raw[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t j = j0 + u * stride + gk;
                raw[u] = (j < N && has) ? RowVec<T>::raw(M + j * d, gi * VEC) : make_uint4(0u, 0u, 0u, 0u);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t j = j0 + u * stride + gk;
                const bool ok = j < N;
                f(ok ? j : -1, gi, GL, [&](auto &&g) {
                    if (!ok || !has) return;
                    float x[VEC];
                    RowVec<T>::unpack(raw[u], x);
#pragma unroll
                    for (int i = 0; i < VEC; ++i) g(gi * VEC + i, i, x[i]);
                });
            }
        }
    } else {
        constexpr int U = 4;
        for (int64_t j0 = w; j0 < N; j0 += (int64_t)NW * U) {
            float x[U][4];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t j = j0 + (int64_t)u * NW;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int c = lane + 64 * t;
                    x[u][t] = (j < N && c < d) ? Elem<T>::load(M + j * d, c) : 0.f;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t j = j0 + (int64_t)u * NW;
                if (j >= N) break;  // uniform across the wave
                f(j, lane, 64, [&](auto &&g) {
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        if (lane + 64 * t < d) g(lane + 64 * t, t, x[u][t]);
                });
            }
        }
    }
}

// For every key j of M [N][d]: h(j, s_j) on one lane, with s_j the key's
// elements folded by acc = term(c, slot, x, acc) from 0 on each lane and
// summed over the lanes.  Rows of 16 lanes per key (d = 128 in bf16, say)
// sum the 16 keys a lane has in flight by a transposed reduction: at each
// of four exchanges a lane gives away half of its partial sums and adds
// the partner's half of its own, so after 15 shuffles (not 64) lane i of
// the group holds the whole sum of the group's i-th key.  Other widths
// reduce every key over its group.
template <typename T, typename Term, typename H>
__device__ void for_key_sums(const T *M, int64_t N, int d, Term &&term, H &&h) {
    constexpr int VEC = RowVec<T>::VEC, U = 16;
    if (d % VEC == 0 && group_lanes(d, VEC) == U) {
        const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, NW = blockDim.x >> 6;
        constexpr int KPW = 64 / U;
        const int gi = lane % U, gk = lane / U;
        const bool has = gi < d / VEC;
        const int64_t stride = (int64_t)NW * KPW;
        for (int64_t j0 = (int64_t)w * KPW; j0 < N; j0 += stride * U) {
            uint4 raw[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t j = j0 + u * stride + gk;
                raw[u] = (j < N && has) ? RowVec<T>::raw(M + j * d, gi * VEC) : make_uint4(0u, 0u, 0u, 0u);
            }
            double acc[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float x[VEC];
                RowVec<T>::unpack(raw[u], x);
                double a = 0.0;
#pragma unroll
                for (int i = 0; i < VEC; ++i) a = term(gi * VEC + i, i, x[i], a);
                acc[u] = has ? a : 0.0;
            }
#pragma unroll
            for (int half = U / 2; half > 0; half >>= 1) {
                const bool upper = (gi & half) != 0;
#pragma unroll
                for (int i = 0; i < half; ++i) {
                    const double give = upper ? acc[i] : acc[i + half];
                    const double keep = upper ? acc[i + half] : acc[i];
                    acc[i] = keep + __shfl_xor(give, half);
                }
            }
            const int64_t j = j0 + (int64_t)gi * stride + gk;
            if (j < N) h(j, acc[0]);
        }
    } else {
        for_keys(M, N, d, [&](int64_t j, int gi, int GL, auto &&walk) {
            double a = 0.0;
            walk([&](int c, int slot, float x) { a = term(c, slot, x, a); });
            a = group_sum(a, GL);
            if (j >= 0 && gi == 0) h(j, a);
        });
    }
}

// The columns for_keys hands this lane, by slot: fn(c, slot) once per column.
template <typename T, typename F>
__device__ void lane_columns(int d, F &&fn) {
    const int lane = threadIdx.x & 63;
    constexpr int VEC = RowVec<T>::VEC;
    if (d % VEC == 0) {
        const int gi = lane % group_lanes(d, VEC);
        if (gi < d / VEC) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) fn(gi * VEC + i, i);
        }
    } else {
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (lane + 64 * t < d) fn(lane + 64 * t, t);
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

// Sum over the 64 lanes of a wave, on every lane.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// Lane l's v (l wave-uniform), on every lane.
__device__ __forceinline__ double lane_value(double v, int l) {
    const uint64_t b = __double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Position of the k-th (from 0) set bit of m; m holds more than k bits.
__device__ __forceinline__ int nth_bit(uint64_t m, int k) {
    for (; k > 0; --k) m &= m - 1;
    return __ffsll((unsigned long long)m) - 1;
}

// Keys per thread that wave_top holds in registers.
constexpr int kTopRegs = 16;

// (a, ia) ahead of (b, ib) in the order (value desc, index asc); index -1
// marks no key, behind every key.
__device__ __forceinline__ bool top_ahead(double a, int ia, double b, int ib) {
    return ia >= 0 && (ib < 0 || a > b || (a == b && ia < ib));
}

// wave_top's per-wave picks for rows too long for registers: every pick
// rescans the thread's keys in LDS for the best one after the last pick.
__device__ inline void wave_top_scan(const double *vals, int64_t N, int M, double *cv, int64_t *ci,
                                     const unsigned char *skip, int smin) {
    const int tid = threadIdx.x, NT = blockDim.x, lane = tid & 63, w = tid >> 6;
    double pv = INFINITY;
    int64_t pi = -1;
    for (int t = 0; t < M; ++t) {
        double bv = 0.0;
        int64_t bi = -1;
        for (int64_t j = tid; j < N; j += NT) {
            if (skip && skip[j] < smin) continue;
            const double x = vals[j];
            const bool after = x < pv || (x == pv && j > pi);
            if (after && (bi < 0 || x > bv || (x == bv && j < bi))) { bv = x; bi = j; }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const double ov = __shfl_xor(bv, off);
            const int64_t oi = __shfl_xor(bi, off);
            if (oi >= 0 && (bi < 0 || ov > bv || (ov == bv && oi < bi))) { bv = ov; bi = oi; }
        }
        if (lane == 0) {
            cv[w * M + t] = bv;
            ci[w * M + t] = bi;
        }
        if (bi >= 0) {  // none left: the later rounds find none either
            pv = bv;
            pi = bi;
        }
    }
}

// The M (<= 64) largest values of vals[0, N) in the order (value desc,
// index asc), keys with skip[j] < smin left out (no skip: all keys), their
// indices into out[0, M).  Each wave takes the next best of its own keys M
// times (shuffles only, no workgroup barrier), then the waves' lists are
// merged by counting ranks.  cv, ci: LDS scratch of (blockDim.x / 64) M
// entries.
//
// Rows of up to kTopRegs keys per thread: each thread sorts its keys in
// registers once (a bitonic network), so a pick is one wave reduction of
// the threads' heads and a shift in the thread that held the winner.
// Longer rows rescan the thread's keys in LDS for every pick.
__device__ inline void wave_top(const double *vals, int64_t N, int M, int *out, double *cv, int64_t *ci,
                                const unsigned char *skip = nullptr, int smin = 0) {
    const int tid = threadIdx.x, NT = blockDim.x, lane = tid & 63, w = tid >> 6, nw = NT >> 6;
    if (N <= (int64_t)kTopRegs * NT) {
        double v[kTopRegs];
        int id[kTopRegs];
#pragma unroll
        for (int i = 0; i < kTopRegs; ++i) {
            const int j = tid + NT * i;
            v[i] = 0.0;
            id[i] = -1;
            if (j < N && !(skip && skip[j] < smin)) {
                v[i] = vals[j];
                id[i] = j;
            }
        }
#pragma unroll
        for (int k = 2; k <= kTopRegs; k <<= 1) {
#pragma unroll
            for (int jj = k >> 1; jj > 0; jj >>= 1) {
#pragma unroll
                for (int i = 0; i < kTopRegs; ++i) {
                    const int l = i ^ jj;
                    if (l > i) {
                        // blocks with (i & k) == 0 put the better key first
                        const bool sw = (i & k) == 0 ? top_ahead(v[l], id[l], v[i], id[i])
                                                     : top_ahead(v[i], id[i], v[l], id[l]);
                        const double tv = v[i];
                        const int ti = id[i];
                        v[i] = sw ? v[l] : tv;
                        id[i] = sw ? id[l] : ti;
                        v[l] = sw ? tv : v[l];
                        id[l] = sw ? ti : id[l];
                    }
                }
            }
        }
        for (int t = 0; t < M; ++t) {
            double bv = v[0];
            int bi = id[0];
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                const double ov = __shfl_xor(bv, off);
                const int oi = __shfl_xor(bi, off);
                if (top_ahead(ov, oi, bv, bi)) {
                    bv = ov;
                    bi = oi;
                }
            }
            if (lane == 0) {
                cv[w * M + t] = bv;
                ci[w * M + t] = bi;
            }
            if (bi >= 0 && id[0] == bi) {  // keys are distinct: one thread
#pragma unroll
                for (int i = 0; i + 1 < kTopRegs; ++i) {
                    v[i] = v[i + 1];
                    id[i] = id[i + 1];
                }
                id[kTopRegs - 1] = -1;
            }
        }
    } else {
        wave_top_scan(vals, N, M, cv, ci, skip, smin);
    }
    __syncthreads();
    for (int c = tid; c < nw * M; c += NT) {
        const int64_t i = ci[c];
        if (i < 0) continue;
        const double v = cv[c];
        int rank = 0;
        for (int e = 0; e < nw * M; ++e) {
            const int64_t oi = ci[e];
            rank += oi >= 0 && (cv[e] > v || (cv[e] == v && oi < i));
        }
        if (rank < M) out[rank] = (int)i;
    }
    __syncthreads();
}

}  // namespace fw
