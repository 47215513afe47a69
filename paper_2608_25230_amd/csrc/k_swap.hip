// Swap rule: the balancing selector of Section 2.1.  Start at the top-k set
// and repeatedly apply the single (kept i, dropped j) swap that most
// decreases es, accepting only a strict decrease, for at most max_iters swaps.
//
// With g = sum_{a in S} u_a, u_a = p_a (v_a - mu), P = p(S) (Lemma 2.2):
//   es(S - i + j)^2 = ||g - u_i + u_j||^2 / (P - p_i + p_j)^2
//   ||g - u_i + u_j||^2 = ||g||^2 + ||u_i||^2 + ||u_j||^2 - 2 g.u_i + 2 g.u_j
//                         - 2 u_i.u_j,
// so one sweep over all pairs needs the cross terms u_i.u_j.
//
// Rows of at most 64 keys run entirely in float64 on the residual Gram
// matrix, one workgroup per row.  Longer rows keep per-row state in the
// workspace; each iteration computes g.u_x for every key, evaluates every
// pair (cross terms from v_i.v_j: u_i.u_j = p_i p_j (v_i.v_j - v_i.mu -
// v_j.mu + |mu|^2)) in float32 with a per-row argmin (ties to the smaller
// (i, j)), then applies the winning swap and updates g in float64.  Gaps in
// the trajectory are ||g|| / P from float64 sums.
//
// Pruned pair search (long rows).  By Cauchy-Schwarz, |u_i.u_j| <= r_i r_j
// with r_x = ||u_x||, so every pair's numerator is at least
//     A_i + B_j - 2 r_i r_j,   A_i = ||g - u_i||^2,  B_j = ||u_j||^2 + 2 g.u_j,
// and its denominator is (P - p_i + p_j)^2.  An upper
// bound UB on the best value (the best of the 8 x 8 pairs of smallest A_i and
// B_j, evaluated exactly) leaves only the pairs whose lower bound reaches UB:
// two fused multiply-adds and a compare per pair, no cross terms.  Those few
// are evaluated exactly in float64 (||g - u_i + u_j||^2 / (P - p_i + p_j)^2,
// ties to the smaller i n + j).  A row whose survivors overflow the list
// falls back to the full sweep.
#include "fw_internal.hpp"
#include "instance64.hpp"
#include "rowpass.hpp"

namespace fw {

// ===========================================================================
// rows with n <= 64: one workgroup per row, float64
// ===========================================================================
template <typename T>
__global__ void __launch_bounds__(256)
swap_small_kernel(const T *__restrict__ q, const T *__restrict__ k, const T *__restrict__ v,
                  const float *__restrict__ scale, const float *__restrict__ bias, int64_t G,
                  int n, int d, int kk, int max_iters, int32_t *s_idx, float *gap_traj,
                  int32_t *n_swaps, float *dropped) {
    extern __shared__ __align__(16) unsigned char smem[];
    double *Gm = (double *)smem;            // n*n
    double *ps = Gm + n * n;                // n
    double *zs = ps + n;                    // n
    double *mu = zs + n;                    // d
    double *R = mu + d;                     // n
    double *redd = R + n;                   // NT
    uint64_t *redm = (uint64_t *)(redd + blockDim.x);  // NT
    int *lists = (int *)(redm + blockDim.x);           // n
    float *Vs = (float *)(lists + n + (n & 1));        // n*(d+1)
    const int tid = threadIdx.x, NT = blockDim.x;
    const int64_t r = blockIdx.x, h = r / G;
    const T *qr = q + r * d;
    const T *kh = k + h * (int64_t)n * d;
    const T *vh = v + h * (int64_t)n * d;
    instance64(qr, kh, vh, scale ? scale[h] : default_scale(d), bias, n, d, Vs, zs, ps, mu, Gm, n);
    uint64_t S = topk_mask64(zs, n, kk, nullptr);
    const int T_len = max_iters + 1;
    float *traj = gap_traj + r * T_len;
    double es = exact_gap(S, n, vh, ps, mu, d, redd);
    if (tid == 0) traj[0] = (float)es;
    int it = 0;
    const int nout = n - kk;
    while (it < max_iters && nout > 0) {
        // R_x = g . u_x = sum_{a in S} Gm_xa; current value ||g||^2 / P^2
        for (int x = tid; x < n; x += NT) {
            double s = 0.0;
            for (uint64_t a = S; a; a &= a - 1) s += Gm[x * n + (__ffsll((unsigned long long)a) - 1)];
            R[x] = s;
        }
        if (tid == 0) {
            int a = 0, b = kk;
            for (int x = 0; x < n; ++x) lists[((S >> x) & 1ull) ? a++ : b++] = x;
        }
        __syncthreads();
        double Sv = 0.0;
        for (uint64_t a = S; a; a &= a - 1) Sv += R[__ffsll((unsigned long long)a) - 1];
        const double P = mass64(S, ps);
        const double cur = Sv / (P * P);
        double bv = INFINITY;
        int bp = 0x7FFFFFFF;
        for (int pi = tid; pi < kk * nout; pi += NT) {
            const int i = lists[pi / nout], j = lists[kk + pi % nout];
            const double num = Sv + Gm[i * n + i] + Gm[j * n + j] - 2.0 * R[i] + 2.0 * R[j] - 2.0 * Gm[i * n + j];
            const double den = P - ps[i] + ps[j];
            const double val = num / (den * den);
            if (val < bv) { bv = val; bp = pi; }
        }
        redd[tid] = bv;
        redm[tid] = (uint64_t)(uint32_t)bp;
        __syncthreads();
        if (tid == 0) {
            for (int t = 1; t < NT; ++t)
                if (redd[t] < redd[0] || (redd[t] == redd[0] && redm[t] < redm[0])) {
                    redd[0] = redd[t];
                    redm[0] = redm[t];
                }
        }
        __syncthreads();
        const double best = redd[0];
        const int pi = (int)redm[0];
        __syncthreads();
        if (!(best < cur)) break;
        S ^= (1ull << lists[pi / nout]) ^ (1ull << lists[kk + pi % nout]);
        ++it;
        es = exact_gap(S, n, vh, ps, mu, d, redd);
        if (tid == 0) traj[it] = (float)es;
    }
    if (tid == 0) {
        for (int t = it + 1; t < T_len; ++t) traj[t] = __int_as_float(0x7fc00000);
        n_swaps[r] = it;
        int i = 0;
        double dm = 0.0;
        for (int x = 0; x < n; ++x) {
            if ((S >> x) & 1ull) s_idx[r * kk + i++] = x;
            else dm += ps[x];
        }
        if (dropped) dropped[r] = (float)dm;
    }
}

// ===========================================================================
// rows with n > 64: workspace state, float32 pair search
// ===========================================================================
struct SwapState {
    const float *z, *row_m, *row_l;
    const uint32_t *thr_key;
    const int32_t *thr_cut;
    float *p;        // [R][n]
    uint8_t *inS;    // [R][n]
    int32_t *Sl;     // [R][k]
    float *w;        // [R][n]   v_j . mu
    float *bq;       // [R][n]   ||u_j||^2
    float *a;        // [R][n]   g . u_j
    double *mu;      // [R][d]
    double *g;       // [R][d]
    double *sc;      // [R][4]   P, ||g||^2, |mu|^2, cur
    int32_t *st;     // [R][2]   active, swaps
    float *pv;       // [R][nblk] partial best values
    int64_t *pp;     // [R][nblk] partial best pair index i*n + j
    float4 *jd;      // [R][n]   per key: (B_j or +inf if kept, p_j, 2 w_j, P + p_j)
    float2 *br;      // [R][n]   per key: (B_j or +inf if kept, ||u_j||) for the pruned search
    double *ub;      // [R][2]   upper bound on the best pair value (and a spare slot)
    int64_t *ubp;    // [R]      the pair that gave the upper bound
    int32_t *cnt;    // [R]      surviving pairs
    int32_t *fb;     // [R]      1: survivors overflowed, the full sweep runs
    int32_t *fbl;    // [R]      the rows whose survivors overflowed, in any order
    int32_t *fbn;    // [1]      their count (cleared by the init and apply passes)
    int64_t *cand;   // [R][kSwapCand] surviving pairs i n + j
    int32_t *ord;    // [R][k]    kept keys in the bound pass's order (k <= kSwapSort)
    float4 *kd;      // [R][k]    per kept key in that order: its bound-test terms and index
    int a_all;       // a is written for every key (else for the kept keys only: the
                     // MFMA sweep of the pruned search reads B_j from br instead)
    int nblk;
};

constexpr int kSwapCand = 8192;  // surviving pairs kept per row (8192 and 16384 measured alike, 4096 11 % slower)
constexpr int kSwapSweepRows = 64;  // rows a fallback sweep takes at a time
constexpr int kSwapSL = 16;      // keys per slice of the bound pass's whole-slice test (<= 32)
constexpr int kSwapSort = 2048;  // kept keys ordered for the bound pass

// Elements [c0, c0 + 8) of a row of d (those below d), as floats: one
// 16-byte load for bf16 rows with d a multiple of 8, else one load each.
template <typename T>
__device__ __forceinline__ void load8(const T *row, int c0, int d, float (&x)[8]) {
    if (sizeof(T) == 2 && d % 8 == 0) {
        RowVec<uint16_t>::unpack(RowVec<uint16_t>::raw((const uint16_t *)row, c0), x);
        return;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = c0 + e < d ? Elem<T>::load(row, c0 + e) : 0.f;
}

template <typename T>
__global__ void __launch_bounds__(256)
swap_init_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, int kk, SwapState s,
                 float *gap_traj, int T_len) {
    __shared__ double redd[256];
    __shared__ int scan[256];
    const int tid = threadIdx.x, NT = blockDim.x;
    const int64_t r = blockIdx.x, h = r / G;
    if (s.fbn && r == 0 && tid == 0) *s.fbn = 0;
    const T *vh = v + h * n * d;
    const float m = s.row_m[r], inv_l = 1.0f / s.row_l[r];
    const uint32_t key = s.thr_key[r];
    const int64_t cut = s.thr_cut[r];
    float *p = s.p + r * n;
    uint8_t *inS = s.inS + r * n;
    const float *zr = s.z + r * n;
    // weights and membership (coalesced), then the kept list in ascending
    // order from per-thread chunks of the membership bytes
    for (int64_t j = tid; j < n; j += NT) {
        const float zz = zr[j];
        p[j] = expf(zz - m) * inv_l;
        const uint32_t u = ord_key(zz);
        inS[j] = (uint8_t)((u > key) || (u == key && j <= cut));
    }
    __syncthreads();
    const int64_t chunk = (n + NT - 1) / NT;
    const int64_t lo = tid * chunk, hi = (lo + chunk < n) ? lo + chunk : n;
    int c = 0;
    for (int64_t j = lo; j < hi; ++j) c += inS[j];
    int total;
    int pos = block_exclusive_scan(c, scan, &total);
    for (int64_t j = lo; j < hi; ++j)
        if (inS[j]) s.Sl[r * kk + pos++] = (int32_t)j;
    __syncthreads();
    // mu = sum_j p_j v_j, float64: 16 key lanes x 16 column groups (a
    // column group per thread and pass), the key lanes' sums added in order
    double *mu = s.mu + r * d;
    {
        const int jl = tid & 15, cg = tid >> 4;
        for (int c0 = 8 * cg; c0 < d; c0 += 128) {
            double acc[8];
#pragma unroll
            for (int x = 0; x < 8; ++x) acc[x] = 0.0;
            for (int64_t j = jl; j < n; j += 16) {
                const double pj = (double)p[j];
                float xv[8];
                load8(vh + j * d, c0, d, xv);
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    if (c0 + x < d) acc[x] = fma(pj, (double)xv[x], acc[x]);
            }
#pragma unroll
            for (int x = 0; x < 8; ++x) {
#pragma unroll
                for (int off = 1; off < 16; off <<= 1) acc[x] += __shfl_xor(acc[x], off);
            }
            if (jl == 0) {
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    if (c0 + x < d) mu[c0 + x] = acc[x];
            }
        }
    }
    __syncthreads();
    double mu2 = 0.0;
    for (int cc = 0; cc < d; ++cc) mu2 += mu[cc] * mu[cc];
    // w_j = v_j . mu and ||u_j||^2 = p_j^2 ||v_j - mu||^2: 16 lanes per key,
    // partial sums by a butterfly.  bf16 rows with d a multiple of 8: lane l
    // takes the 8-column chunks l, l + 16, .. (a 16-byte load each); other
    // rows: columns lane, lane + 16, ...
    {
        const int jl = tid >> 4, cl = tid & 15;
        const bool chunks = sizeof(T) == 2 && d % 8 == 0;
        for (int64_t j0 = 0; j0 < n; j0 += NT / 16) {
            const int64_t j = j0 + jl;
            double dw = 0.0, du = 0.0;
            if (j < n && chunks) {
                for (int c0 = 8 * cl; c0 < d; c0 += 128) {
                    float xv[8];
                    load8(vh + j * d, c0, d, xv);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const double x = (double)xv[e], m = mu[c0 + e];
                        dw = fma(x, m, dw);
                        du = fma(x - m, x - m, du);
                    }
                }
            } else if (j < n) {
                for (int cc = cl; cc < d; cc += 16) {
                    const double x = (double)Elem<T>::load(vh, j * d + cc), m = mu[cc];
                    dw = fma(x, m, dw);
                    du = fma(x - m, x - m, du);
                }
            }
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                dw += __shfl_xor(dw, off);
                du += __shfl_xor(du, off);
            }
            if (j < n && cl == 0) {
                s.w[r * n + j] = (float)dw;
                s.bq[r * n + j] = (float)((double)p[j] * (double)p[j] * du);
            }
        }
    }
    // g = sum_{a in S} u_a, P = p(S): 16 kept-key lanes x 16 column groups,
    // the key lanes' sums added by a butterfly
    double *g = s.g + r * d;
    {
        const int kl = tid & 15, cg = tid >> 4;
        for (int c0 = 8 * cg; c0 < d; c0 += 128) {
            double acc[8];
#pragma unroll
            for (int x = 0; x < 8; ++x) acc[x] = 0.0;
            for (int i = kl; i < kk; i += 16) {
                const int64_t a = s.Sl[r * kk + i];
                const double pa = (double)p[a];
                float xv[8];
                load8(vh + a * d, c0, d, xv);
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    if (c0 + x < d) acc[x] = fma(pa, (double)xv[x] - mu[c0 + x], acc[x]);
            }
#pragma unroll
            for (int x = 0; x < 8; ++x) {
#pragma unroll
                for (int off = 1; off < 16; off <<= 1) acc[x] += __shfl_xor(acc[x], off);
            }
            if (kl == 0) {
#pragma unroll
                for (int x = 0; x < 8; ++x)
                    if (c0 + x < d) g[c0 + x] = acc[x];
            }
        }
    }
    __syncthreads();
    double P = 0.0;
    for (int i = tid; i < kk; i += NT) P += (double)p[s.Sl[r * kk + i]];
    P = block_reduce(P, redd, OpSum());
    double g2 = 0.0;
    for (int cc = tid; cc < d; cc += NT) g2 += g[cc] * g[cc];
    g2 = block_reduce(g2, redd, OpSum());
    if (tid == 0) {
        double *sc = s.sc + r * 4;
        sc[0] = P;
        sc[1] = g2;
        sc[2] = mu2;
        sc[3] = g2 / (P * P);
        s.st[r * 2 + 0] = (kk < n) ? 1 : 0;
        s.st[r * 2 + 1] = 0;
        gap_traj[r * T_len] = (float)(sqrt(g2) / P);
    }
}

// a_j = g . u_j = p_j (v_j . g - mu . g)
template <typename T>
__global__ void __launch_bounds__(256)
swap_dots_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, SwapState s) {
    __shared__ float gs[256];
    __shared__ double redd[256];
    const int64_t r = blockIdx.y;
    if (!s.st[r * 2]) return;
    const int tid = threadIdx.x;
    const int64_t h = r / G;
    const T *vh = v + h * n * d;
    const double *g = s.g + r * d, *mu = s.mu + r * d;
    double mg = 0.0;
    for (int c = tid; c < d; c += blockDim.x) {
        gs[c] = (float)g[c];
        mg += mu[c] * g[c];
    }
    mg = block_reduce(mg, redd, OpSum());
    const float P = (float)s.sc[r * 4 + 0];
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + tid; j < n; j += (int64_t)gridDim.x * blockDim.x) {
        float acc = 0.f;
        for (int c = 0; c < d; ++c) acc = fmaf(Elem<T>::load(vh, j * d + c), gs[c], acc);
        const float pj = s.p[r * n + j];
        const float aj = pj * (float)((double)acc - mg);
        const bool kept = s.inS[r * n + j];
        if (kept || s.a_all) s.a[r * n + j] = aj;
        const float bj = kept ? INFINITY : s.bq[r * n + j] + 2.f * aj;
        if (s.jd && !s.br) s.jd[r * n + j] = make_float4(bj, pj, 2.f * s.w[r * n + j], P + pj);
        if (s.br) s.br[r * n + j] = make_float2(bj, sqrtf(s.bq[r * n + j]));
    }
}

// The same dots for RB rows of one key/value unit at once (G % RB == 0,
// d <= 256): each key's values are read once for the RB rows, whose g
// vectors sit in LDS.  Per row the same float32 sum in column order.  Rows
// of whole 16-byte chunks are read a chunk per load (8 bf16 or 4 float
// values), and g by vector LDS reads of the same columns.
template <typename T, int RB>
__global__ void __launch_bounds__(256)
swap_dots_group_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, SwapState s) {
    __shared__ float gs[RB][256];
    __shared__ double mgs[RB];
    __shared__ float Ps[RB];
    const int tid = threadIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * RB;
    const int64_t h = r0 / G;
    const T *vh = v + h * n * d;
    for (int e = tid; e < RB * d; e += blockDim.x) {
        const int rr = e / d, c = e - rr * d;
        gs[rr][c] = (float)s.g[(r0 + rr) * d + c];
    }
    // mu . g per row: 16 lanes per row, their partial sums added by a butterfly
    for (int rr0 = 0; rr0 < RB; rr0 += 16) {
        const int rr = rr0 + (tid >> 4), ln = tid & 15;
        double mg = 0.0;
        if (rr < RB)
            for (int c = ln; c < d; c += 16) mg += s.mu[(r0 + rr) * d + c] * s.g[(r0 + rr) * d + c];
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) mg += __shfl_xor(mg, off);
        if (rr < RB && ln == 0) {
            mgs[rr] = mg;
            Ps[rr] = (float)s.sc[(r0 + rr) * 4 + 0];
        }
    }
    __syncthreads();
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + tid; j < n; j += (int64_t)gridDim.x * blockDim.x) {
        float acc[RB];
#pragma unroll
        for (int rr = 0; rr < RB; ++rr) acc[rr] = 0.f;
        constexpr int VEC = RowVec<T>::VEC;
        if (d % VEC == 0) {
            const T *row = vh + j * d;
            for (int c0 = 0; c0 < d; c0 += VEC) {
                float x[VEC];
                RowVec<T>::unpack(RowVec<T>::raw(row, c0), x);
#pragma unroll
                for (int rr = 0; rr < RB; ++rr)
#pragma unroll
                    for (int i = 0; i < VEC; ++i) acc[rr] = fmaf(x[i], gs[rr][c0 + i], acc[rr]);
            }
        } else {
            for (int c = 0; c < d; ++c) {
                const float x = Elem<T>::load(vh, j * d + c);
#pragma unroll
                for (int rr = 0; rr < RB; ++rr) acc[rr] = fmaf(x, gs[rr][c], acc[rr]);
            }
        }
#pragma unroll
        for (int rr = 0; rr < RB; ++rr) {
            const int64_t r = r0 + rr;
            if (!s.st[r * 2]) continue;
            const float pj = s.p[r * n + j];
            const float aj = pj * (float)((double)acc[rr] - mgs[rr]);
            const bool kept = s.inS[r * n + j];
            if (kept || s.a_all) s.a[r * n + j] = aj;
            const float bj = kept ? INFINITY : s.bq[r * n + j] + 2.f * aj;
            if (s.jd && !s.br) s.jd[r * n + j] = make_float4(bj, pj, 2.f * s.w[r * n + j], Ps[rr] + pj);
            if (s.br) s.br[r * n + j] = make_float2(bj, sqrtf(s.bq[r * n + j]));
        }
    }
}

// The rows a sweep workgroup takes: blockIdx.y over every active row, or,
// under the pruned search, the listed rows whose survivors overflowed,
// gridDim.y of them at a time (so that a sweep with no such row costs a
// small grid, not one workgroup per tile of every row).
template <typename F>
__device__ __forceinline__ void sweep_rows(const SwapState &s, F &&body) {
    if (!s.fbl) {
        const int64_t r = blockIdx.y;
        if (s.st[r * 2]) body(r);
        return;
    }
    const int nfb = *s.fbn;
    for (int yy = blockIdx.y; yy < nfb; yy += gridDim.y) {
        const int64_t r = s.fbl[yy];
        if (s.st[r * 2]) body(r);
        __syncthreads();  // LDS is reused by the next row
    }
}

// The per-key records of the full sweep, (B_j or +inf if kept, p_j, 2 w_j,
// P + p_j), for the rows the fallback sweep takes: under the pruned search
// the dots pass does not write them for every row (they are the same values
// it would have written).
__global__ void __launch_bounds__(256) swap_jd_kernel(int64_t n, SwapState s) {
    sweep_rows(s, [&](int64_t r) {
        const float P = (float)s.sc[r * 4 + 0];
        for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256) {
            const float pj = s.p[r * n + j];
            s.jd[r * n + j] = make_float4(s.br[r * n + j].x, pj, 2.f * s.w[r * n + j], P + pj);
        }
    });
}

// every (kept i, dropped j) pair of a tile: 32 kept x 128 keys per workgroup
template <typename T>
__device__ __forceinline__ void pairs_row(const T *__restrict__ v, int64_t G, int64_t n, int d, int kk,
                                          const SwapState &s, int64_t r) {
    constexpr int TI = 32, TJ = 128, TD = 32;
    __shared__ float Vi[TI][TD + 1];
    __shared__ float Vj[TJ][TD + 1];
    __shared__ int idx_i[TI];
    __shared__ float redv[256];
    __shared__ int64_t redp[256];
    const int tid = threadIdx.x;
    const int64_t h = r / G;
    const T *vh = v + h * n * d;
    const int itiles = (kk + TI - 1) / TI;
    const int it = blockIdx.x % itiles;
    const int64_t jt = blockIdx.x / itiles;
    const int i0 = it * TI;
    const int64_t j0 = jt * TJ;
    if (tid < TI) idx_i[tid] = (i0 + tid < kk) ? s.Sl[r * kk + i0 + tid] : -1;
    __syncthreads();
    const int ty = tid / 32, tx = tid % 32;  // rows ty*4.., keys tx + 32*c
    float acc[4][4] = {};
    for (int c0 = 0; c0 < d; c0 += TD) {
        for (int e = tid; e < TI * TD; e += 256) {
            const int rr = e / TD, cc = e % TD;
            const int a = idx_i[rr];
            Vi[rr][cc] = (a >= 0 && c0 + cc < d) ? Elem<T>::load(vh, (int64_t)a * d + c0 + cc) : 0.f;
        }
        for (int e = tid; e < TJ * TD; e += 256) {
            const int rr = e / TD, cc = e % TD;
            const int64_t j = j0 + rr;
            Vj[rr][cc] = (j < n && c0 + cc < d) ? Elem<T>::load(vh, j * d + c0 + cc) : 0.f;
        }
        __syncthreads();
#pragma unroll 8
        for (int cc = 0; cc < TD; ++cc) {
            float ai[4], bj[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) ai[u] = Vi[ty * 4 + u][cc];
#pragma unroll
            for (int u = 0; u < 4; ++u) bj[u] = Vj[tx + 32 * u][cc];
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w) acc[u][w] = fmaf(ai[u], bj[w], acc[u][w]);
        }
        __syncthreads();
    }
    const double *sc = s.sc + r * 4;
    const float P = (float)sc[0], g2 = (float)sc[1], mu2 = (float)sc[2];
    const float *p = s.p + r * n, *w = s.w + r * n, *bq = s.bq + r * n, *a = s.a + r * n;
    const uint8_t *inS = s.inS + r * n;
    float bv = INFINITY;
    int64_t bp = INT64_MAX;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = idx_i[ty * 4 + u];
        if (i < 0) continue;
        const float pi = p[i], wi = w[i], Ai = g2 + bq[i] - 2.f * a[i];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const int64_t j = j0 + tx + 32 * x;
            if (j >= n || inS[j]) continue;
            const float pj = p[j];
            const float cij = pi * pj * (acc[u][x] - wi - w[j] + mu2);
            const float num = Ai + bq[j] + 2.f * a[j] - 2.f * cij;
            const float den = P - pi + pj;
            const float val = num / (den * den);
            const int64_t pidx = (int64_t)i * n + j;
            if (val < bv || (val == bv && pidx < bp)) { bv = val; bp = pidx; }
        }
    }
    redv[tid] = bv;
    redp[tid] = bp;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if (tid < st) {
            const float v2 = redv[tid + st];
            const int64_t p2 = redp[tid + st];
            if (v2 < redv[tid] || (v2 == redv[tid] && p2 < redp[tid])) { redv[tid] = v2; redp[tid] = p2; }
        }
        __syncthreads();
    }
    if (tid == 0) {
        s.pv[r * s.nblk + blockIdx.x] = redv[0];
        s.pp[r * s.nblk + blockIdx.x] = redp[0];
    }
}

template <typename T>
__global__ void __launch_bounds__(256)
swap_pairs_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, int kk, SwapState s) {
    sweep_rows(s, [&](int64_t r) { pairs_row<T>(v, G, n, d, kk, s, r); });
}

// ---------------------------------------------------------------------------
// every (kept i, key j) pair on MFMA: bf16 rows, d = 128, n a multiple of 16.
// A workgroup (8 waves) takes 512 consecutive kept keys of one row -- each
// wave 64 of them as the MFMA's A operand in registers -- and a chunk of
// SPJ keys, streamed as 16-key tiles through a double-buffered LDS stage
// shared by the waves (whole key rows per load, 16-byte chunk c of row r at
// position c ^ r).  The cross term v_i . v_j is the MFMA output; the
// epilogue keeps, per (lane, kept key), the smallest pair value and the tile
// where it was first reached, so ties resolve to the smaller (i, j).
//   num = (A_i + B_j) + p_i p_j (2 w_i - 2|mu|^2 + 2 w_j - 2 v_i.v_j)
//   A_i = ||g||^2 + ||u_i||^2 - 2 g.u_i,  B_j = ||u_j||^2 + 2 g.u_j
//   den = P - p_i + p_j,  value = num / den^2
// ---------------------------------------------------------------------------
namespace {
typedef __bf16 sbf16x8 __attribute__((ext_vector_type(8)));
typedef float sf32x4 __attribute__((ext_vector_type(4)));
constexpr int SPI = 512;        // kept keys per workgroup
constexpr int SPJ = 2048;       // keys per workgroup
constexpr int SPT = 8;          // tiles per stage
constexpr int SPD = 128;        // head dimension
constexpr int SP_STAGE = SPT * 16 * SPD * 2;  // bytes of V per stage
#define SP_LDS(ptr) ((__attribute__((address_space(3))) void *)(ptr))
#define SP_VM(k) case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
__device__ __forceinline__ void sp_wait_vm(int n) {
    switch (n) {
        SP_VM(0) SP_VM(1) SP_VM(4) SP_VM(5)
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}
#undef SP_VM
}  // namespace

__device__ __forceinline__ void pairs_mfma_row(const uint16_t *__restrict__ v, int64_t G, int64_t n, int kk,
                                               const SwapState &s, int64_t r) {
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *vbuf = smem;                                   // [2][SP_STAGE]
    float4 *jbuf = (float4 *)(smem + 2 * SP_STAGE);               // [2][SPT * 16]
    float *redv = (float *)(smem + 2 * SP_STAGE + 2 * SPT * 16 * 16);  // [8]
    int64_t *redp = (int64_t *)(redv + 8);                        // [8]
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, rl = lane & 15, grp = lane >> 4;
    const int64_t nchunk = (n + SPJ - 1) / SPJ;
    const int ib = (int)(blockIdx.x / nchunk);
    const int64_t jc = blockIdx.x % nchunk;
    const int64_t h = r / G;
    const uint16_t *vh = v + h * n * SPD;
    const int32_t *Sl = s.Sl + r * kk;
    const float4 *jd = s.jd + r * n;
    const int ibase = ib * SPI + w * 64;  // this wave's first kept-list position
    // A operand: kept keys ibase + 16 it + rl, columns 32 s + 8 grp
    sbf16x8 qa[4][4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int ip = ibase + 16 * it + rl;
        const int a = ip < kk ? Sl[ip] : 0;
#pragma unroll
        for (int st = 0; st < 4; ++st) qa[it][st] = *(const sbf16x8 *)(vh + (int64_t)a * SPD + 32 * st + 8 * grp);
    }
    // per kept-key slot (it, e): list position ibase + 16 it + 4 grp + e
    const double *sc = s.sc + r * 4;
    const float g2 = (float)sc[1], mu2 = (float)sc[2];
    float Ai[4][4], pi[4][4], Xi[4][4];
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int ip = ibase + 16 * it + 4 * grp + e;
            const int a = ip < kk ? Sl[ip] : 0;
            const float pa = s.p[r * n + a];
            Ai[it][e] = ip < kk ? g2 + s.bq[r * n + a] - 2.f * s.a[r * n + a] : INFINITY;
            pi[it][e] = pa;
            Xi[it][e] = 2.f * s.w[r * n + a] - 2.f * mu2;
        }
    float bv[4][4];
    int bt[4][4];
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int e = 0; e < 4; ++e) { bv[it][e] = INFINITY; bt[it][e] = -1; }

    // stage loads: wave w < SPT fetches tile w of the stage (4 loads of 4 key
    // rows); waves 0..1 fetch the stage's per-key data (64 keys each)
    const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(vh), (short)0, (int)(n * SPD * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t jres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float4 *>(jd), (short)0, (int)(n * 16), 0x00020000);
    uint32_t kvo[4], kro[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
        const int rr = 4 * st + grp;
        kvo[st] = ((uint32_t)rr * SPD + 8 * ((lane & 15) ^ rr)) * 2;
        kro[st] = (uint32_t)(rl * 256 + (((4 * st + grp) ^ rl) * 16));
    }
    const int64_t j0 = jc * SPJ;
    const int jn = (int)((n - j0) < SPJ ? (n - j0) : SPJ);  // keys of this chunk (multiple of 16)
    const int nst = (jn / 16 + SPT - 1) / SPT;
    auto issue = [&](int stg) {
        const int64_t sj = j0 + (int64_t)stg * SPT * 16;
        unsigned char *vb = vbuf + (stg & 1) * SP_STAGE;
        if (w < SPT && sj + 16 * w < j0 + jn) {
#pragma unroll
            for (int st = 0; st < 4; ++st)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(vres, SP_LDS(vb + w * 4096 + st * 1024), 16, kvo[st],
                                                         (uint32_t)((sj + 16 * w) * SPD * 2), 0, 0);
        }
        if (w < 2)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(jres, SP_LDS(jbuf + (stg & 1) * SPT * 16 + 64 * w), 16,
                                                     (uint32_t)lane * 16, (uint32_t)((sj + 64 * w) * 16), 0, 0);
    };
    issue(0);
    for (int stg = 0; stg < nst; ++stg) {
        if (stg + 1 < nst) issue(stg + 1);
        // this wave's loads of stage stg have landed once at most those of
        // stage stg + 1 are outstanding; the barrier makes every wave's visible
        int mine = 0;
        if (stg + 1 < nst) {
            const int64_t nj = j0 + (int64_t)(stg + 1) * SPT * 16;
            mine = ((w < SPT && nj + 16 * w < j0 + jn) ? 4 : 0) + (w < 2 ? 1 : 0);
        }
        sp_wait_vm(mine);
        __syncthreads();
        const unsigned char *vb = vbuf + (stg & 1) * SP_STAGE;
        const float4 *jb = jbuf + (stg & 1) * SPT * 16;
        const int tiles = min(SPT, jn / 16 - stg * SPT);
        for (int t = 0; t < tiles; ++t) {
            const unsigned char *kt = vb + t * 4096;
            sbf16x8 kb[4];
#pragma unroll
            for (int st = 0; st < 4; ++st) kb[st] = *(const sbf16x8 *)(kt + kro[st]);
            sf32x4 acc[4];
#pragma unroll
            for (int it = 0; it < 4; ++it) {
                acc[it] = (sf32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    acc[it] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[it][st], kb[st], acc[it], 0, 0, 0);
            }
            const float4 jv = jb[t * 16 + rl];  // this lane's key
            const int tg = stg * SPT + t;       // tile index within the chunk
#pragma unroll
            for (int it = 0; it < 4; ++it)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float tt = fmaf(-2.f, acc[it][e], Xi[it][e] + jv.z);
                    const float num = fmaf(pi[it][e] * jv.y, tt, Ai[it][e] + jv.x);
                    const float den = jv.w - pi[it][e];
                    const float val = num * __builtin_amdgcn_rcpf(den * den);
                    const bool better = val < bv[it][e];
                    bv[it][e] = better ? val : bv[it][e];
                    bt[it][e] = better ? tg : bt[it][e];
                }
        }
        __syncthreads();  // the stage buffer is refilled two stages on
    }
    // lane winner (value, i, j) with ties to the smaller i, then j
    float lv = INFINITY;
    int64_t lp = INT64_MAX;
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (bt[it][e] < 0 || !(bv[it][e] < INFINITY)) continue;
            const int ip = ibase + 16 * it + 4 * grp + e;
            const int64_t pidx = (int64_t)Sl[ip] * n + (j0 + 16 * (int64_t)bt[it][e] + rl);
            if (bv[it][e] < lv || (bv[it][e] == lv && pidx < lp)) { lv = bv[it][e]; lp = pidx; }
        }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(lv, off);
        const int64_t op = __shfl_xor(lp, off);
        if (ov < lv || (ov == lv && op < lp)) { lv = ov; lp = op; }
    }
    if (lane == 0) { redv[w] = lv; redp[w] = lp; }
    __syncthreads();
    if (tid == 0) {
        for (int ww = 1; ww < 8; ++ww)
            if (redv[ww] < lv || (redv[ww] == lv && redp[ww] < lp)) { lv = redv[ww]; lp = redp[ww]; }
        s.pv[r * s.nblk + blockIdx.x] = lv;
        s.pp[r * s.nblk + blockIdx.x] = lp;
    }
}

__global__ void __launch_bounds__(512)
swap_pairs_mfma_kernel(const uint16_t *__restrict__ v, int64_t G, int64_t n, int kk, SwapState s) {
    sweep_rows(s, [&](int64_t r) { pairs_mfma_row(v, G, n, kk, s, r); });
}

// (value, index) minimum over the workgroup, ties to the smaller index
__device__ inline void block_argmin_vi(double &v, int64_t &i, double *redv, int64_t *redi) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const double ov = __shfl_xor(v, off);
        const int64_t oi = __shfl_xor(i, off);
        if (ov < v || (ov == v && oi < i)) { v = ov; i = oi; }
    }
    if (lane == 0) { redv[w] = v; redi[w] = i; }
    __syncthreads();
    v = redv[0];
    i = redi[0];
    for (int x = 1; x < nw; ++x)
        if (redv[x] < v || (redv[x] == v && redi[x] < i)) { v = redv[x]; i = redi[x]; }
    __syncthreads();
}

// exact value of the swap (i out, j in): ||g - u_i + u_j||^2 / (P - p_i + p_j)^2,
// float64, over the columns c = c0, c0 + step, ... (a partial numerator)
template <typename T>
__device__ inline double swap_num_part(const T *vh, int d, int64_t i, int64_t j, double pi, double pj,
                                       const double *g, const double *mu, int c0, int step) {
    double acc = 0.0;
    for (int c = c0; c < d; c += step) {
        const double x = g[c] - pi * ((double)Elem<T>::load(vh, i * d + c) - mu[c]) +
                         pj * ((double)Elem<T>::load(vh, j * d + c) - mu[c]);
        acc = fma(x, x, acc);
    }
    return acc;
}

// The same numerator over every column in order (one thread per pair), the
// two key rows read a 16-byte chunk per load when d allows it: the same sum,
// term for term, as swap_num_part with c0 = 0, step = 1.
template <typename T>
__device__ inline double swap_num_rows(const T *vh, int d, int64_t i, int64_t j, double pi, double pj,
                                       const double *g, const double *mu) {
    constexpr int VEC = RowVec<T>::VEC;
    if (d % VEC != 0) return swap_num_part(vh, d, i, j, pi, pj, g, mu, 0, 1);
    const T *ri = vh + i * d, *rj = vh + j * d;
    double acc = 0.0;
    for (int c0 = 0; c0 < d; c0 += VEC) {
        float xi[VEC], xj[VEC];
        RowVec<T>::unpack(RowVec<T>::raw(ri, c0), xi);
        RowVec<T>::unpack(RowVec<T>::raw(rj, c0), xj);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const int c = c0 + e;
            const double x = g[c] - pi * ((double)xi[e] - mu[c]) + pj * ((double)xj[e] - mu[c]);
            acc = fma(x, x, acc);
        }
    }
    return acc;
}

// per row: the 8 smallest A_i (kept) and B_j (dropped), the exact values of
// their 64 pairs, and from them the upper bound
template <typename T>
__global__ void __launch_bounds__(256)
swap_ub_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, int kk, SwapState s) {
    __shared__ double redv[4];
    __shared__ int64_t redi[4];
    __shared__ double gs[256], ms[256];
    __shared__ int64_t topi[8], topj[8];
    const int64_t r = blockIdx.x;
    if (!s.st[r * 2]) return;
    const int tid = threadIdx.x, NT = blockDim.x;
    const double *sc = s.sc + r * 4;
    const double P = sc[0], g2 = sc[1];
    const float *p = s.p + r * n, *a = s.a + r * n, *bq = s.bq + r * n;
    const int32_t *Sl = s.Sl + r * kk;
    const float2 *br = s.br + r * n;
    for (int c = tid; c < d; c += NT) {
        gs[c] = s.g[r * d + c];
        ms[c] = s.mu[r * d + c];
    }
    // eight smallest B_j and A_i: each thread keeps its own eight (value,
    // index ascending) in one pass, then eight rounds over the threads' lists
    // in LDS pick the workgroup's, each after the previous (value, index)
    // one buffer for the threads' eight-entry lists and, once those are
    // merged, the kept keys' sort (four workgroups per CU fit)
    __shared__ __align__(16) unsigned char ubuf[256 * 8 * 16];
    static_assert(kSwapSort * 8 <= 256 * 8 * 16, "sort keys fit the list buffer");
    double *lv = (double *)ubuf;
    int64_t *li = (int64_t *)(ubuf + 256 * 8 * 8);
    auto top8 = [&](auto &&get, int64_t cnt, int64_t *dst) __attribute__((always_inline)) {
        double tv[8];
        int64_t ti[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) { tv[q] = INFINITY; ti[q] = INT64_MAX; }
        for (int64_t e = tid; e < cnt; e += NT) {
            int64_t id;
            const double x = get(e, id);
            if (!(x < tv[7] || (x == tv[7] && id < ti[7]))) continue;
            tv[7] = x;
            ti[7] = id;
#pragma unroll
            for (int q = 7; q > 0; --q) {
                const bool sw = tv[q] < tv[q - 1] || (tv[q] == tv[q - 1] && ti[q] < ti[q - 1]);
                const double v0 = tv[q - 1];
                const int64_t i0 = ti[q - 1];
                tv[q - 1] = sw ? tv[q] : v0;
                ti[q - 1] = sw ? ti[q] : i0;
                tv[q] = sw ? v0 : tv[q];
                ti[q] = sw ? i0 : ti[q];
            }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) { lv[tid * 8 + q] = tv[q]; li[tid * 8 + q] = ti[q]; }
        __syncthreads();
        double pv = -INFINITY;
        int64_t pi = -1;
        for (int u = 0; u < 8; ++u) {
            double bv = INFINITY;
            int64_t bi = INT64_MAX;
            for (int q = 0; q < 8; ++q) {
                const double x = lv[tid * 8 + q];
                const int64_t id = li[tid * 8 + q];
                if (!(x < INFINITY)) continue;
                const bool after = x > pv || (x == pv && id > pi);
                if (after && (x < bv || (x == bv && id < bi))) { bv = x; bi = id; }
            }
            block_argmin_vi(bv, bi, redv, redi);
            if (tid == 0) dst[u] = bi < INT64_MAX ? bi : -1;
            pv = bv;
            pi = bi;
        }
    };
    // (the same pass sums the dropped keys' r_j and p_j for the order below)
    double sr = 0.0, sp = 0.0, nd = 0.0;
    top8([&](int64_t j, int64_t &id) {
        id = j;
        const float2 b = br[j];
        if (b.x < INFINITY) {
            sr += (double)b.y;
            sp += (double)p[j];
            nd += 1.0;
        }
        return (double)b.x;
    }, n, topj);
    top8([&](int64_t t, int64_t &id) {
        const int64_t i = Sl[t];
        id = i;
        return g2 + (double)bq[i] - 2.0 * (double)a[i];
    }, (int64_t)kk, topi);
    __syncthreads();
    // the 64 pairs: four lanes per pair, each a quarter of the columns
    const int pr = tid >> 2, qt = tid & 3;
    const int64_t i = topi[pr >> 3], j = topj[pr & 7];
    const T *vh = v + (r / G) * n * d;
    double num = 0.0;
    if (i >= 0 && j >= 0) num = swap_num_part(vh, d, i, j, (double)p[i], (double)p[j], gs, ms, qt, 4);
    num += __shfl_xor(num, 1);
    num += __shfl_xor(num, 2);
    double val = INFINITY;
    int64_t pidx = INT64_MAX;
    if (i >= 0 && j >= 0 && qt == 0) {
        const double den = P - (double)p[i] + (double)p[j];
        val = num / (den * den);
        pidx = i * n + j;
    }
    block_argmin_vi(val, pidx, redv, redi);
    if (tid == 0) {
        s.ub[r * 2 + 0] = val;
        s.ub[r * 2 + 1] = 0.0;
        s.ubp[r] = pidx;
        s.cnt[r] = 0;
    }
    if (!s.ord) return;
    // Order the kept keys for the bound pass by how readily their pairs pass
    // a slice test (largest first), so that the few that do share waves and
    // the other waves skip whole slices: kappa_i = c_i + 2 r_i rt + 2 UB Pi pt
    // with rt, pt four times the mean r_j and p_j of the dropped keys.
    sr = block_reduce(sr, redv, OpSum());
    sp = block_reduce(sp, redv, OpSum());
    nd = block_reduce(nd, redv, OpSum());
    const double rt = 4.0 * sr / fmax(nd, 1.0), pt = 4.0 * sp / fmax(nd, 1.0);
    float *skey = (float *)ubuf;  // the lists are dead: their merges ended with a barrier
    int32_t *sval = (int32_t *)(ubuf + kSwapSort * 4);
    int np2 = 1;
    while (np2 < kk) np2 <<= 1;
    for (int t = tid; t < np2; t += NT) {
        float key = INFINITY;
        int32_t iv = -1;
        if (t < kk) {
            iv = Sl[t];
            const double bqi = (double)bq[iv];
            const double Ai = g2 + bqi - 2.0 * (double)a[iv];
            const double Pi = P - (double)p[iv];
            const double kap = val * Pi * Pi - Ai + 2.0 * sqrt(bqi) * rt + 2.0 * val * Pi * pt;
            key = (float)(-kap);
        }
        skey[t] = key;
        sval[t] = iv;
    }
    __syncthreads();
    for (int size = 2; size <= np2; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = tid; t < np2; t += NT) {
                const int u = t ^ stride;
                if (u > t) {
                    const bool up = (t & size) == 0;
                    const float kt = skey[t], ku = skey[u];
                    if ((kt > ku) == up && kt != ku) {
                        skey[t] = ku;
                        skey[u] = kt;
                        const int32_t vt = sval[t];
                        sval[t] = sval[u];
                        sval[u] = vt;
                    }
                }
            }
            __syncthreads();
        }
    }
    // each kept key's terms of the bound test, in the order, so that every
    // workgroup of the bound pass reads them contiguously instead of
    // gathering them per key (see swap_bound_kernel for the test)
    for (int t = tid; t < kk; t += NT) {
        const int32_t i = sval[t];
        s.ord[r * kk + t] = i;
        const double bqi = (double)bq[i];
        const double Ai = g2 + bqi - 2.0 * (double)a[i];
        const double Pi = P - (double)p[i];
        s.kd[r * kk + t] = make_float4((float)(val * (1.0 + 1e-5) * Pi * Pi - Ai + 1e-4 * g2),
                                       (float)(-2.0 * sqrt(bqi)), (float)(-2.0 * val * (1.0 + 1e-5) * Pi),
                                       __int_as_float(i));
    }
}

// every (kept i, dropped j) pair of a tile against the lower bound: BT KT
// kept keys (KT per thread) x JC keys per workgroup.  With Pi = P - p_i the
// test  A_i + B_j - 2 r_i r_j <= UB (Pi + p_j)^2  is, expanded,
//     (B_j - UB p_j^2) - 2 r_i r_j - 2 UB Pi p_j <= UB Pi^2 - A_i,
// two fused multiply-adds and a compare per pair; the keys' terms are staged
// in LDS per tile and read by all threads alike, each read serving a thread's
// KT kept keys.  Each 16-key slice of a tile is first tested as a whole, with
// its smallest B_j - UB p_j^2 and largest r_j and p_j (a lower bound for
// every pair of the slice): a wave whose kept keys all fail skips the slice.
// A wave holds 64 KT consecutive kept keys of the bound pass's order (lane l
// keys l, l + 64, ..), so the few that pass share waves.
template <int JC, int BT, int KT>
__global__ void __launch_bounds__(BT)
swap_bound_kernel(int64_t n, int kk, SwapState s) {
    __shared__ float4 tile[2][BT];
    __shared__ float4 slice[2][BT / kSwapSL];
    const int64_t r = blockIdx.y;
    if (!s.st[r * 2]) return;
    const int tid = threadIdx.x, lane = tid & 63;
    constexpr int KB = BT * KT;  // kept keys per workgroup
    const int nic = (kk + KB - 1) / KB, ic = blockIdx.x % nic, jc = blockIdx.x / nic;
    const double *sc = s.sc + r * 4;
    const double P = sc[0], g2 = sc[1], UB = s.ub[r * 2 + 0];
    // the kept keys most likely to pass (first in the order) fill one wave
    // per workgroup; which wave rotates with the key chunk, so that those
    // waves of the workgroups on a CU sit on different SIMDs
    const int wv = ((tid >> 6) + jc) % (BT / 64);
    int64_t i[KT];
    float ci[KT], m2r[KT], m2u[KT];
#pragma unroll
    for (int q = 0; q < KT; ++q) {
        const int t = ic * KB + wv * 64 * KT + q * 64 + lane;
        i[q] = -1;
        ci[q] = -INFINITY;
        m2r[q] = 0.f;
        m2u[q] = 0.f;
        if (t < kk && s.kd) {  // formed by the upper-bound pass, in this order
            const float4 e = s.kd[r * kk + t];
            ci[q] = e.x;
            m2r[q] = e.y;
            m2u[q] = e.z;
            i[q] = __float_as_int(e.w);
        } else if (t < kk) {
            i[q] = s.Sl[r * kk + t];
            const double bqi = (double)s.bq[r * n + i[q]];
            const double Ai = g2 + bqi - 2.0 * (double)s.a[r * n + i[q]];
            const double Pi = P - (double)s.p[r * n + i[q]];
            // margins cover the float32 rounding of A, B and the test itself
            ci[q] = (float)(UB * (1.0 + 1e-5) * Pi * Pi - Ai + 1e-4 * g2);
            m2r[q] = (float)(-2.0 * sqrt(bqi));
            m2u[q] = (float)(-2.0 * UB * (1.0 + 1e-5) * Pi);
        }
    }
    const float ubf = (float)(UB * (1.0 + 1e-5));
    const float2 *br = s.br + r * n;
    const float *pr = s.p + r * n;
    const int64_t j0 = (int64_t)jc * JC, j1 = j0 + JC < n ? j0 + JC : n;
    auto pass = [&](const float4 &b, int q) __attribute__((always_inline)) {
        return fmaf(m2u[q], b.z, fmaf(m2r[q], b.y, b.x)) <= ci[q];
    };
    // the next tile's keys are loaded while this one is tested; two LDS
    // buffers, one barrier per tile
    float2 nb = make_float2(INFINITY, 0.f);
    float np = 0.f;
    if (j0 + tid < j1) {
        nb = br[j0 + tid];
        np = pr[j0 + tid];
    }
    int buf = 0;
    for (int64_t jt = j0; jt < j1; jt += BT, buf ^= 1) {
        float4 (&tile_b)[BT] = tile[buf];
        {
            const float2 b = nb;
            const float pj = np;
            if (jt + BT + tid < j1) {
                nb = br[jt + BT + tid];
                np = pr[jt + BT + tid];
            }
            float4 e = make_float4(INFINITY, 0.f, 0.f, 0.f);
            if (jt + tid < j1) e = make_float4(b.x - ubf * pj * pj, b.y, pj, 0.f);
            tile_b[tid] = e;
            float mb = e.x, mr = e.x < INFINITY ? e.y : 0.f, mp = e.x < INFINITY ? e.z : 0.f;
#pragma unroll
            for (int off = kSwapSL / 2; off > 0; off >>= 1) {
                mb = fminf(mb, __shfl_xor(mb, off));
                mr = fmaxf(mr, __shfl_xor(mr, off));
                mp = fmaxf(mp, __shfl_xor(mp, off));
            }
            if ((tid & (kSwapSL - 1)) == 0) slice[buf][tid / kSwapSL] = make_float4(mb, mr, mp, 0.f);
        }
        __syncthreads();
        for (int u0 = 0; u0 < BT; u0 += kSwapSL) {
            const float4 sl = slice[buf][u0 / kSwapSL];
            bool hs = false;
#pragma unroll
            for (int q = 0; q < KT; ++q) hs |= pass(sl, q);
            if (!__ballot(hs)) continue;
            uint64_t any = 0;
#pragma unroll
            for (int u = 0; u < kSwapSL; ++u) {
                const float4 b = tile_b[u0 + u];
                bool h = false;
#pragma unroll
                for (int q = 0; q < KT; ++q) h |= pass(b, q);
                any |= __ballot(h);
            }
            if (any) {  // rare: each kept key's survivors of the slice, one list slot range per wave
#pragma unroll
                for (int q = 0; q < KT; ++q) {
                    uint32_t m = 0;
#pragma unroll
                    for (int u = 0; u < kSwapSL; ++u) m |= (pass(tile_b[u0 + u], q) ? 1u : 0u) << u;
                    const int c = __popc(m);
                    if (!__ballot(c > 0)) continue;
                    int incl = c;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const int y = __shfl_up(incl, off);
                        if (lane >= off) incl += y;
                    }
                    int base = 0;
                    if (lane == 63) base = atomicAdd(&s.cnt[r], incl);
                    base = __shfl(base, 63);
                    int pos = base + incl - c;
                    for (; m; m &= m - 1, ++pos)
                        if (pos < kSwapCand) s.cand[r * kSwapCand + pos] = i[q] * n + (jt + u0 + __ffs(m) - 1);
                }
            }
        }
    }
}

// the survivors (and the upper bound's own pair) evaluated exactly; the
// winner goes to the first partial slot of the row, the others are cleared
template <typename T>
__global__ void __launch_bounds__(256)
swap_cand_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, SwapState s) {
    __shared__ double redv[4];
    __shared__ int64_t redi[4];
    __shared__ double gs[256], ms[256];
    const int64_t r = blockIdx.x;
    if (!s.st[r * 2]) return;
    const int tid = threadIdx.x, NT = blockDim.x;
    const int cnt = s.cnt[r];
    if (cnt > kSwapCand) {  // overflow: the full sweep decides this row
        if (tid == 0) {
            s.fb[r] = 1;
            s.fbl[atomicAdd(s.fbn, 1)] = (int32_t)r;
        }
        return;
    }
    if (tid == 0) s.fb[r] = 0;
    for (int c = tid; c < d; c += NT) {
        gs[c] = s.g[r * d + c];
        ms[c] = s.mu[r * d + c];
    }
    __syncthreads();
    const double P = s.sc[r * 4 + 0];
    const float *p = s.p + r * n;
    const T *vh = v + (r / G) * n * d;
    double bv = INFINITY;
    int64_t bp = INT64_MAX;
    for (int c = tid; c <= cnt; c += NT) {
        const int64_t pidx = c < cnt ? s.cand[r * kSwapCand + c] : s.ubp[r];
        if (pidx < 0 || pidx >= n * n) continue;
        const int64_t i = pidx / n, j = pidx % n;
        const double num = swap_num_rows(vh, d, i, j, (double)p[i], (double)p[j], gs, ms);
        const double den = P - (double)p[i] + (double)p[j];
        const double val = num / (den * den);
        if (val < bv || (val == bv && pidx < bp)) { bv = val; bp = pidx; }
    }
    block_argmin_vi(bv, bp, redv, redi);
    for (int b = tid; b < s.nblk; b += NT) {
        s.pv[r * s.nblk + b] = b == 0 ? (float)bv : INFINITY;
        s.pp[r * s.nblk + b] = b == 0 ? bp : INT64_MAX;
    }
}

// reduce the tile winners, then apply the swap (or retire the row)
template <typename T>
__global__ void __launch_bounds__(256)
swap_apply_kernel(const T *__restrict__ v, int64_t G, int64_t n, int d, int kk, SwapState s,
                  float *gap_traj, int T_len) {
    __shared__ float redv[256];
    __shared__ int64_t redp[256];
    __shared__ double redd[256];
    __shared__ int decide;
    const int64_t r = blockIdx.x;
    if (s.fbn && r == 0 && threadIdx.x == 0) *s.fbn = 0;  // the sweep that read it is done
    if (!s.st[r * 2]) return;
    const int tid = threadIdx.x;
    float bv = INFINITY;
    int64_t bp = INT64_MAX;
    for (int b = tid; b < s.nblk; b += blockDim.x) {
        const float v2 = s.pv[r * s.nblk + b];
        const int64_t p2 = s.pp[r * s.nblk + b];
        if (v2 < bv || (v2 == bv && p2 < bp)) { bv = v2; bp = p2; }
    }
    redv[tid] = bv;
    redp[tid] = bp;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if (tid < st) {
            const float v2 = redv[tid + st];
            const int64_t p2 = redp[tid + st];
            if (v2 < redv[tid] || (v2 == redv[tid] && p2 < redp[tid])) { redv[tid] = v2; redp[tid] = p2; }
        }
        __syncthreads();
    }
    // the float32 search proposes (i, j); accept only on a strict decrease of
    // the float64 value ||g - u_i + u_j||^2 / (P - p_i + p_j)^2
    double *sc = s.sc + r * 4;
    if (!(redv[0] < INFINITY) || redp[0] < 0 || redp[0] >= (int64_t)n * n) {  // no finite candidate
        if (tid == 0) s.st[r * 2] = 0;
        return;
    }
    const int64_t i = redp[0] / n, j = redp[0] % n;
    const int64_t h = r / G;
    const T *vh = v + h * n * d;
    const float *p = s.p + r * n;
    double *g = s.g + r * d;
    const double *mu = s.mu + r * d;
    double g2 = 0.0;
    for (int c = tid; c < d; c += blockDim.x) {
        const double ui = (double)p[i] * ((double)Elem<T>::load(vh, i * d + c) - mu[c]);
        const double uj = (double)p[j] * ((double)Elem<T>::load(vh, j * d + c) - mu[c]);
        const double gn = g[c] - ui + uj;
        g2 += gn * gn;
    }
    g2 = block_reduce(g2, redd, OpSum());
    const double P = sc[0] - (double)p[i] + (double)p[j];
    if (tid == 0) decide = (g2 / (P * P) < sc[3]) ? 1 : 0;
    __syncthreads();
    if (!decide) {
        if (tid == 0) s.st[r * 2] = 0;
        return;
    }
    for (int c = tid; c < d; c += blockDim.x) {
        const double ui = (double)p[i] * ((double)Elem<T>::load(vh, i * d + c) - mu[c]);
        const double uj = (double)p[j] * ((double)Elem<T>::load(vh, j * d + c) - mu[c]);
        g[c] = g[c] - ui + uj;
    }
    if (tid == 0) {
        s.inS[r * n + i] = 0;
        s.inS[r * n + j] = 1;
        for (int t = 0; t < kk; ++t)
            if (s.Sl[r * kk + t] == (int32_t)i) { s.Sl[r * kk + t] = (int32_t)j; break; }
        sc[0] = P;
        sc[1] = g2;
        sc[3] = g2 / (P * P);
        const int sw = ++s.st[r * 2 + 1];
        gap_traj[r * T_len + sw] = (float)(sqrt(g2) / P);
    }
}

__global__ void __launch_bounds__(256)
swap_final_kernel(int64_t n, int kk, SwapState s, int32_t *s_idx, float *gap_traj, int T_len,
                  int32_t *n_swaps, float *dropped) {
    __shared__ int scan[256];
    __shared__ double redd[256];
    const int64_t r = blockIdx.x;
    const int tid = threadIdx.x, NT = blockDim.x;
    const uint8_t *inS = s.inS + r * n;
    const float *p = s.p + r * n;
    const int64_t chunk = (n + NT - 1) / NT;
    const int64_t lo = tid * chunk, hi = (lo + chunk < n) ? lo + chunk : n;
    int c = 0;
    double dm = 0.0;
    for (int64_t j = lo; j < hi; ++j) {
        c += inS[j];
        if (!inS[j]) dm += (double)p[j];
    }
    int total;
    int pos = block_exclusive_scan(c, scan, &total);
    for (int64_t j = lo; j < hi; ++j)
        if (inS[j]) s_idx[r * kk + pos++] = (int32_t)j;
    dm = block_reduce(dm, redd, OpSum());
    const int sw = s.st[r * 2 + 1];
    for (int t = sw + 1 + tid; t < T_len; t += NT) gap_traj[r * T_len + t] = __int_as_float(0x7fc00000);
    if (tid == 0) {
        n_swaps[r] = sw;
        if (dropped) dropped[r] = (float)dm;
    }
}

// ===========================================================================
// host side
// ===========================================================================
namespace {

constexpr int kSwapJC = 1024;  // keys per workgroup of the bound pass
constexpr int kSwapBT = 256;   // threads per workgroup of the bound pass
constexpr int kSwapKT = 4;     // kept keys per thread of the bound pass
constexpr int kSwapRB = 32;    // rows of one unit per workgroup of the dots pass

// the MFMA pair sweep: bf16, d = 128, whole 16-key tiles
bool swap_mfma_ok(const fw_rows &rows) {
    return rows.dtype == FW_BF16 && rows.d == SPD && rows.n % 16 == 0 && rows.n * SPD * 2 < ((int64_t)1 << 31);
}

size_t small_lds(int n, int d, int nt) {
    size_t b = (size_t)n * n * 8 + (size_t)n * 8 * 3 + (size_t)d * 8 + (size_t)nt * 16;
    b += (size_t)(n + (n & 1)) * 4 + (size_t)n * instance_pitch(d) * 4;
    return b;
}

struct SwapLayout {
    SwapState s;
    float *z, *row_m, *row_l;
    uint32_t *thr_key;
    int32_t *thr_cut;
    size_t bytes;
};

SwapLayout swap_layout(const fw_rows &rows, int k, void *ws) {
    const size_t R = (size_t)rows.H * rows.G, n = rows.n, d = rows.d;
    SwapLayout L{};
    size_t off = 0;
    char *base = (char *)ws;
    auto take = [&](size_t bytes) -> void * {
        off = align_up(off, 256);
        void *p = base ? base + off : nullptr;
        off += bytes;
        return p;
    };
    if (swap_mfma_ok(rows)) {
        L.s.nblk = (int)(((k + SPI - 1) / SPI) * (((int64_t)n + SPJ - 1) / SPJ));
    } else {
        const int itiles = (k + 31) / 32;
        const int64_t jtiles = ((int64_t)n + 127) / 128;
        L.s.nblk = (int)(itiles * jtiles);
    }
    L.z = (float *)take(R * n * 4);
    L.row_m = (float *)take(R * 4);
    L.row_l = (float *)take(R * 4);
    L.thr_key = (uint32_t *)take(R * 4);
    L.thr_cut = (int32_t *)take(R * 4);
    L.s.p = (float *)take(R * n * 4);
    L.s.inS = (uint8_t *)take(R * n);
    L.s.Sl = (int32_t *)take(R * k * 4);
    L.s.w = (float *)take(R * n * 4);
    L.s.bq = (float *)take(R * n * 4);
    L.s.a = (float *)take(R * n * 4);
    L.s.mu = (double *)take(R * d * 8);
    L.s.g = (double *)take(R * d * 8);
    L.s.sc = (double *)take(R * 4 * 8);
    L.s.st = (int32_t *)take(R * 2 * 4);
    L.s.pv = (float *)take(R * L.s.nblk * 4);
    L.s.pp = (int64_t *)take(R * L.s.nblk * 8);
    L.s.jd = swap_mfma_ok(rows) ? (float4 *)take(R * n * 16) : nullptr;
    if (d <= 256) {  // the pruned search stages g and mu (float64) per workgroup
        L.s.br = (float2 *)take(R * n * 8);
        L.s.ub = (double *)take(R * 2 * 8);
        L.s.ubp = (int64_t *)take(R * 8);
        L.s.cnt = (int32_t *)take(R * 4);
        L.s.fb = (int32_t *)take(R * 4);
        L.s.fbl = (int32_t *)take(R * 4);
        L.s.fbn = (int32_t *)take(16);
        L.s.cand = (int64_t *)take(R * (size_t)kSwapCand * 8);
        if (k <= kSwapSort) {
            L.s.ord = (int32_t *)take(R * (size_t)k * 4);
            L.s.kd = (float4 *)take(R * (size_t)k * 16);
        }
    }
    // the dots pass writes a only for the kept keys when the fallback sweep
    // is the MFMA one (it takes B_j from br); the float sweep reads a[j]
    L.s.a_all = (L.s.br && swap_mfma_ok(rows)) ? 0 : 1;
    L.s.z = L.z;
    L.s.row_m = L.row_m;
    L.s.row_l = L.row_l;
    L.s.thr_key = L.thr_key;
    L.s.thr_cut = L.thr_cut;
    L.bytes = align_up(off, 256);
    return L;
}

}  // namespace

size_t swap_ws_bytes(const fw_rows &rows, int k, int max_iters) {
    (void)max_iters;
    if (rows.n <= 64) return 256;
    return swap_layout(rows, k, nullptr).bytes;
}

template <typename T>
static hipError_t swap_large(const fw_rows &rows, int k, int max_iters, int32_t *s_idx,
                             float *gap_traj, int32_t *n_swaps, float *dropped, void *ws,
                             hipStream_t st) {
    SwapLayout L = swap_layout(rows, k, ws);
    const int64_t H = rows.H, G = rows.G, n = rows.n, R = H * G;
    const int d = (int)rows.d;
    hipError_t e = launch_scores(rows.dtype, rows.q, rows.k, rows.scale, rows.bias, H, G, n, d, L.z, st);
    if (e != hipSuccess) return e;
    KsArg ks{};
    ks.n = 1;
    ks.k[0] = k;
    ks.perm[0] = 0;
    e = launch_select(L.z, R, n, ks, L.row_m, L.row_l, L.thr_key, L.thr_cut, nullptr, k, st);
    if (e != hipSuccess) return e;
    const T *v = (const T *)rows.v;
    const int T_len = max_iters + 1;
    hipLaunchKernelGGL(swap_init_kernel<T>, dim3((unsigned)R), dim3(256), 0, st, v, G, n, d, k, L.s,
                       gap_traj, T_len);
    const unsigned dot_blocks = (unsigned)((n + 255) / 256 < 64 ? (n + 255) / 256 : 64);
    for (int it = 0; it < max_iters; ++it) {
        if (G % kSwapRB == 0 && d <= 256)
            hipLaunchKernelGGL((swap_dots_group_kernel<T, kSwapRB>), dim3(dot_blocks, (unsigned)(R / kSwapRB)),
                               dim3(256), 0, st, v, G, n, d, L.s);
        else
            hipLaunchKernelGGL(swap_dots_kernel<T>, dim3(dot_blocks, (unsigned)R), dim3(256), 0, st, v, G,
                               n, d, L.s);
        if (L.s.br) {  // pruned search; the sweep below then runs only for overflowing rows
            hipLaunchKernelGGL(swap_ub_kernel<T>, dim3((unsigned)R), dim3(256), 0, st, v, G, n, d, k, L.s);
            hipLaunchKernelGGL((swap_bound_kernel<kSwapJC, kSwapBT, kSwapKT>),
                               dim3((unsigned)(((k + kSwapBT * kSwapKT - 1) / (kSwapBT * kSwapKT)) *
                                               ((n + kSwapJC - 1) / kSwapJC)),
                                    (unsigned)R),
                               dim3(kSwapBT), 0, st, n, k, L.s);
            hipLaunchKernelGGL(swap_cand_kernel<T>, dim3((unsigned)R), dim3(256), 0, st, v, G, n, d, L.s);
        }
        // under the pruned search the sweep takes only the listed rows
        const unsigned sweep_y = L.s.fbl ? (unsigned)(R < kSwapSweepRows ? R : kSwapSweepRows) : (unsigned)R;
        if (swap_mfma_ok(rows) && L.s.br)  // the listed rows' sweep records
            hipLaunchKernelGGL(swap_jd_kernel, dim3((unsigned)((n + 1023) / 1024), sweep_y), dim3(256), 0, st,
                               n, L.s);
        if (swap_mfma_ok(rows))
            hipLaunchKernelGGL(swap_pairs_mfma_kernel, dim3((unsigned)L.s.nblk, sweep_y), dim3(512),
                               (size_t)(2 * SP_STAGE + 2 * SPT * 16 * 16 + 8 * 4 + 8 * 8), st,
                               (const uint16_t *)rows.v, G, n, k, L.s);
        else
            hipLaunchKernelGGL(swap_pairs_kernel<T>, dim3((unsigned)L.s.nblk, sweep_y), dim3(256), 0,
                               st, v, G, n, d, k, L.s);
        hipLaunchKernelGGL(swap_apply_kernel<T>, dim3((unsigned)R), dim3(256), 0, st, v, G, n, d, k,
                           L.s, gap_traj, T_len);
    }
    hipLaunchKernelGGL(swap_final_kernel, dim3((unsigned)R), dim3(256), 0, st, n, k, L.s, s_idx,
                       gap_traj, T_len, n_swaps, dropped);
    return hipGetLastError();
}

hipError_t launch_swap(const fw_rows &rows, int k, int max_iters, int32_t *s_idx, float *gap_traj,
                       int32_t *n_swaps, float *dropped, void *ws, hipStream_t st) {
    const int64_t R = rows.H * rows.G;
    if (rows.n <= 64) {
        const int n = (int)rows.n, d = (int)rows.d;
        int nt = 256;
        while (nt > 64 && small_lds(n, d, nt) > 160 * 1024) nt >>= 1;
        const size_t lds = small_lds(n, d, nt);
        if (rows.dtype == FW_BF16)
            hipLaunchKernelGGL(swap_small_kernel<uint16_t>, dim3((unsigned)R), dim3(nt), lds, st,
                               (const uint16_t *)rows.q, (const uint16_t *)rows.k, (const uint16_t *)rows.v,
                               rows.scale, rows.bias, rows.G, n, d, k, max_iters, s_idx, gap_traj,
                               n_swaps, dropped);
        else
            hipLaunchKernelGGL(swap_small_kernel<float>, dim3((unsigned)R), dim3(nt), lds, st,
                               (const float *)rows.q, (const float *)rows.k, (const float *)rows.v,
                               rows.scale, rows.bias, rows.G, n, d, k, max_iters, s_idx, gap_traj,
                               n_swaps, dropped);
        return hipGetLastError();
    }
    if (rows.dtype == FW_BF16)
        return swap_large<uint16_t>(rows, k, max_iters, s_idx, gap_traj, n_swaps, dropped, ws, st);
    return swap_large<float>(rows, k, max_iters, s_idx, gap_traj, n_swaps, dropped, ws, st);
}

}  // namespace fw
