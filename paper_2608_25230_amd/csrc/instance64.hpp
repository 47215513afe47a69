// One attention row as an instance of Definition 2.1, in float64: logits,
// weights p = softmax(z), dense output mu and the Gram matrix of the
// residuals u_j = p_j (v_j - mu) (Lemma 2.2), for rows of at most 64 keys.
// Every sum runs in a fixed order, so results are bitwise repeatable.
#pragma once

#include "fw_common.hpp"

namespace fw {

// The documented default scale 1/sqrt(d), as the float32 value callers pass.
__device__ __forceinline__ float default_scale(int d) { return (float)(1.0 / sqrt((double)d)); }

// Row pitch (floats) of the values staged in LDS: d + 1 keeps the column
// reads of different rows on different banks.
__host__ __device__ inline int instance_pitch(int d) { return d + 1; }

// Elements [first, n d) of a row-major [n][d] matrix into LDS at row pitch
// `pitch` (floats), every thread of the workgroup taking elements NT apart
// (first a multiple of NT), eight global loads in flight per thread.
template <typename T>
__device__ __forceinline__ void stage_rows_from(const T *src, int n, int d, float *dst, int pitch, int first) {
    const int NT = blockDim.x;
    const int rstep = NT / d, cstep = NT - rstep * d;
    const int e = first + threadIdx.x;
    int r = e / d, c = e - (e / d) * d;
    const int tot = n * d;
    for (int e0 = e; e0 < tot; e0 += 8 * NT) {
        float buf[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (e0 + u * NT < tot) buf[u] = Elem<T>::load(src, e0 + u * NT);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (e0 + u * NT < tot) dst[r * pitch + c] = buf[u];
            r += rstep;
            c += cstep;
            if (c >= d) {
                c -= d;
                ++r;
            }
        }
    }
}

template <typename T>
__device__ __forceinline__ void stage_rows(const T *src, int n, int d, float *dst, int pitch) {
    stage_rows_from(src, n, d, dst, pitch, 0);
}

// The Gram entries of instance64 for L lanes per 4 x 4 block (L a power of
// two up to 8, at most blockDim.x / L blocks at a time).  The columns a lane
// takes are c = part + i L: a uniform count of whole rounds (d / L) and at
// most one more, so the loads are fixed offsets from nine row pointers
// (constants throughout for d = 128 and L >= 4).
template <int L>
__device__ __forceinline__ void gram_blocks(int n, int d, int pitch, int nb, int nblk, const float *Vs,
                                            const double *ps, const double *mu, double *Gm, int gp, double *Yd) {
    const int tid = threadIdx.x, NT = blockDim.x;
    constexpr int lgL = L == 8 ? 3 : L == 4 ? 2 : L == 2 ? 1 : 0;
    const int ntask = ((nblk * L + 63) / 64) * 64;
    const int full = d / L;
    for (int task = tid; task < ntask; task += NT) {
        const int blk = task >> lgL, part = task & (L - 1);
        int A = 0, rem = blk < nblk ? blk : 0;
        while (rem >= nb - A) { rem -= nb - A; ++A; }
        const int B = A + rem;
        const float *ra[4], *rb[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            ra[x] = Vs + min(4 * A + x, n - 1) * pitch + part;
            rb[x] = Vs + min(4 * B + x, n - 1) * pitch + part;
        }
        const double *mc = mu + part;
        double sg[4][4];
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int y = 0; y < 4; ++y) sg[x][y] = 0.0;
        auto col = [&](int o) __attribute__((always_inline)) {
            const double m = mc[o];
            double va[4], vb[4];
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                va[x] = (double)ra[x][o] - m;
                vb[x] = (double)rb[x][o] - m;
            }
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) sg[x][y] = fma(va[x], vb[y], sg[x][y]);
        };
        if (L >= 4 && d == 128) {  // the common head size: every offset a constant
#pragma unroll
            for (int i = 0; i < 128 / L; ++i) {
                col(i * L);
                if (i & 1) __builtin_amdgcn_sched_barrier(0);
            }
        } else {
            int i = 0;
            for (; i + 2 <= full; i += 2) {
                col(i * L);
                col((i + 1) * L);
            }
            for (; i < full; ++i) col(i * L);
            if (part < d - full * L) col(full * L);
        }
        for (int off = 1; off < L; off <<= 1)
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) sg[x][y] += __shfl_xor(sg[x][y], off);
        if (blk < nblk) {
            // lane `part` of the group writes entries part, part + L, .. of 16
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int ii = 4 * A + e / 4, jj = 4 * B + e % 4;
                if ((e & (L - 1)) == part && ii < n && jj < n) {
                    const double g = ps[ii] * ps[jj] * sg[e / 4][e % 4];
                    Gm[ii * gp + jj] = g;
                    Gm[jj * gp + ii] = g;
                    if (Yd) {
                        Yd[ii * gp + jj] = sg[e / 4][e % 4];
                        Yd[jj * gp + ii] = sg[e / 4][e % 4];
                    }
                }
            }
        }
    }
}

// Whole workgroup: Gm[i][j] = p_i p_j <v_i - mu, v_j - mu> (row pitch gp)
// for the n rows of Vs (pitch `pitch` floats), and, when Yd is given, the
// inner products themselves, in 4 x 4 blocks of rows (4A .. 4A + 3) x
// (4B .. 4B + 3), A <= B, each on L adjacent lanes that split the columns and
// add their sums by a butterfly; rows past n read row n - 1 and are not
// written.  Whole waves take part, so every butterfly sees its group.
__device__ __forceinline__ void gram_matrix(int n, int d, int pitch, const float *Vs, const double *ps,
                                            const double *mu, double *Gm, int gp, double *Yd) {
    const int nb = (n + 3) >> 2, nblk = nb * (nb + 1) / 2;
    int lgL = 3;
    while (lgL > 0 && (nblk << lgL) > (int)blockDim.x) --lgL;
    switch (lgL) {
        case 3: gram_blocks<8>(n, d, pitch, nb, nblk, Vs, ps, mu, Gm, gp, Yd); break;
        case 2: gram_blocks<4>(n, d, pitch, nb, nblk, Vs, ps, mu, Gm, gp, Yd); break;
        case 1: gram_blocks<2>(n, d, pitch, nb, nblk, Vs, ps, mu, Gm, gp, Yd); break;
        default: gram_blocks<1>(n, d, pitch, nb, nblk, Vs, ps, mu, Gm, gp, Yd); break;
    }
}

// Whole workgroup; n <= 64 <= blockDim.x, blockDim.x a multiple of 64.
// Vs [n][d + 1] float (LDS) stages the keys, then the values; zs, ps [n],
// mu [d], Gm [n][gp] (LDS, row pitch gp >= n) receive the instance.  Global
// reads are coalesced (whole rows); the logits, weights, dense output and
// Gram are formed from LDS, each sum in a fixed order.
template <typename T>
__device__ __forceinline__ void instance64(const T *qr, const T *kh, const T *vh, float scale, const float *bias,
                           int n, int d, float *Vs, double *zs, double *ps, double *mu, double *Gm, int gp) {
    const int tid = threadIdx.x, NT = blockDim.x;
    const int pitch = instance_pitch(d);
    float *qs = (float *)mu;  // the query, in the dense output's space until that is formed
    stage_rows(kh, n, d, Vs, pitch);
    for (int c = tid; c < d; c += NT) qs[c] = Elem<T>::load(qr, c);
    // the first 16 values per thread are loaded now and land in LDS after
    // the logits (their loads overlap that phase)
    const int tot = n * d;
    float vpre[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
        if (tid + u * NT < tot) vpre[u] = Elem<T>::load(vh, tid + u * NT);
    __syncthreads();
    {
        // logits: lpk adjacent lanes per key (a power of two dividing 64),
        // strided partial sums combined by a fixed butterfly
        int lpk = 8;
        while (lpk > 1 && lpk * n > NT) lpk >>= 1;
        const int key = tid / lpk, part = tid & (lpk - 1);
        double dot = 0.0;
        if (key < n)
            for (int c = part; c < d; c += lpk) dot = fma((double)qs[c], (double)Vs[key * pitch + c], dot);
        for (int off = 1; off < lpk; off <<= 1) dot += __shfl_xor(dot, off);
        if (key < n && part == 0) zs[key] = (double)scale * dot + (bias ? (double)bias[key] : 0.0);
    }
    __syncthreads();
    {
        const int rstep = NT / d, cstep = NT - rstep * d;
        int r = tid / d, c = tid - (tid / d) * d;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            if (tid + u * NT < tot) Vs[r * pitch + c] = vpre[u];
            r += rstep;
            c += cstep;
            if (c >= d) {
                c -= d;
                ++r;
            }
        }
        if (tot > 16 * NT) stage_rows_from(vh, n, d, Vs, pitch, 16 * NT);
    }
    if (tid < 64) {  // softmax on one wave, fixed reduction order
        const double z = tid < n ? zs[tid] : -INFINITY;
        double m = z;
        for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
        const double ez = tid < n ? exp(z - m) : 0.0;
        double l = ez;
        for (int off = 32; off > 0; off >>= 1) l += __shfl_xor(l, off);
        if (tid < n) ps[tid] = ez / l;
    }
    __syncthreads();
    for (int c = tid; c < d; c += NT) {
        double s = 0.0;
        for (int j = 0; j < n; ++j) s = fma(ps[j], (double)Vs[j * pitch + c], s);
        mu[c] = s;
    }
    __syncthreads();
    gram_matrix(n, d, pitch, Vs, ps, mu, Gm, gp, nullptr);
    __syncthreads();
}

// Top-k set of the row as a bit mask: rank by (logit desc, index asc).  When
// idx is given, idx[rank] = key for the k best.  Every wave forms the mask
// itself from zs (no barrier); n <= 64.
__device__ inline uint64_t topk_mask64(const double *zs, int n, int k, int32_t *idx) {
    const int lane = threadIdx.x & 63;
    int rank = n;
    if (lane < n) {
        const double z = zs[lane];
        rank = 0;
        for (int i = 0; i < n; ++i) rank += (zs[i] > z) || (zs[i] == z && i < lane);
        if (rank < k && idx && threadIdx.x < 64) idx[rank] = lane;
    }
    return __ballot(rank < k);
}

// es(A) = ||sum_{j in A} p_j (v_j - mu)|| / p(A) from the d-dimensional sums
// (Lemma 2.2, second form), reading values from global memory.  The full key
// set gives m_A = mu, so es = 0 exactly.
template <typename T>
__device__ double exact_gap(uint64_t A, int n, const T *vh, const double *ps, const double *mu,
                            int d, double *red) {
    if (__popcll(A) == n) return 0.0;
    double g2 = 0.0;
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
        double gc = 0.0;
        for (uint64_t m = A; m; m &= m - 1) {
            const int j = __ffsll((unsigned long long)m) - 1;
            gc += ps[j] * ((double)Elem<T>::load(vh, (size_t)j * d + c) - mu[c]);
        }
        g2 += gc * gc;
    }
    g2 = block_reduce(g2, red, OpSum());
    double P = 0.0;
    for (uint64_t m = A; m; m &= m - 1) P += ps[__ffsll((unsigned long long)m) - 1];
    return sqrt(g2) / P;
}

// The same error from values staged in LDS (Vs [n][pitch] floats).
__device__ inline double exact_gap_lds(uint64_t A, int n, const float *Vs, int pitch, const double *ps,
                                       const double *mu, int d, double *red) {
    if (__popcll(A) == n) return 0.0;
    double g2 = 0.0;
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
        double gc = 0.0;
        for (uint64_t m = A; m; m &= m - 1) {
            const int j = __ffsll((unsigned long long)m) - 1;
            gc += ps[j] * ((double)Vs[j * pitch + c] - mu[c]);
        }
        g2 += gc * gc;
    }
    g2 = block_reduce(g2, red, OpSum());
    double P = 0.0;
    for (uint64_t m = A; m; m &= m - 1) P += ps[__ffsll((unsigned long long)m) - 1];
    return sqrt(g2) / P;
}

__device__ inline double mass64(uint64_t A, const double *ps) {
    double P = 0.0;
    for (uint64_t m = A; m; m &= m - 1) P += ps[__ffsll((unsigned long long)m) - 1];
    return P;
}

// es of two sets at once from values staged in LDS (one workgroup
// reduction for both).
__device__ inline double2 exact_gap2_lds(uint64_t A, uint64_t B, int n, const float *Vs, int pitch,
                                         const double *ps, const double *mu, int d, double *red) {
    double ga = 0.0, gb = 0.0;
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
        double sa = 0.0, sb = 0.0;
        for (int j = 0; j < n; ++j) {
            const double u = ps[j] * ((double)Vs[j * pitch + c] - mu[c]);
            if ((A >> j) & 1ull) sa += u;
            if ((B >> j) & 1ull) sb += u;
        }
        ga += sa * sa;
        gb += sb * sb;
    }
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        ga += __shfl_xor(ga, off);
        gb += __shfl_xor(gb, off);
    }
    if (lane == 0) {
        red[2 * w] = ga;
        red[2 * w + 1] = gb;
    }
    __syncthreads();
    double ta = red[0], tb = red[1];
    for (int i = 1; i < nw; ++i) {
        ta += red[2 * i];
        tb += red[2 * i + 1];
    }
    __syncthreads();
    const double pa = mass64(A, ps), pb = mass64(B, ps);
    return make_double2(__popcll(A) == n ? 0.0 : sqrt(ta) / pa, __popcll(B) == n ? 0.0 : sqrt(tb) / pb);
}


}  // namespace fw
