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

// Whole workgroup; n <= 64 <= blockDim.x.  Vs [n][d + 1] float (LDS) stages
// the keys, then the values; zs, ps [n], mu [d], Gm [n][gp] (LDS, row pitch
// gp >= n) receive the instance.  Global reads are coalesced (whole rows); the logits, weights,
// dense output and Gram are formed from LDS.
template <typename T>
__device__ void instance64(const T *qr, const T *kh, const T *vh, float scale, const float *bias,
                           int n, int d, float *Vs, double *zs, double *ps, double *mu, double *Gm, int gp) {
    const int tid = threadIdx.x, NT = blockDim.x;
    const int pitch = instance_pitch(d);
    float *qs = (float *)mu;  // the query, in the dense output's space until that is formed
    for (int e = tid; e < n * d; e += NT) Vs[(e / d) * pitch + e % d] = Elem<T>::load(kh, e);
    for (int c = tid; c < d; c += NT) qs[c] = Elem<T>::load(qr, c);
    __syncthreads();
    if (tid < n) {
        double dot = 0.0;
        for (int c = 0; c < d; ++c) dot = fma((double)qs[c], (double)Vs[tid * pitch + c], dot);
        zs[tid] = (double)scale * dot + (bias ? (double)bias[tid] : 0.0);
    }
    __syncthreads();
    for (int e = tid; e < n * d; e += NT) Vs[(e / d) * pitch + e % d] = Elem<T>::load(vh, e);
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
    for (int e = tid; e < n * (n + 1) / 2; e += NT) {
        // e -> (i, j), i <= j, row-major over the upper triangle
        int i = 0, rem = e;
        while (rem >= n - i) { rem -= n - i; ++i; }
        const int j = i + rem;
        double s = 0.0;
        for (int c = 0; c < d; ++c) s = fma((double)Vs[i * pitch + c] - mu[c], (double)Vs[j * pitch + c] - mu[c], s);
        const double gij = ps[i] * ps[j] * s;
        Gm[i * gp + j] = gij;
        Gm[j * gp + i] = gij;
    }
    __syncthreads();
}

// Top-k set of the row as a bit mask: rank by (logit desc, index asc).  When
// idx is given, idx[rank] = key for the k best.  `scratch` holds blockDim.x
// 64-bit words.
__device__ inline uint64_t topk_mask64(const double *zs, int n, int k, int32_t *idx,
                                       uint64_t *scratch) {
    const int tid = threadIdx.x;
    int rank = n;
    if (tid < n) {
        rank = 0;
        for (int i = 0; i < n; ++i) rank += (zs[i] > zs[tid]) || (zs[i] == zs[tid] && i < tid);
        if (rank < k && idx) idx[rank] = tid;
    }
    scratch[tid] = (tid < n && rank < k) ? (1ull << tid) : 0ull;
    __syncthreads();
    uint64_t m = 0;
    for (int i = 0; i < n; ++i) m |= scratch[i];
    __syncthreads();
    return m;
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

__device__ inline double mass64(uint64_t A, const double *ps) {
    double P = 0.0;
    for (uint64_t m = A; m; m &= m - 1) P += ps[__ffsll((unsigned long long)m) - 1];
    return P;
}

}  // namespace fw
