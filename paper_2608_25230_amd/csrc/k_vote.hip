// Group vote (Section 2.1: deployment fixes one kept set per key/value head
// and applies it to the group of query rows that share the head), float64.
//
// One workgroup per group (the rows of all query heads of a unit at one
// position).  For each member row in turn: logits over the unit's keys,
// softmax, the row's own top-mass set (logit desc, index asc), its weights
// added into the group's summed mass, the dense output, and the error of its
// own top-mass set.  Then the vote: the s keys of largest summed mass (index
// asc on ties).  Finally each member's forced-weight error with the vote's
// set and the vote's dropped mass, from the vote keys' logits recomputed with
// the row's own maximum and normaliser.
#include "fw_internal.hpp"
#include "instance64.hpp"
#include "rowpass.hpp"

namespace fw {

namespace {

constexpr int VT = 256;  // threads per group workgroup

struct VoteLds {
    size_t xq, red, own, vote, rowsc, mu, zz, score, total;
};

__host__ __device__ inline VoteLds vote_lds(int64_t N, int d, int gs, int s) {
    VoteLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.xq = take((size_t)d * 8);
    L.red = take((size_t)VT * 16);
    L.own = take((size_t)s * 4);
    L.vote = take((size_t)s * 4);
    L.rowsc = take((size_t)gs * 2 * 8);  // per member: max logit, normaliser
    L.mu = take((size_t)gs * d * 8);     // per member: dense output
    L.zz = take((size_t)N * 8);
    L.score = take((size_t)N * 8);
    L.total = o;
    return L;
}

struct VoteArgs {
    const void *q, *k, *v;
    const float *scale, *bias;
    int64_t H, G, N;
    int d, s, gs;
    int32_t *vote_idx;
    float *es_vote, *es_top, *dropped;
};

// es(A) = ||sum_{i in A} p_i (v_i - mu)|| / p(A) for a list of keys with
// their masses (d-dimensional sums, one column per thread).
template <typename T>
__device__ double es_list(const T *vh, int d, const int *keys, const double *pk, int s, const double *mu,
                          double *red) {
    double g2 = 0.0;
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
        double g = 0.0;
        for (int i = 0; i < s; ++i) g = fma(pk[i], (double)Elem<T>::load(vh, (int64_t)keys[i] * d + c) - mu[c], g);
        g2 = fma(g, g, g2);
    }
    g2 = block_reduce(g2, red, OpSum());
    double pm = 0.0;
    for (int i = 0; i < s; ++i) pm += pk[i];
    return sqrt(g2) / pm;
}

}  // namespace

template <typename T>
__global__ void __launch_bounds__(VT) vote_group_kernel(VoteArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, NT = blockDim.x;
    const int64_t N = a.N;
    const int d = a.d, s = a.s, gs = a.gs;
    const VoteLds L = vote_lds(N, d, gs, s);
    double *xq = (double *)(smem + L.xq);
    double *redd = (double *)(smem + L.red);
    int64_t *redi = (int64_t *)(redd + NT);
    int *own = (int *)(smem + L.own);
    int *vote = (int *)(smem + L.vote);
    double *rowsc = (double *)(smem + L.rowsc);
    double *mus = (double *)(smem + L.mu);
    double *zz = (double *)(smem + L.zz);
    double *score = (double *)(smem + L.score);
    double *pk = redd + NT;  // the vote keys' masses ([s] <= NT doubles, after the row loop)

    const int64_t T_ = a.G / gs;  // positions per unit
    const int64_t bl = xcd_order(blockIdx.x, gridDim.x);  // a unit's groups on one XCD
    const int64_t h = bl / T_, t = bl % T_;
    const T *kh = (const T *)a.k + h * N * d;
    const T *vh = (const T *)a.v + h * N * d;
    const double scale = a.scale ? (double)a.scale[h] : (double)default_scale(d);
    for (int64_t j = tid; j < N; j += NT) score[j] = 0.0;

    for (int m = 0; m < gs; ++m) {
        const int64_t r = h * a.G + (int64_t)m * T_ + t;  // query head m, position t
        const T *qr = (const T *)a.q + r * d;
        double *mu = mus + (size_t)m * d;
        for (int c = tid; c < d; c += NT) xq[c] = (double)Elem<T>::load(qr, c);
        __syncthreads();
        double xr[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) xr[i] = 0.0;
        lane_columns<T>(d, [&](int c, int slot) { xr[slot] = xq[c]; });
        for_keys(kh, N, d, [&](int64_t j, int gi, int GL, auto &&walk) {
            double acc = 0.0;
            walk([&](int, int slot, float x) { acc = fma(xr[slot], (double)x, acc); });
            acc = group_sum(acc, GL);
            if (j >= 0 && gi == 0) zz[j] = scale * acc + (a.bias ? (double)a.bias[j] : 0.0);
        });
        __syncthreads();
        double zmax = -INFINITY;
        for (int64_t j = tid; j < N; j += NT) zmax = fmax(zmax, zz[j]);
        zmax = block_reduce(zmax, redd, OpMax());
        // the row's own top-mass set
        {
            double pv = INFINITY;
            int64_t pi = -1;
            for (int u = 0; u < s; ++u) {
                double bv = 0.0;
                int64_t bi = -1;
                for (int64_t j = tid; j < N; j += NT) {
                    const double z = zz[j];
                    const bool after = z < pv || (z == pv && j > pi);
                    if (after && (bi < 0 || z > bv || (z == bv && j < bi))) { bv = z; bi = j; }
                }
                block_argmax(bv, bi, redd, redi);
                if (tid == 0) own[u] = bi >= 0 ? (int)bi : 0;  // s <= n: a key is always found
                pv = bv;
                pi = bi;
            }
        }
        double lsum = 0.0;
        for (int64_t j = tid; j < N; j += NT) lsum += exp(zz[j] - zmax);
        lsum = block_reduce(lsum, redd, OpSum());
        // weights in place of the logits; the group's summed mass
        for (int64_t j = tid; j < N; j += NT) {
            const double p = exp(zz[j] - zmax) / lsum;
            zz[j] = p;
            score[j] += p;
        }
        if (tid == 0) {
            rowsc[2 * m] = zmax;
            rowsc[2 * m + 1] = lsum;
        }
        __syncthreads();
        // dense output: each lane accumulates its columns over the keys it visits
        {
            constexpr int VEC = RowVec<T>::VEC;
            double part[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) part[i] = 0.0;
            const bool vec = d % VEC == 0;
            const int GL = vec ? group_lanes(d, VEC) : 64;
            for_keys(vh, N, d, [&](int64_t j, int, int, auto &&walk) {
                if (j < 0) return;
                const double p = zz[j];
                walk([&](int, int slot, float x) { part[slot] = fma(p, (double)x, part[slot]); });
            });
            for (int c = tid; c < d; c += NT) mu[c] = 0.0;
            __syncthreads();
            const int lane = tid & 63, gi = vec ? lane % GL : lane;
            for (int rnd = 0; rnd < NT / 64 * (64 / GL); ++rnd) {
                if ((tid >> 6) * (64 / GL) + lane / GL == rnd) {
                    if (vec) {
#pragma unroll
                        for (int i = 0; i < VEC; ++i) {
                            const int c = gi * VEC + i;
                            if (c < d) mu[c] += part[i];
                        }
                    } else {
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            const int c = gi + 64 * u;
                            if (c < d) mu[c] += part[u];
                        }
                    }
                }
                __syncthreads();
            }
        }
        // the row's own top-mass error (keys with their weights, ascending order
        // is not needed: the sums run over the list)
        {
            double *pown = redd + NT;  // masses of the own keys ([s] <= NT doubles)
            for (int u = tid; u < s; u += NT) pown[u] = zz[own[u]];
            __syncthreads();
            const double es = es_list<T>(vh, d, own, pown, s, mu, redd);
            if (tid == 0) a.es_top[r] = (float)(s >= N ? 0.0 : es);
        }
        __syncthreads();  // zz, own and pown are reused by the next member
    }

    // ---- the vote: s keys of largest summed mass, index asc on ties ---------------
    {
        double pv = INFINITY;
        int64_t pi = -1;
        for (int u = 0; u < s; ++u) {
            double bv = 0.0;
            int64_t bi = -1;
            for (int64_t j = tid; j < N; j += NT) {
                const double x = score[j];
                const bool after = x < pv || (x == pv && j > pi);
                if (after && (bi < 0 || x > bv || (x == bv && j < bi))) { bv = x; bi = j; }
            }
            block_argmax(bv, bi, redd, redi);
            if (tid == 0) {
                vote[u] = bi >= 0 ? (int)bi : 0;
                a.vote_idx[(h * T_ + t) * s + u] = vote[u];
            }
            pv = bv;
            pi = bi;
        }
    }
    __syncthreads();

    // ---- each member under the vote's set -------------------------------------------
    for (int m = 0; m < gs; ++m) {
        const int64_t r = h * a.G + (int64_t)m * T_ + t;
        const T *qr = (const T *)a.q + r * d;
        const double zmax = rowsc[2 * m], lsum = rowsc[2 * m + 1];
        for (int c = tid; c < d; c += NT) xq[c] = (double)Elem<T>::load(qr, c);
        __syncthreads();
        // the vote keys' weights for this row, from their logits recomputed in
        // float64 (summed in column order: rounding-level differences from the
        // row pass's grouped sums) with the row's own maximum and normaliser
        for (int u = tid; u < s; u += NT) {
            const int j = vote[u];
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc = fma(xq[c], (double)Elem<T>::load(kh, (int64_t)j * d + c), acc);
            const double z = scale * acc + (a.bias ? (double)a.bias[j] : 0.0);
            pk[u] = exp(z - zmax) / lsum;
        }
        __syncthreads();
        const double es = es_list<T>(vh, d, vote, pk, s, mus + (size_t)m * d, redd);
        if (tid == 0) {
            double pv = 0.0;
            for (int u = 0; u < s; ++u) pv += pk[u];
            a.es_vote[r] = (float)(s >= N ? 0.0 : es);
            if (a.dropped) a.dropped[r] = (float)(s >= N ? 0.0 : 1.0 - pv);
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
bool vote_supported(const fw_rows &rows, int s, int gs) {
    if (gs < 1 || rows.G % gs != 0 || s < 1 || s > rows.n || s > VT) return false;
    return vote_lds(rows.n, (int)rows.d, gs, s).total <= 160 * 1024;
}

hipError_t launch_vote(const fw_rows &rows, int s, int gs, int32_t *vote_idx, float *es_vote, float *es_top,
                       float *dropped, hipStream_t st) {
    if (!vote_supported(rows, s, gs)) return hipErrorInvalidConfiguration;
    VoteArgs a{};
    a.q = rows.q;
    a.k = rows.k;
    a.v = rows.v;
    a.scale = rows.scale;
    a.bias = rows.bias;
    a.H = rows.H;
    a.G = rows.G;
    a.N = rows.n;
    a.d = (int)rows.d;
    a.s = s;
    a.gs = gs;
    a.vote_idx = vote_idx;
    a.es_vote = es_vote;
    a.es_top = es_top;
    a.dropped = dropped;
    const size_t lds = vote_lds(rows.n, (int)rows.d, gs, s).total;
    const unsigned groups = (unsigned)(rows.H * (rows.G / gs));
    if (rows.dtype == FW_BF16)
        hipLaunchKernelGGL(vote_group_kernel<uint16_t>, dim3(groups), dim3(VT), lds, st, a);
    else
        hipLaunchKernelGGL(vote_group_kernel<float>, dim3(groups), dim3(VT), lds, st, a);
    return hipGetLastError();
}

}  // namespace fw
