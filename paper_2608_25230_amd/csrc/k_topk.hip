// Top-k forced-weight evaluation of attention rows (Definition 2.1; gap via
// the first form of Lemma 2.2).
//
// Three passes:
//   scores  z[r][j] = scale_h * <q_r, k_j> + bias_j        (fp32 accumulate)
//   select  per row: max m, sum l of exp(z - m), and for every budget the
//           exact k-th largest logit (radix select on order-preserving keys,
//           ties by index), optionally the top-kmax indices in rank order
//   tiers   per row: disjoint tier sums T_t = sum p_j v_j, M_t = sum p_j over
//           ranks [0,k_0), [k_0,k_1), ..., [k_last, n), then o, o_S, the gap
//           (1 - p(S)) * ||m_{S^c} - m_S|| and the dropped mass.
#include "fw_internal.hpp"
#include "select.hpp"

namespace fw {

// ---------------------------------------------------------------------------
// scores: tiles of 32 rows x 64 keys, d in chunks of 32 staged through LDS
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256)
scores_kernel(const T *__restrict__ q, const T *__restrict__ k, const float *__restrict__ scale,
              const float *__restrict__ bias, int64_t H, int64_t G, int64_t n, int d,
              float *__restrict__ z) {
    constexpr int TR = 32, TK = 64, TD = 32;
    __shared__ float Qs[TR][TD + 1];
    __shared__ float Ks[TK][TD + 1];
    const int64_t row_tiles = (G + TR - 1) / TR;
    const int64_t key_tiles = (n + TK - 1) / TK;
    int64_t b = blockIdx.x;
    const int64_t kt = b % key_tiles;
    b /= key_tiles;
    const int64_t rt = b % row_tiles;
    const int64_t h = b / row_tiles;
    if (h >= H) return;
    const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
    const int64_t g0 = rt * TR, j0 = kt * TK;
    const T *qh = q + (h * G) * (int64_t)d;
    const T *kh = k + (h * n) * (int64_t)d;
    float acc[2][4] = {};
    for (int c0 = 0; c0 < d; c0 += TD) {
        for (int e = tid; e < TR * TD; e += 256) {
            int rr = e / TD, cc = e % TD;
            int64_t g = g0 + rr;
            Qs[rr][cc] = (g < G && c0 + cc < d) ? Elem<T>::load(qh, g * d + c0 + cc) : 0.f;
        }
        for (int e = tid; e < TK * TD; e += 256) {
            int kk = e / TD, cc = e % TD;
            int64_t j = j0 + kk;
            Ks[kk][cc] = (j < n && c0 + cc < d) ? Elem<T>::load(kh, j * d + c0 + cc) : 0.f;
        }
        __syncthreads();
#pragma unroll 8
        for (int cc = 0; cc < TD; ++cc) {
            float a0 = Qs[ty * 2][cc], a1 = Qs[ty * 2 + 1][cc];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float kv = Ks[tx + 16 * i][cc];
                acc[0][i] = fmaf(a0, kv, acc[0][i]);
                acc[1][i] = fmaf(a1, kv, acc[1][i]);
            }
        }
        __syncthreads();
    }
    const float sc = scale ? scale[h] : (float)(1.0 / sqrt((double)d));
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        int64_t g = g0 + ty * 2 + a;
        if (g >= G) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            int64_t j = j0 + tx + 16 * i;
            if (j >= n) continue;
            float v = sc * acc[a][i];
            if (bias) v += bias[j];
            z[(h * G + g) * n + j] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// select: one workgroup per row
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
select_kernel(const float *__restrict__ z, int64_t R, int64_t n, KsArg ks, float *__restrict__ row_m,
              float *__restrict__ row_l, uint32_t *__restrict__ thr_key, int32_t *__restrict__ thr_cut,
              int32_t *__restrict__ topk_idx, int kmax, int sort_len) {
    extern __shared__ unsigned long long sortbuf[];
    __shared__ int hist[256];
    __shared__ int scan[256];
    __shared__ int sh[4];
    __shared__ float redf[256];
    const int64_t r = blockIdx.x;
    if (r >= R) return;
    const int tid = threadIdx.x, nt = blockDim.x;
    const float *zr = z + r * n;

    float m = -INFINITY;
    for (int64_t j = tid; j < n; j += nt) m = fmaxf(m, zr[j]);
    m = block_reduce(m, redf, OpMax());
    float s = 0.f;
    for (int64_t j = tid; j < n; j += nt) s += expf(zr[j] - m);
    s = block_reduce(s, redf, OpSum());
    if (tid == 0) { row_m[r] = m; row_l[r] = s; }

    uint32_t kmax_key = 0;
    int64_t kmax_cut = 0;
    for (int t = 0; t < ks.n; ++t) {
        uint32_t key;
        int rem;
        radix_select_desc(zr, n, ks.k[t], hist, sh, &key, &rem);
        int64_t cut = nth_tie(zr, n, key, rem, scan, sh);
        if (tid == 0) {
            thr_key[r * ks.n + t] = key;
            thr_cut[r * ks.n + t] = (int32_t)cut;
        }
        if (ks.k[t] == kmax) { kmax_key = key; kmax_cut = cut; }
    }
    if (topk_idx == nullptr) return;

    // gather the top-kmax as 64-bit sort keys, then bitonic sort descending
    for (int i = tid; i < sort_len; i += nt) sortbuf[i] = 0ull;
    __syncthreads();
    const int64_t chunk = (n + nt - 1) / nt;
    const int64_t lo = tid * chunk, hi = (lo + chunk < n) ? lo + chunk : n;
    int c = 0;
    for (int64_t j = lo; j < hi; ++j) {
        uint32_t u = ord_key(zr[j]);
        c += (u > kmax_key) || (u == kmax_key && j <= kmax_cut);
    }
    int total;
    int pos = block_exclusive_scan(c, scan, &total);
    for (int64_t j = lo; j < hi; ++j) {
        uint32_t u = ord_key(zr[j]);
        if ((u > kmax_key) || (u == kmax_key && j <= kmax_cut))
            sortbuf[pos++] = ((unsigned long long)u << 32) | (0xFFFFFFFFu - (uint32_t)j);
    }
    __syncthreads();
    for (int size = 2; size <= sort_len; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < sort_len / 2; i += nt) {
                int lo2 = 2 * stride * (i / stride) + (i % stride);
                int hi2 = lo2 + stride;
                bool desc = (lo2 & size) == 0;
                unsigned long long a = sortbuf[lo2], bb = sortbuf[hi2];
                if (desc ? (a < bb) : (a > bb)) { sortbuf[lo2] = bb; sortbuf[hi2] = a; }
            }
            __syncthreads();
        }
    }
    for (int i = tid; i < kmax; i += nt)
        topk_idx[r * kmax + i] = (int32_t)(0xFFFFFFFFu - (uint32_t)(sortbuf[i] & 0xFFFFFFFFull));
}

// ---------------------------------------------------------------------------
// tiers: one wave per row, 4 rows per workgroup; lane owns columns lane+64*c
// ---------------------------------------------------------------------------
template <typename T, int NC, int NT>
__global__ void __launch_bounds__(256)
tiers_kernel(const T *__restrict__ v, const float *__restrict__ z, const float *__restrict__ row_m,
             const float *__restrict__ row_l, const uint32_t *__restrict__ thr_key,
             const int32_t *__restrict__ thr_cut, int64_t H, int64_t G, int64_t n, int d, KsArg ks,
             float *__restrict__ o, float *__restrict__ o_s, float *__restrict__ gap,
             float *__restrict__ dropped) {
    constexpr int RPB = 4, TK = 64;
    __shared__ float p_s[RPB][TK];
    __shared__ int tier_s[RPB][TK];
    const int64_t row_tiles = (G + RPB - 1) / RPB;
    const int64_t h = blockIdx.x / row_tiles;
    const int64_t g = (blockIdx.x % row_tiles) * RPB + threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave, wr = threadIdx.x / kWave;
    const bool live = (h < H) && (g < G);
    const int64_t r = h * G + g;
    const int nk = ks.n;
    uint32_t key[NT > 1 ? NT - 1 : 1];
    int64_t cut[NT > 1 ? NT - 1 : 1];
    float m = 0.f, inv_l = 0.f;
    if (live) {
        m = row_m[r];
        inv_l = 1.0f / row_l[r];
#pragma unroll
        for (int t = 0; t < NT - 1; ++t) {
            key[t] = thr_key[r * nk + t];
            cut[t] = thr_cut[r * nk + t];
        }
    }
    float acc[NT][NC];
    float mass[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        mass[t] = 0.f;
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[t][c] = 0.f;
    }
    const T *vh = v + h * n * (int64_t)d;
    for (int64_t j0 = 0; j0 < n; j0 += TK) {
        {
            int64_t j = j0 + lane;
            float p = 0.f;
            int tier = NT - 1;
            if (live && j < n) {
                float zz = z[r * n + j];
                p = expf(zz - m) * inv_l;
                uint32_t u = ord_key(zz);
#pragma unroll
                for (int t = NT - 2; t >= 0; --t)
                    if (u > key[t] || (u == key[t] && j <= cut[t])) tier = t;
            }
            p_s[wr][lane] = p;
            tier_s[wr][lane] = tier;
        }
        __syncthreads();
        const int jn = (n - j0 < TK) ? (int)(n - j0) : TK;
        if (live) {
            for (int jj = 0; jj < jn; ++jj) {
                const float p = p_s[wr][jj];
                const int tier = tier_s[wr][jj];  // uniform across the wave
                float vv[NC];
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    int col = lane + kWave * c;
                    vv[c] = (col < d) ? Elem<T>::load(vh, (j0 + jj) * d + col) : 0.f;
                }
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    if (tier == t) {
                        mass[t] += p;
#pragma unroll
                        for (int c = 0; c < NC; ++c) acc[t][c] = fmaf(p, vv[c], acc[t][c]);
                    }
                }
            }
        }
        __syncthreads();
    }
    if (!live) return;
    // epilogue
    float mtot = 0.f;
#pragma unroll
    for (int t = 0; t < NT; ++t) mtot += mass[t];
    const float inv_tot = 1.0f / mtot;
    if (o) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            int col = lane + kWave * c;
            if (col >= d) continue;
            float s = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) s += acc[t][c];
            o[r * d + col] = s * inv_tot;
        }
    }
    const int64_t R = H * G;
#pragma unroll
    for (int t = 0; t < NT - 1; ++t) {
        float km = 0.f, rm = 0.f;
#pragma unroll
        for (int u = 0; u < NT; ++u) {
            if (u <= t) km += mass[u]; else rm += mass[u];
        }
        float ss = 0.f;
        float oS[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            float kt = 0.f, rt = 0.f;
#pragma unroll
            for (int u = 0; u < NT; ++u) {
                if (u <= t) kt += acc[u][c]; else rt += acc[u][c];
            }
            oS[c] = kt / km;
            int col = lane + kWave * c;
            if (rm > 0.f && col < d) {
                float diff = rt / rm - oS[c];
                ss = fmaf(diff, diff, ss);
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
        const int out = ks.perm[t];
        if (o_s) {
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                int col = lane + kWave * c;
                if (col < d) o_s[((int64_t)out * R + r) * d + col] = oS[c];
            }
        }
        if (lane == 0) {
            gap[(int64_t)out * R + r] = (rm > 0.f) ? (rm * inv_tot) * sqrtf(ss) : 0.f;
            dropped[(int64_t)out * R + r] = rm * inv_tot;
        }
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_scores(int dtype, const void *q, const void *k, const float *scale,
                         const float *bias, int64_t H, int64_t G, int64_t n, int d, float *z,
                         hipStream_t st) {
    const int64_t blocks = H * ((G + 31) / 32) * ((n + 63) / 64);
    if (dtype == FW_BF16)
        hipLaunchKernelGGL(scores_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, st,
                           (const uint16_t *)q, (const uint16_t *)k, scale, bias, H, G, n, d, z);
    else
        hipLaunchKernelGGL(scores_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st,
                           (const float *)q, (const float *)k, scale, bias, H, G, n, d, z);
    return hipGetLastError();
}

hipError_t launch_select(const float *z, int64_t R, int64_t n, const KsArg &ks, float *row_m,
                         float *row_l, uint32_t *thr_key, int32_t *thr_cut, int32_t *topk_idx,
                         int kmax, hipStream_t st) {
    int sort_len = 1;
    while (sort_len < kmax) sort_len <<= 1;
    const size_t lds = topk_idx ? (size_t)sort_len * sizeof(unsigned long long) : 0;
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)R), dim3(256), lds, st, z, R, n, ks, row_m,
                       row_l, thr_key, thr_cut, topk_idx, kmax, sort_len);
    return hipGetLastError();
}

template <typename T, int NC>
static void tiers_nt(int nt, dim3 grid, hipStream_t st, const T *v, const float *z,
                     const float *row_m, const float *row_l, const uint32_t *thr_key,
                     const int32_t *thr_cut, int64_t H, int64_t G, int64_t n, int d,
                     const KsArg &ks, float *o, float *o_s, float *gap, float *dropped) {
#define FW_TIERS_CASE(NTV)                                                                        \
    case NTV:                                                                                     \
        hipLaunchKernelGGL((tiers_kernel<T, NC, NTV>), grid, dim3(256), 0, st, v, z, row_m, row_l, \
                           thr_key, thr_cut, H, G, n, d, ks, o, o_s, gap, dropped);               \
        break;
    switch (nt) {
        FW_TIERS_CASE(2) FW_TIERS_CASE(3) FW_TIERS_CASE(4) FW_TIERS_CASE(5)
        FW_TIERS_CASE(6) FW_TIERS_CASE(7) FW_TIERS_CASE(8) FW_TIERS_CASE(9)
        default: break;
    }
#undef FW_TIERS_CASE
}

template <typename T>
static void tiers_nc(int nc, int nt, dim3 grid, hipStream_t st, const T *v, const float *z,
                     const float *row_m, const float *row_l, const uint32_t *thr_key,
                     const int32_t *thr_cut, int64_t H, int64_t G, int64_t n, int d,
                     const KsArg &ks, float *o, float *o_s, float *gap, float *dropped) {
    switch (nc) {
        case 1: tiers_nt<T, 1>(nt, grid, st, v, z, row_m, row_l, thr_key, thr_cut, H, G, n, d, ks, o, o_s, gap, dropped); break;
        case 2: tiers_nt<T, 2>(nt, grid, st, v, z, row_m, row_l, thr_key, thr_cut, H, G, n, d, ks, o, o_s, gap, dropped); break;
        case 3: tiers_nt<T, 3>(nt, grid, st, v, z, row_m, row_l, thr_key, thr_cut, H, G, n, d, ks, o, o_s, gap, dropped); break;
        default: tiers_nt<T, 4>(nt, grid, st, v, z, row_m, row_l, thr_key, thr_cut, H, G, n, d, ks, o, o_s, gap, dropped); break;
    }
}

hipError_t launch_tiers(int dtype, const void *v, const float *z, const float *row_m,
                        const float *row_l, const uint32_t *thr_key, const int32_t *thr_cut,
                        int64_t H, int64_t G, int64_t n, int d, const KsArg &ks, float *o,
                        float *o_s, float *gap, float *dropped, hipStream_t st) {
    const int nc = (d + kWave - 1) / kWave;
    const int nt = ks.n + 1;
    dim3 grid((unsigned)(H * ((G + 3) / 4)));
    if (dtype == FW_BF16)
        tiers_nc<uint16_t>(nc, nt, grid, st, (const uint16_t *)v, z, row_m, row_l, thr_key, thr_cut,
                           H, G, n, d, ks, o, o_s, gap, dropped);
    else
        tiers_nc<float>(nc, nt, grid, st, (const float *)v, z, row_m, row_l, thr_key, thr_cut, H, G,
                        n, d, ks, o, o_s, gap, dropped);
    return hipGetLastError();
}

}  // namespace fw
