// Observation-window importance and the per-unit dropped-mass curve
// (Section 4, "ContourKV"; Definition 2.1's least achievable dropped mass as
// a function of the budget).
//
//   r_j      = (1/G) sum_g softmax_j(z_g),  z_gj = scale_h <q_g, k_j> + bias_j
//   curve[k] = sum of all but the k largest r, k = 0..n (curve[n] = 0)
//
// Passes: (1) per key chunk, each window row's local max and local sum of
// exponentials; (2) combine the chunks per row in a fixed order; (3) recompute
// the logits, weights and their window mean; (4) per unit, a stable LSD radix
// sort of the scores (descending, ties by index); (5) a float64 suffix scan.
#include "fw_internal.hpp"

namespace fw {

namespace {
constexpr int kChunk = 512;   // keys per workgroup in the logit passes
constexpr int kRowGrp = 16;   // window rows per LDS tile
constexpr int kSortThreads = 1024;
}  // namespace

// Pass 1 (MODE 0) and pass 3 (MODE 1) share the logit computation: each
// thread owns two keys of the chunk; window rows are processed 16 at a time.
template <typename T, int MODE>
__global__ void __launch_bounds__(256)
window_logits_kernel(const T *__restrict__ q, const T *__restrict__ k, const float *__restrict__ scale,
                     const float *__restrict__ bias, int64_t G, int64_t n, int d, int nchunks,
                     float *__restrict__ part_m, float *__restrict__ part_s,
                     const float *__restrict__ row_m, const float *__restrict__ row_il,
                     float *__restrict__ importance) {
    __shared__ float Qs[kRowGrp][257];
    __shared__ float zt[kRowGrp][kChunk + 1];
    __shared__ float red[256];
    const int tid = threadIdx.x;
    const int64_t h = blockIdx.x / nchunks;
    const int ch = blockIdx.x % nchunks;
    const int64_t j0 = (int64_t)ch * kChunk;
    const T *qh = q + h * G * d;
    const T *kh = k + h * n * d;
    const float sc = scale ? scale[h] : (float)(1.0 / sqrt((double)d));
    float racc[2] = {0.f, 0.f};
    for (int64_t g0 = 0; g0 < G; g0 += kRowGrp) {
        const int gn = (G - g0 < kRowGrp) ? (int)(G - g0) : kRowGrp;
        for (int e = tid; e < kRowGrp * d; e += 256) {
            const int rr = e / d, cc = e % d;
            Qs[rr][cc] = (rr < gn) ? Elem<T>::load(qh, (g0 + rr) * d + cc) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int jl = tid + 256 * u;
            const int64_t j = j0 + jl;
            float acc[kRowGrp];
#pragma unroll
            for (int g = 0; g < kRowGrp; ++g) acc[g] = 0.f;
            if (j < n) {
                for (int c = 0; c < d; ++c) {
                    const float kv = Elem<T>::load(kh, j * d + c);
#pragma unroll
                    for (int g = 0; g < kRowGrp; ++g) acc[g] = fmaf(Qs[g][c], kv, acc[g]);
                }
            }
            const float bj = (bias && j < n) ? bias[j] : 0.f;
#pragma unroll
            for (int g = 0; g < kRowGrp; ++g) {
                const float zz = sc * acc[g] + bj;
                if (MODE == 0) {
                    zt[g][jl] = (j < n && g < gn) ? zz : -INFINITY;
                } else if (j < n && g < gn) {
                    const int64_t row = h * G + g0 + g;
                    racc[u] += expf(zz - row_m[row]) * row_il[row];
                }
            }
        }
        if (MODE == 0) {
            __syncthreads();
            // 16 threads per row: local max, then local sum, over 512 keys
            const int g = tid / 16, l = tid % 16;
            float m = -INFINITY;
            for (int jl = l; jl < kChunk; jl += 16) m = fmaxf(m, zt[g][jl]);
            red[tid] = m;
            __syncthreads();
            m = red[g * 16];
            for (int t = 1; t < 16; ++t) m = fmaxf(m, red[g * 16 + t]);
            __syncthreads();
            float s = 0.f;
            for (int jl = l; jl < kChunk; jl += 16) s += (zt[g][jl] == -INFINITY) ? 0.f : expf(zt[g][jl] - m);
            red[tid] = s;
            __syncthreads();
            if (l == 0 && g < gn) {
                float st = 0.f;
                for (int t = 0; t < 16; ++t) st += red[g * 16 + t];
                const int64_t row = h * G + g0 + g;
                part_m[row * nchunks + ch] = m;
                part_s[row * nchunks + ch] = st;
            }
        }
        __syncthreads();
    }
    if (MODE == 1) {
        const float invG = 1.0f / (float)G;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int64_t j = j0 + tid + 256 * u;
            if (j < n) importance[h * n + j] = racc[u] * invG;
        }
    }
}

// Pass 2: combine the per-chunk statistics of every window row.
__global__ void window_combine_kernel(int64_t rows, int nchunks, const float *part_m,
                                      const float *part_s, float *row_m, float *row_il) {
    const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (row >= rows) return;
    float m = -INFINITY;
    for (int c = 0; c < nchunks; ++c) m = fmaxf(m, part_m[row * nchunks + c]);
    double s = 0.0;
    for (int c = 0; c < nchunks; ++c) {
        const float pm = part_m[row * nchunks + c];
        if (pm != -INFINITY) s += (double)part_s[row * nchunks + c] * exp((double)pm - (double)m);
    }
    row_m[row] = m;
    row_il[row] = (float)(1.0 / s);
}

// Pass 4: stable LSD radix sort of one unit's scores, descending (keys are
// the complement of the order-preserving bits), payload = key index (only
// when the order is asked for: a separate instance, whose payload registers
// and LDS traffic are gone).  One workgroup per unit; four 8-bit passes.
// The digit histograms of all four passes come from one read.  Each pass
// takes tiles of kSortTile keys, 8 per thread in index order (wave, slot,
// lane): a key's rank among the equal digits of its wave comes from ballots
// slot by slot with running per-wave counters, the tile is placed
// digit-ordered in LDS, and then written out as contiguous runs (coalesced)
// at the digit's running global offset.  (Longer tiles, 12 or 16 keys per
// thread, run out of registers at 16 waves per workgroup.)
constexpr int kSortWaves = kSortThreads / 64;
constexpr int kSortE = 8;
constexpr int kSortTile = kSortThreads * kSortE;
template <bool with_vals>
__global__ void __launch_bounds__(kSortThreads)
unit_sort_kernel(const float *__restrict__ importance, int64_t n, uint32_t *keys_a, uint32_t *keys_b,
                 int32_t *vals_a, int32_t *vals_b) {
    __shared__ int gb[4][256];             // per pass: running global offset of each digit
    __shared__ int wc[kSortWaves][256];    // per wave: digit counts, then their cross-wave prefix
    __shared__ int tdp[256], ttot[256];    // tile: digit prefix, digit totals
    __shared__ uint32_t stk[kSortTile];
    __shared__ int32_t stv[with_vals ? kSortTile : 1];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t h = blockIdx.x;
    const float *imp = importance + h * n;
    uint32_t *ka = keys_a + h * n, *kb = keys_b + h * n;
    int32_t *va = vals_a + h * n, *vb = vals_b + h * n;
    const uint64_t below_mask = (1ull << lane) - 1ull;
    for (int i = tid; i < 4 * 256; i += kSortThreads) (&gb[0][0])[i] = 0;
    __syncthreads();
    // (scores of a unit often share their top bytes: a digit common to every
    // live lane of the wave is added once)
    for (int64_t j0 = (int64_t)wv * 64; j0 < n; j0 += kSortThreads) {
        const int64_t j = j0 + lane;
        const bool live = j < n;
        const uint32_t key = live ? ~ord_key(imp[j]) : 0u;
        const uint64_t lv = __ballot(live);
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint32_t d = (key >> (8 * p)) & 255u;
            const uint32_t d0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)d);
            if (__ballot(live && d == d0) == lv) {
                if (lane == 0) atomicAdd(&gb[p][d0], __popcll(lv));
            } else if (live) {
                atomicAdd(&gb[p][d], 1);
            }
        }
    }
    __syncthreads();
    if (wv < 4) {  // exclusive prefix over the digits, one wave per pass
        int v[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) { v[q] = gb[wv][4 * lane + q]; sum += v[q]; }
        int incl = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off);
            if (lane >= off) incl += y;
        }
        int run = incl - sum;
#pragma unroll
        for (int q = 0; q < 4; ++q) { gb[wv][4 * lane + q] = run; run += v[q]; }
    }
    __syncthreads();
    for (int p = 0; p < 4; ++p) {
        const int shift = 8 * p;
        const uint32_t *sk = (p & 1) ? kb : ka;
        const int32_t *sv = (p & 1) ? vb : va;
        uint32_t *dk = (p & 1) ? ka : kb;
        int32_t *dv = (p & 1) ? va : vb;
        // the keys of tile t0 + kSortTile load while tile t0 is ranked and written
        uint32_t nkey[kSortE];
        int32_t nval[kSortE];
        auto load_tile = [&](int64_t t0) {
#pragma unroll
            for (int s = 0; s < kSortE; ++s) {
                const int64_t e = t0 + (int64_t)wv * 64 * kSortE + s * 64 + lane;
                const bool live = e < n;
                if (p == 0) {
                    nkey[s] = live ? ~ord_key(imp[e]) : 0u;
                    nval[s] = (int32_t)e;
                } else {
                    nkey[s] = live ? sk[e] : 0u;
                    nval[s] = (with_vals && live) ? sv[e] : 0;
                }
            }
        };
        load_tile(0);
        for (int64_t t0 = 0; t0 < n; t0 += kSortTile) {
            for (int i = lane; i < 256; i += 64) wc[wv][i] = 0;
            uint32_t key[kSortE];
            int32_t val[kSortE];
            int lr[kSortE];
            // the slot's digit (256: past the end), recomputed where used
            const int64_t ebase = t0 + (int64_t)wv * 64 * kSortE + lane;
            auto digit = [&](int s) -> int {
                return (ebase + s * 64 < n) ? (int)((key[s] >> shift) & 255u) : 256;
            };
#pragma unroll
            for (int s = 0; s < kSortE; ++s) {
                key[s] = nkey[s];
                val[s] = nval[s];
            }
            if (t0 + kSortTile < n) load_tile(t0 + kSortTile);
#pragma unroll
            for (int s = 0; s < kSortE; ++s) {
                // lanes of this wave holding the same digit in this slot
                const int dg = digit(s);
                uint64_t same = __ballot(dg < 256);
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                    const uint64_t bal = __ballot((dg >> b) & 1);
                    same &= ((dg >> b) & 1) ? bal : ~bal;
                }
                const int below = __popcll(same & below_mask);
                int pre = 0;
                if (dg < 256) pre = wc[wv][dg];
                lr[s] = pre + below;
                if (dg < 256 && below == 0) wc[wv][dg] = pre + __popcll(same);
            }
            lds_barrier();
            if (tid < 256) {
                int c[kSortWaves];
#pragma unroll
                for (int w = 0; w < kSortWaves; ++w) c[w] = wc[w][tid];
                int run = 0;
#pragma unroll
                for (int w = 0; w < kSortWaves; ++w) { wc[w][tid] = run; run += c[w]; }
                ttot[tid] = run;
            }
            lds_barrier();
            if (wv == 0) {
                int v[4], sum = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) { v[q] = ttot[4 * lane + q]; sum += v[q]; }
                int incl = sum;
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const int y = __shfl_up(incl, off);
                    if (lane >= off) incl += y;
                }
                int run = incl - sum;
#pragma unroll
                for (int q = 0; q < 4; ++q) { tdp[4 * lane + q] = run; run += v[q]; }
            }
            lds_barrier();
#pragma unroll
            for (int s = 0; s < kSortE; ++s) {
                const int dg = digit(s);
                if (dg < 256) {
                    const int lp = tdp[dg] + wc[wv][dg] + lr[s];
                    stk[lp] = key[s];
                    if (with_vals) stv[lp] = val[s];
                }
            }
            lds_barrier();
            const int cnt = (int)((n - t0 < kSortTile) ? n - t0 : kSortTile);
            for (int i = tid; i < cnt; i += kSortThreads) {
                const uint32_t kk = stk[i];
                const int d = (int)((kk >> shift) & 255u);
                const int64_t gp = (int64_t)gb[p][d] + (i - tdp[d]);
                dk[gp] = kk;
                if (with_vals) dv[gp] = stv[i];
            }
            lds_barrier();
            if (tid < 256) gb[p][tid] += ttot[tid];
            lds_barrier();
        }
        __syncthreads();  // this pass's global writes are the next pass's input
    }
    // four passes: the result is back in keys_a / vals_a
}

// Pass 5: curve[k] = sum_{i >= k} sorted[i] (float64) read from the sorted
// keys themselves, and the order.  Tiles of 8192 positions from the end: a
// coalesced load into LDS, per-thread sums of 8 consecutive positions, a
// suffix scan of the thread sums (wave shuffles, then across waves), and a
// coalesced store.
constexpr int kCurveTile = 8 * kSortThreads;
__global__ void __launch_bounds__(kSortThreads)
unit_curve_kernel(const uint32_t *__restrict__ keys, int64_t n, const int32_t *__restrict__ vals,
                  float *__restrict__ curve, int32_t *__restrict__ order) {
    __shared__ float tile[kCurveTile];
    __shared__ double wsum[kSortThreads / 64];
    __shared__ double carry_s;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t h = blockIdx.x;
    const uint32_t *kh = keys + h * n;
    float *ch = curve + h * (n + 1);
    if (tid == 0) carry_s = 0.0;
    for (int64_t t0 = ((n - 1) / kCurveTile) * kCurveTile; t0 >= 0; t0 -= kCurveTile) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t e = t0 + i * kSortThreads + tid;
            tile[i * kSortThreads + tid] = e < n ? key_to_float(~kh[e]) : 0.f;
        }
        __syncthreads();
        double part = 0.0;
#pragma unroll
        for (int q = 0; q < 8; ++q) part += (double)tile[8 * tid + q];
        // inclusive suffix sum over the lanes of this wave
        double suf = part;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const double y = __shfl_down(suf, off);
            if (lane + off < 64) suf += y;
        }
        if (lane == 0) wsum[wv] = suf;  // the wave's total
        __syncthreads();
        double after = carry_s;  // everything right of this wave
        for (int w2 = wv + 1; w2 < kSortThreads / 64; ++w2) after += wsum[w2];
        double acc = after + (suf - part);  // right of this thread's 8 positions
#pragma unroll
        for (int q = 7; q >= 0; --q) {
            acc += (double)tile[8 * tid + q];
            tile[8 * tid + q] = (float)acc;
        }
        __syncthreads();
        if (tid == 0) {
            double tot = 0.0;
            for (int w2 = 0; w2 < kSortThreads / 64; ++w2) tot += wsum[w2];
            carry_s += tot;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t e = t0 + i * kSortThreads + tid;
            if (e < n) {
                ch[e] = tile[i * kSortThreads + tid];
                if (order) order[h * n + e] = vals[h * n + e];
            }
        }
        __syncthreads();
    }
    if (tid == 0) ch[n] = 0.f;
}

// ---------------------------------------------------------------------------
namespace {
struct CurveLayout {
    float *part_m, *part_s, *row_m, *row_il;
    uint32_t *ka, *kb;
    int32_t *va, *vb;
    size_t bytes;
};

CurveLayout curve_layout(const fw_rows &rows, void *ws) {
    const size_t H = rows.H, G = rows.G, n = rows.n;
    const size_t nch = (n + kChunk - 1) / kChunk;
    CurveLayout L{};
    size_t off = 0;
    char *base = (char *)ws;
    auto take = [&](size_t bytes) -> void * {
        off = align_up(off, 256);
        void *p = base ? base + off : nullptr;
        off += bytes;
        return p;
    };
    L.part_m = (float *)take(H * G * nch * 4);
    L.part_s = (float *)take(H * G * nch * 4);
    L.row_m = (float *)take(H * G * 4);
    L.row_il = (float *)take(H * G * 4);
    L.ka = (uint32_t *)take(H * n * 4);
    L.kb = (uint32_t *)take(H * n * 4);
    L.va = (int32_t *)take(H * n * 4);
    L.vb = (int32_t *)take(H * n * 4);
    L.bytes = align_up(off, 256);
    return L;
}
}  // namespace

size_t curve_ws_bytes(const fw_rows &rows) { return curve_layout(rows, nullptr).bytes; }

template <typename T>
static hipError_t curve_impl(const fw_rows &rows, float *importance, float *curve, int32_t *order,
                             void *ws, hipStream_t st) {
    CurveLayout L = curve_layout(rows, ws);
    const int64_t H = rows.H, G = rows.G, n = rows.n;
    const int d = (int)rows.d;
    const int nch = (int)((n + kChunk - 1) / kChunk);
    const dim3 grid((unsigned)(H * nch));
    const T *q = (const T *)rows.q, *k = (const T *)rows.k;
    if (window_mfma_supported(rows)) {
        // bf16, d = 128, up to 64 window rows: MFMA scores (k_window.hip)
        launch_window_mfma(rows, L.part_m, L.part_s, L.row_m, L.row_il, importance, st);
    } else {
        hipLaunchKernelGGL((window_logits_kernel<T, 0>), grid, dim3(256), 0, st, q, k, rows.scale,
                           rows.bias, G, n, d, nch, L.part_m, L.part_s, nullptr, nullptr, nullptr);
        hipLaunchKernelGGL(window_combine_kernel, dim3((unsigned)((H * G + 255) / 256)), dim3(256), 0, st,
                           H * G, nch, L.part_m, L.part_s, L.row_m, L.row_il);
        hipLaunchKernelGGL((window_logits_kernel<T, 1>), grid, dim3(256), 0, st, q, k, rows.scale,
                           rows.bias, G, n, d, nch, nullptr, nullptr, L.row_m, L.row_il, importance);
    }
    if (order)
        hipLaunchKernelGGL((unit_sort_kernel<true>), dim3((unsigned)H), dim3(kSortThreads), 0, st,
                           importance, n, L.ka, L.kb, L.va, L.vb);
    else
        hipLaunchKernelGGL((unit_sort_kernel<false>), dim3((unsigned)H), dim3(kSortThreads), 0, st,
                           importance, n, L.ka, L.kb, L.va, L.vb);
    hipLaunchKernelGGL(unit_curve_kernel, dim3((unsigned)H), dim3(kSortThreads), 0, st,
                       (const uint32_t *)L.ka, n, (const int32_t *)L.va, curve, order);
    return hipGetLastError();
}

hipError_t launch_curve(const fw_rows &rows, float *importance, float *curve, int32_t *order,
                        void *ws, hipStream_t st) {
    if (rows.dtype == FW_BF16) return curve_impl<uint16_t>(rows, importance, curve, order, ws, st);
    return curve_impl<float>(rows, importance, curve, order, ws, st);
}

}  // namespace fw
