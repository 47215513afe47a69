// Observation-window importance on MFMA (Section 4, ContourKV's window score):
//
//   r_j = (1/G) sum_g exp(z_gj - m_g) / l_g,   z_gj = scale_h <q_g, k_j> + bias_j,
//   m_g = max_j z_gj,  l_g = sum_j exp(z_gj - m_g)
//
// for bf16 rows with d = 128 and G = 16 RT window rows (RT = 1..4).  Two
// passes over K: (A) per key chunk, every row's running max and sum of
// exponentials; (B) after the chunks are combined per row, the weights and
// their mean over the window.  All exponentials are base 2 on log2e-scaled
// logits.
//
// A workgroup is 4 waves; wave w takes KW consecutive keys of the chunk and
// all G rows.  The window rows are the MFMA's A operand and stay in
// registers; K streams through a per-wave LDS ring as whole key rows (16-byte
// chunk c of row r stored at chunk position c ^ r), KD - 1 tiles ahead.
// The MFMA result gives lane l key l % 16 of the tile and rows
// 16 rt + 4 (l / 16) + i.
#include "fw_internal.hpp"

namespace fw {

namespace {
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int WW = 4;              // waves per workgroup
constexpr int WTH = 64 * WW;
constexpr int WD = 128;            // head dimension
constexpr int KW = 1024;           // keys per wave
constexpr int WCH = KW * WW;       // keys per workgroup (one chunk)
constexpr int WKD = 4;             // K tiles per ring
constexpr int WRING = WKD * 4096;  // ring bytes per wave
constexpr float WLOG2E = 1.4426950408889634f;
constexpr float WNEG = -1.0e30f;   // running max before any key (finite)

__device__ __forceinline__ rsrc_t wrsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
#define W_LDS(p) ((__attribute__((address_space(3))) void *)(p))
#define W_VM(k) case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
__device__ __forceinline__ void wwait_vm(int n) {
    switch (n) {
        W_VM(0) W_VM(4) W_VM(8) W_VM(12)
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}
#undef W_VM

// (m, l) (+) (m2, l2) in base 2
__device__ __forceinline__ void lse_merge(float &m, float &l, float m2, float l2) {
    const float M = fmaxf(m, m2);
    l = l * __builtin_amdgcn_exp2f(m - M) + l2 * __builtin_amdgcn_exp2f(m2 - M);
    m = M;
}

struct WinArgs {
    const uint16_t *q, *k;
    const float *scale, *bias;
    int64_t H, G, n;
    int nch;                // chunks per unit
    float *part_m, *part_l; // [H][G][nch] (pass A)
    const float *row_m, *row_il;  // [H][G] base-2 max and 1 / sum (pass B)
    float *importance;      // [H][n]
};

// Shared by both passes: the wave's K tiles through the ring, one MFMA group
// per tile, and a per-tile callback on the 16 RT logits of the lane (base-2
// units, key index j, valid flag).
template <int RT, bool BIAS, typename F>
__device__ __forceinline__ void window_stream(const WinArgs &a, int64_t h, int64_t j0w, unsigned char *ring,
                                              const float *bsl, F &&tile_fn) {
    const int lane = threadIdx.x & 63, rl = lane & 15, grp = lane >> 4;
    const float sl2 = (a.scale ? a.scale[h] : (float)(1.0 / sqrt((double)WD))) * WLOG2E;
    // window rows as the A operand: rows 16 rt + l % 16, columns 32 s + 8 (l / 16)
    bf16x8 qa[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int s = 0; s < 4; ++s)
            qa[rt][s] = *(const bf16x8 *)(a.q + ((h * a.G) + 16 * rt + rl) * WD + 32 * s + 8 * grp);
    const rsrc_t kres = wrsrc(a.k + h * a.n * WD, (uint32_t)(a.n * WD * 2));
    uint32_t kvo[4], kro[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int r = 4 * s + grp;
        kvo[s] = ((uint32_t)(j0w + r) * WD + 8 * ((lane & 15) ^ r)) * 2;
        kro[s] = (uint32_t)(rl * 256 + (((4 * s + grp) ^ rl) * 16));
    }
    constexpr int TILES = KW / 16;
    auto issue = [&](int t) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(kres, W_LDS(ring + (t % WKD) * 4096 + s * 1024), 16, kvo[s],
                                                     (uint32_t)(t * 16 * WD * 2), 0, 0);
    };
#pragma unroll
    for (int t = 0; t < WKD - 1; ++t) issue(t);
    for (int t = 0; t < TILES; ++t) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (t + WKD - 1 < TILES) issue(t + WKD - 1);
        const int after = (TILES - 1 - t < WKD - 1) ? TILES - 1 - t : WKD - 1;
        wwait_vm(4 * after);
        const unsigned char *kt = ring + (t % WKD) * 4096;
        bf16x8 kb[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) kb[s] = *(const bf16x8 *)(kt + kro[s]);
        f32x4 acc[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            acc[rt] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 4; ++s)
                acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[rt][s], kb[s], acc[rt], 0, 0, 0);
        }
        const int64_t j = j0w + 16 * t + rl;
        const bool valid = j < a.n;
        const float b2 = BIAS ? bsl[16 * t + rl] * WLOG2E : 0.f;
        float y[RT][4];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) y[rt][i] = fmaf(acc[rt][i], sl2, b2);
        tile_fn(y, j, valid);
    }
}

template <int RT, bool BIAS>
__device__ __forceinline__ const float *load_bias_slice(const WinArgs &a, int64_t j0w, unsigned char *bslice) {
    if (!BIAS) return nullptr;
    const int lane = threadIdx.x & 63;
    const rsrc_t bres = wrsrc(a.bias, (uint32_t)(a.n * 4));
#pragma unroll
    for (int c = 0; c < KW / 64; ++c)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(bres, W_LDS(bslice + 256 * c), 4, (uint32_t)(j0w + lane) * 4,
                                                 (uint32_t)(256 * c), 0, 0);
    return (const float *)bslice;  // complete once the first K tile has landed
}
}  // namespace

// Pass A: per (unit, chunk), every window row's max and sum of exponentials.
template <int RT, bool BIAS>
__global__ void __launch_bounds__(WTH, 2) window_stats_kernel(WinArgs a) {
    extern __shared__ __align__(16) unsigned char wsm[];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, grp = lane >> 4;
    const int64_t h = blockIdx.x / a.nch;
    const int ch = (int)(blockIdx.x % a.nch);
    const int64_t j0w = (int64_t)ch * WCH + (int64_t)w * KW;
    unsigned char *ring = wsm + (size_t)w * WRING;
    float *red = (float *)(wsm + (size_t)WW * WRING);                       // [2][WW][64]
    unsigned char *bslice = wsm + (size_t)WW * WRING + 2 * WW * 64 * 4 + (size_t)w * KW * 4;
    const float *bsl = load_bias_slice<RT, BIAS>(a, j0w, bslice);
    float m[RT][4], l[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) { m[rt][i] = WNEG; l[rt][i] = 0.f; }
    // running (max, sum) with one exponential per logit: exp2(-|y - m|) is the
    // new term when y <= m, and the rescale of the old sum when y > m
    window_stream<RT, BIAS>(a, h, j0w, ring, bsl, [&](float (&y)[RT][4], int64_t, bool valid) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float yy = valid ? y[rt][i] : -INFINITY;
                const float dd = yy - m[rt][i];
                const float e = __builtin_amdgcn_exp2f(-fabsf(dd));
                l[rt][i] = dd > 0.f ? fmaf(l[rt][i], e, 1.f) : l[rt][i] + e;
                m[rt][i] = fmaxf(m[rt][i], yy);
            }
    });
    // combine the 16 lanes of each row group (different keys), then the waves
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                const float m2 = __shfl_xor(m[rt][i], off), l2 = __shfl_xor(l[rt][i], off);
                lse_merge(m[rt][i], l[rt][i], m2, l2);
            }
    if ((lane & 15) == 0) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = 16 * rt + 4 * grp + i;
                red[(0 * WW + w) * 64 + row] = m[rt][i];
                red[(1 * WW + w) * 64 + row] = l[rt][i];
            }
    }
    __syncthreads();
    if (threadIdx.x < 16 * RT) {
        const int row = threadIdx.x;
        float mm = red[row], ll = red[WW * 64 + row];
        for (int ww = 1; ww < WW; ++ww) lse_merge(mm, ll, red[ww * 64 + row], red[(WW + ww) * 64 + row]);
        const int64_t pr = (h * a.G + row) * a.nch + ch;
        a.part_m[pr] = mm;
        a.part_l[pr] = ll;
    }
}

// Combine the chunks of every row (float64, fixed order): base-2 max and
// 1 / sum of exponentials.
__global__ void window_combine2_kernel(int64_t rows, int nch, const float *part_m, const float *part_l,
                                       float *row_m, float *row_il) {
    const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (row >= rows) return;
    float m = WNEG;
    for (int c = 0; c < nch; ++c) m = fmaxf(m, part_m[row * nch + c]);
    double s = 0.0;
    for (int c = 0; c < nch; ++c)
        s += (double)part_l[row * nch + c] * exp2((double)part_m[row * nch + c] - (double)m);
    row_m[row] = m;
    row_il[row] = (float)(1.0 / s);
}

// Pass B: r_j = (1/G) sum_g exp2(y_gj - m_g) / l_g.
template <int RT, bool BIAS>
__global__ void __launch_bounds__(WTH, 2) window_importance_kernel(WinArgs a) {
    extern __shared__ __align__(16) unsigned char wsm[];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, grp = lane >> 4;
    const int64_t h = blockIdx.x / a.nch;
    const int ch = (int)(blockIdx.x % a.nch);
    const int64_t j0w = (int64_t)ch * WCH + (int64_t)w * KW;
    unsigned char *ring = wsm + (size_t)w * WRING;
    unsigned char *bslice = wsm + (size_t)WW * WRING + 2 * WW * 64 * 4 + (size_t)w * KW * 4;
    const float *bsl = load_bias_slice<RT, BIAS>(a, j0w, bslice);
    float rm[RT][4], ril[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t row = h * a.G + 16 * rt + 4 * grp + i;
            rm[rt][i] = a.row_m[row];
            ril[rt][i] = a.row_il[row];
        }
    const float invG = 1.0f / (float)(16 * RT);
    float *out = a.importance + h * a.n;
    window_stream<RT, BIAS>(a, h, j0w, ring, bsl, [&](float (&y)[RT][4], int64_t j, bool valid) {
        float r = 0.f;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) r = fmaf(__builtin_amdgcn_exp2f(y[rt][i] - rm[rt][i]), ril[rt][i], r);
        r += __shfl_xor(r, 16);
        r += __shfl_xor(r, 32);
        if (grp == 0 && valid) out[j] = r * invG;
    });
}

// ---------------------------------------------------------------------------
bool window_mfma_supported(const fw_rows &rows) {
    return rows.dtype == FW_BF16 && rows.d == WD && rows.G % 16 == 0 && rows.G >= 16 && rows.G <= 64 &&
           rows.n * WD * 2 < (int64_t)1 << 31;
}

size_t window_part_entries(const fw_rows &rows) {
    return (size_t)rows.H * rows.G * (size_t)((rows.n + WCH - 1) / WCH);
}

template <int RT, bool BIAS>
static void launch_window_rt(const WinArgs &a, hipStream_t st) {
    const size_t lds = (size_t)WW * WRING + 2 * WW * 64 * 4 + (BIAS ? (size_t)WW * KW * 4 : 0);
    const dim3 grid((unsigned)(a.H * a.nch));
    hipLaunchKernelGGL((window_stats_kernel<RT, BIAS>), grid, dim3(WTH), lds, st, a);
    hipLaunchKernelGGL(window_combine2_kernel, dim3((unsigned)((a.H * a.G + 255) / 256)), dim3(256), 0, st,
                       a.H * a.G, a.nch, a.part_m, a.part_l, const_cast<float *>(a.row_m),
                       const_cast<float *>(a.row_il));
    hipLaunchKernelGGL((window_importance_kernel<RT, BIAS>), grid, dim3(WTH), lds, st, a);
}

template <int RT>
static void launch_window_b(const WinArgs &a, hipStream_t st) {
    if (a.bias) launch_window_rt<RT, true>(a, st);
    else launch_window_rt<RT, false>(a, st);
}

void launch_window_mfma(const fw_rows &rows, float *part_m, float *part_l, float *row_m, float *row_il,
                        float *importance, hipStream_t st) {
    WinArgs a{};
    a.q = (const uint16_t *)rows.q;
    a.k = (const uint16_t *)rows.k;
    a.scale = rows.scale;
    a.bias = rows.bias;
    a.H = rows.H;
    a.G = rows.G;
    a.n = rows.n;
    a.nch = (int)((rows.n + WCH - 1) / WCH);
    a.part_m = part_m;
    a.part_l = part_l;
    a.row_m = row_m;
    a.row_il = row_il;
    a.importance = importance;
    switch (rows.G / 16) {
        case 1: launch_window_b<1>(a, st); break;
        case 2: launch_window_b<2>(a, st); break;
        case 3: launch_window_b<3>(a, st); break;
        default: launch_window_b<4>(a, st); break;
    }
}

}  // namespace fw
