// Fused top-k forced-weight evaluation for bf16 rows with d = 128 and
// n in {1024, 2048, 4096} (Definition 2.1; gap through Lemma 2.2's first
// form).  One workgroup takes 16 query rows of one key/value unit and every
// key; nothing but the results leaves the chip.
//
//   1. logits   S^T = K Q^T on MFMA (16x16x32 bf16, fp32 accumulate); each of
//               the 8 waves owns n/8 keys and keeps its 16 x n/8 logits in
//               registers (lane l holds row l%16 for 4 keys of every tile)
//   2. softmax  row max, min and sum of exp across lanes and waves
//   3. select   per row a 1024-bin histogram of the logits over [min, max]
//               (bins are monotone in the logit), the bin holding the k-th
//               largest for every budget, the few logits of that bin gathered
//               and sorted: the exact k-th key (logit desc, index asc)
//   4. tiers    P = softmax weights rounded to bf16, split by tier (ranks
//               [0,k_0), [k_0,k_1), ..., rest); O^T_t += V^T P^T_t on MFMA,
//               V staged through LDS and read transposed (ds_read_tr16_b64);
//               one pass over the keys per 32 or 64 columns of d bounds the
//               accumulators
//   5. epilogue partial tier sums of the eight waves combined in LDS; o, o_S,
//               gap (1 - p(S)) ||m_{S^c} - m_S||, dropped mass.
// Rows whose selection is degenerate (all logits equal, non-finite values, or
// more than 128 logits sharing the threshold bin) are listed and recomputed by
// a one-row-per-workgroup fallback that selects by radix over the exact keys.
#include "fw_internal.hpp"
#include "select.hpp"
#include "topk_fused.hpp"

namespace fw {

namespace {
constexpr int FR = 16;        // rows per workgroup
constexpr int FW = 8;         // waves per workgroup
constexpr int FTH = FW * 64;  // threads per workgroup
constexpr int FD = 128;       // head dimension
constexpr int FBINS = 1024;   // histogram bins per row
constexpr int FCAP = 128;     // logits gathered from the threshold bin
constexpr int FIXCAP = 32;    // per row: logits equal to a threshold logit, past its index
constexpr float LOG2E = 1.4426950408889634f;
// keeps the scheduler from hoisting the work of every tile of an unrolled
// per-logit loop at once (which exhausts the register file)
#define FW_TILE_FENCE() __builtin_amdgcn_sched_barrier(0)

constexpr int RING = 16384;   // bytes of streaming ring per wave
constexpr int KD = 4;         // K tiles (16 keys x 128 d, 4 KiB) per ring

struct FusedLds {
    size_t wred, thr, ssb, bias;      // persistent
    size_t hist, lists, cntr, fix;    // selection
    size_t ring;                      // K tiles (phase 1), V blocks (tier products)
    size_t opart;                     // partial tier sums
    size_t total;
};

// columns of d per pass of the tier products: 64 columns are 128 bytes of a
// V row, a whole cache line per row for the block loads
__host__ __device__ constexpr int fused_dq(int) { return 64; }

__host__ __device__ inline FusedLds fused_lds(int nk, int n) {
    const int dq = fused_dq(nk);
    FusedLds L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = align_up(o + bytes, 16); return at; };
    L.wred = take((size_t)4 * FW * FR * 4);    // [quantity][wave][row]
    L.thr = take((size_t)FR * 4 * 4 * 4);      // [row][budget][4 ints]
    L.ssb = take((size_t)(FD / dq) * FR * 4 * 4);  // [pass][row][budget] squared norms
    L.bias = take((size_t)n * 4);              // each wave's slice of the bias
    const size_t base = o;
    L.hist = base;
    L.lists = align_up(base + (size_t)FR * FBINS * 4, 16);
    L.cntr = align_up(L.lists + (size_t)FR * nk * FCAP * 8, 16);
    L.fix = align_up(L.cntr + (size_t)FR * 8 * 4, 16);
    const size_t sel_end = L.fix + (size_t)FR * FIXCAP * 8;
    L.ring = base;
    const size_t r_end = base + (size_t)FW * RING;
    L.opart = base;
    const size_t o_end = base + (size_t)FW * (nk + 1) * FR * (dq + 4) * 4;
    size_t end = sel_end > r_end ? sel_end : r_end;
    end = end > o_end ? end : o_end;
    L.total = align_up(end, 16);
    return L;
}

// 0xFFFF in each 16-bit half of x (two 2-bit tier codes) whose code is at
// most kk, else 0: packed 16-bit subtract, then the sign spread by an
// arithmetic shift
__device__ __forceinline__ uint32_t codes_le(uint32_t x, int kk) {
    const s16x2 d = __builtin_bit_cast(s16x2, x) - (s16x2)(short)(kk + 1);
    return __builtin_bit_cast(uint32_t, d >> (s16x2)(short)15);
}
// reductions over the four lanes of a wave that share a row (l, l^16, l^32, l^48)
__device__ __forceinline__ float rmax4(float v) {
    v = fmaxf(v, __shfl_xor(v, 16));
    return fmaxf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float rmin4(float v) {
    v = fminf(v, __shfl_xor(v, 16));
    return fminf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float rsum4(float v) {
    v += __shfl_xor(v, 16);
    return v + __shfl_xor(v, 32);
}

}  // namespace

// ---------------------------------------------------------------------------
template <int TILES, int NK, bool BIAS, bool SEL>
__global__ void __launch_bounds__(FTH, 1) topk_fused_kernel(FusedArgs a) {
    constexpr int NT = NK + 1;
    constexpr int DQ = fused_dq(NK);
    constexpr int NPASS = FD / DQ, DT = DQ / 16, CPT = DQ / 32;
    constexpr int VCR = DQ / 8, VLQ = DQ / 16;  // V block: 16-byte chunks per row, loads per block
    constexpr int VD = RING / (32 * DQ * 2);      // V blocks per ring
    extern __shared__ __align__(16) unsigned char smem[];
    const FusedLds L = fused_lds(NK, 128 * TILES);
    float *wred = (float *)(smem + L.wred);
    int *thr = (int *)(smem + L.thr);
    float *ssb = (float *)(smem + L.ssb);
    int *hist = (int *)(smem + L.hist);
    unsigned long long *lists = (unsigned long long *)(smem + L.lists);
    int *cntr = (int *)(smem + L.cntr);
    unsigned long long *fixl = (unsigned long long *)(smem + L.fix);
    float *opart = (float *)(smem + L.opart);
#define WRED(qq, ww, rr) wred[((qq) * FW + (ww)) * FR + (rr)]
#define THR(rr, kk, ff) thr[((rr) * 4 + (kk)) * 4 + (ff)]

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int rl = lane & 15, grp = lane >> 4;
    // workgroup -> (unit, row tile); the row tiles of a unit land on one XCD
    // (workgroups are dealt to the 8 XCDs round-robin) so they share its L2
    const int64_t tiles_per_unit = a.G / FR;
    int64_t h, rt;
    {
        const int64_t b = blockIdx.x;
        if ((a.H & 7) == 0) {
            const int64_t xcd = b & 7, s = b >> 3;
            h = (s / tiles_per_unit) * 8 + xcd;
            rt = s % tiles_per_unit;
        } else {
            h = b / tiles_per_unit;
            rt = b % tiles_per_unit;
        }
    }
    const int n = a.n;
    const int64_t row0 = h * a.G + rt * FR;
    const float sc = a.scale ? a.scale[h] : (float)(1.0 / sqrt((double)FD));
    const int kw0 = w * 16 * TILES;  // this wave's first key
    // The row tiles of a unit read the same keys.  Each starts its walk over
    // them at a different tile (logit tile t holds keys kw0 + 16 tk(t) ..),
    // so that at any moment they ask the L2 for different lines, and the
    // later readers of a line find it there.  The shift is even, so the two
    // tiles of a value block stay adjacent.
    const int trot = (int)((rt * 2) & (TILES - 1));
    auto tk = [&](int t) { return (t + trot) & (TILES - 1); };

    // ---- 1. logits --------------------------------------------------------
    // K streams through this wave's ring, KD - 1 tiles ahead of the MFMAs.
    // A tile (16 keys x 128 d) is 4 loads of 4 whole key rows each (1 KiB
    // contiguous per load: few cache lines per instruction).  In LDS the
    // 16-byte chunk c of key row r sits at chunk position c ^ r of the row, so
    // that the MFMA operand reads (16 rows, same chunk) hit distinct banks.
    float S[TILES][4];
    unsigned char *kring = smem + L.ring + (size_t)w * RING;
    const float *bsl = (const float *)(smem + L.bias) + kw0;
    {
        bf16x8 qb[4];
        const uint16_t *qr = a.q + (row0 + rl) * FD + 8 * grp;
#pragma unroll
        for (int s = 0; s < 4; ++s) qb[s] = *(const bf16x8 *)(qr + 32 * s);
        if (BIAS) {  // this wave's bias slice, 256 bytes per load
            const rsrc_t bres = make_rsrc(a.bias, (uint32_t)n * 4);
#pragma unroll
            for (int c = 0; c < TILES / 4; ++c)
                dma4(bres, (void *)(bsl + 64 * c), (uint32_t)(kw0 + lane) * 4, (uint32_t)(256 * c));
        }
        const rsrc_t kres = make_rsrc(a.k + h * (int64_t)n * FD, (uint32_t)n * FD * 2);
        // load s, lane l: key row r = 4 s + l / 16, chunk position l % 16,
        // which holds chunk (l % 16) ^ r of that row
        uint32_t kvo[4], kro[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int r = 4 * s + (lane >> 4);
            kvo[s] = ((uint32_t)(kw0 + r) * FD + 8 * ((lane & 15) ^ r)) * 2;
            // MFMA step s, lane l: key row rl, chunk 4 s + grp
            kro[s] = (uint32_t)(rl * 256 + (((4 * s + grp) ^ rl) * 16));
        }
        auto issue = [&](int t) {
#pragma unroll
            for (int s = 0; s < 4; ++s)
                dma16(kres, kring + (t % KD) * 4096 + s * 1024, kvo[s], (uint32_t)(tk(t) * 16 * FD * 2));
        };
#pragma unroll
        for (int t = 0; t < KD - 1 && t < TILES; ++t) issue(t);
#pragma unroll
        for (int t = 0; t < TILES; ++t) {
            wait_lds();  // the slot refilled next was read one tile ago
            if (t + KD - 1 < TILES) issue(t + KD - 1);
            const int after = (TILES - 1 - t < KD - 1) ? TILES - 1 - t : KD - 1;
            wait_vm(4 * after);
            const unsigned char *kt = kring + (t % KD) * 4096;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 4; ++s)
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8 *)(kt + kro[s]), qb[s], acc, 0, 0, 0);
            if (BIAS) {
                const f32x4 bj = *(const f32x4 *)(bsl + 16 * tk(t) + 4 * grp);
#pragma unroll
                for (int i = 0; i < 4; ++i) S[t][i] = sc * acc[i] + bj[i];
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) S[t][i] = sc * acc[i];
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // ---- 2. row max / min / sum of exp -----------------------------------
    {
        float mx = -INFINITY, mn = INFINITY;
#pragma unroll
        for (int t = 0; t < TILES; ++t) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                mx = fmaxf(mx, S[t][i]);
                mn = fminf(mn, S[t][i]);
            }
            FW_TILE_FENCE();
        }
        mx = rmax4(mx);
        mn = rmin4(mn);
        if (grp == 0) {
            WRED(0, w, rl) = mx;
            WRED(1, w, rl) = mn;
        }
    }
    lds_barrier();
    float m = WRED(0, 0, rl), zmin = WRED(1, 0, rl);
#pragma unroll
    for (int ww = 1; ww < FW; ++ww) {
        m = fmaxf(m, WRED(0, ww, rl));
        zmin = fminf(zmin, WRED(1, ww, rl));
    }
    {
        // normaliser; written as exp2(S log2e - m log2e) so that it is not merged
        // with the weights computed later (which would keep 128 values alive)
        const float mL = -m * LOG2E;
        float es = 0.f;
#pragma unroll
        for (int t = 0; t < TILES; ++t) {
#pragma unroll
            for (int i = 0; i < 4; ++i) es += __builtin_amdgcn_exp2f(fmaf(S[t][i], LOG2E, mL));
            FW_TILE_FENCE();
        }
        es = rsum4(es);
        if (grp == 0) WRED(2, w, rl) = es;
    }
    for (int e = tid; e < FR * FBINS; e += FTH) hist[e] = 0;
    for (int e = tid; e < FR * 8; e += FTH) cntr[e] = 0;
    lds_barrier();
    float lsum = 0.f;
#pragma unroll
    for (int ww = 0; ww < FW; ++ww) lsum += WRED(2, ww, rl);
    const float inv_l = 1.0f / lsum;
    const float range = m - zmin;
    const bool degenerate = !(range > 0.f) || !(range < INFINITY) || !(lsum > 0.f) || !(lsum < INFINITY);
    const float inv_w = degenerate ? 0.f : (float)FBINS / range;

    // ---- 3. selection -----------------------------------------------------
    // bin(z) = min(FBINS - 1, int(fma(z, -inv_w, m inv_w))): non-increasing in
    // z (a rounded affine map), so bins are ordered by logit, highest first.
    // The histogram and the threshold-bin pass below evaluate the same
    // expression on the same operands and agree bit for bit.
    const float bnw = -inv_w, bmw = m * inv_w;
#pragma unroll
    for (int t = 0; t < TILES; ++t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int bin = min(FBINS - 1, (int)fmaf(S[t][i], bnw, bmw));
            atomicAdd(&hist[rl * FBINS + bin], 1);
        }
        FW_TILE_FENCE();
    }
    lds_barrier();
    // wave w scans rows 2w, 2w+1; lane owns bins [16 lane, 16 lane + 16),
    // read once into registers
    for (int rr = 0; rr < FR / FW; ++rr) {
        const int r = (FR / FW) * w + rr;
        int hv[16];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            typedef int i32x4 __attribute__((ext_vector_type(4)));
            const i32x4 x = *(const i32x4 *)&hist[r * FBINS + 16 * lane + 4 * q4];
            hv[4 * q4] = x[0]; hv[4 * q4 + 1] = x[1]; hv[4 * q4 + 2] = x[2]; hv[4 * q4 + 3] = x[3];
        }
        int c = 0;
#pragma unroll
        for (int b = 0; b < 16; ++b) c += hv[b];
        int incl = c;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off);
            if (lane >= off) incl += y;
        }
        for (int kk = 0; kk < NK; ++kk) {
            const int kv = a.ks.k[kk];
            const unsigned long long bal = __ballot(incl >= kv);
            const int f = __ffsll(bal) - 1;
            if (lane == f) {
                int cum = incl - c, bsel = 16 * lane + 15, need = 1, cnt = 0;
                bool found = false;
#pragma unroll
                for (int b = 0; b < 16; ++b) {
                    const bool here = !found && cum + hv[b] >= kv;
                    bsel = here ? 16 * lane + b : bsel;
                    need = here ? kv - cum : need;
                    cnt = here ? hv[b] : cnt;
                    found |= here;
                    cum += hv[b];
                }
                THR(r, kk, 0) = bsel;
                THR(r, kk, 1) = need;
                THR(r, kk, 2) = cnt;
            }
        }
    }
    lds_barrier();
    {
        // logits in the threshold bin of some budget (a few per row): one
        // branch per logit, one LDS atomic per appended key
        int tb[NK];
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) tb[kk] = THR(rl, kk, 0);
        const float m1 = opaque(bmw), w1 = opaque(bnw);
#pragma unroll
        for (int t = 0; t < TILES; ++t) {
            // the tile's four logits tested together: one branch per tile
            int bin[4], hit[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                bin[i] = min(FBINS - 1, (int)fmaf(S[t][i], w1, m1));
                hit[i] = 0;
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) hit[i] |= (int)(bin[i] == tb[kk]);
            }
            if (hit[0] | hit[1] | hit[2] | hit[3]) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (!hit[i]) continue;
                    const uint32_t j = (uint32_t)(kw0 + 16 * tk(t) + 4 * grp + i);
                    const unsigned long long e = ((unsigned long long)ord_key(S[t][i]) << 32) | (0xFFFFFFFFu - j);
#pragma unroll
                    for (int kk = 0; kk < NK; ++kk)
                        if (bin[i] == tb[kk]) {
                            const int p = atomicAdd(&cntr[rl * 8 + kk], 1);
                            if (p < FCAP) lists[(rl * NK + kk) * FCAP + p] = e;
                        }
                }
            }
            FW_TILE_FENCE();
        }
    }
    lds_barrier();
    // the need-th largest entry of each (row, budget) list, within one wave:
    // rank by counting for lists of up to 64 entries, else a bitonic sort of
    // two entries per lane (entries are distinct: the low word is the index)
    for (int li = w; li < FR * NK; li += FW) {
        const int r = li / NK, kk = li % NK;
        const int cnt = cntr[r * 8 + kk];
        const int need = THR(r, kk, 1);
        unsigned long long sel = 0ull;
        // Logits equal to the threshold logit but past its index are out of
        // the set, yet the one-compare tier rule below counts them in: they
        // are listed per row (entry = key, inverted index) and their tiers
        // recomputed by the exact rule.  A full list sends the row to the
        // exact fallback.
        bool fix_over = false;
        auto fix_out = [&](unsigned long long e, bool valid) {
            const uint32_t sk = (uint32_t)(sel >> 32), jc = 0xFFFFFFFFu - (uint32_t)sel;
            const bool x = valid && (uint32_t)(e >> 32) == sk && (0xFFFFFFFFu - (uint32_t)e) > jc;
            const unsigned long long bx = __ballot(x);
            if (bx) {
                int base = 0;
                if (lane == 0) base = atomicAdd(&cntr[r * 8 + 6], __popcll(bx));
                base = __shfl(base, 0);
                const int pos = base + __popcll(bx & ((1ull << lane) - 1ull));
                if (x && pos < FIXCAP) fixl[r * FIXCAP + pos] = e;
                fix_over |= base + __popcll(bx) > FIXCAP;
            }
        };
        if (cnt <= 64) {
            const unsigned long long e = (lane < cnt) ? lists[li * FCAP + lane] : 0ull;
            // rank = entries above e, read as LDS broadcasts (every lane the
            // same address), four independent reads per step
            const unsigned long long *lp = lists + li * FCAP;
            int rank = 0;
            for (int jj = 0; jj < cnt; jj += 4) {
#pragma unroll
                for (int u = 0; u < 4; ++u) rank += (int)(jj + u < cnt) & (int)(lp[jj + u] > e);
            }
            const unsigned long long bal = __ballot(lane < cnt && rank == need - 1);
            const int f = bal ? __ffsll(bal) - 1 : 0;
            sel = ((unsigned long long)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(e >> 32), f) << 32) |
                  (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)e, f);
            fix_out(e, lane < cnt);
        } else {
            unsigned long long e0 = (lane < cnt) ? lists[li * FCAP + lane] : 0ull;
            unsigned long long e1 = (lane + 64 < cnt) ? lists[li * FCAP + lane + 64] : 0ull;
            for (int size = 2; size <= 2 * 64; size <<= 1) {
                for (int stride = size >> 1; stride > 0; stride >>= 1) {
                    if (stride == 64) {  // partner of element x is x ^ 64: same lane
                        const unsigned long long hi = e0 > e1 ? e0 : e1, lo = e0 > e1 ? e1 : e0;
                        e0 = hi;
                        e1 = lo;
                    } else {
                        const unsigned long long p0 = __shfl_xor(e0, stride), p1 = __shfl_xor(e1, stride);
                        const bool upper = (lane & stride) != 0;
                        const bool d0 = (lane & size) == 0, d1 = ((lane + 64) & size) == 0;
                        const unsigned long long mx0 = e0 > p0 ? e0 : p0, mn0 = e0 > p0 ? p0 : e0;
                        const unsigned long long mx1 = e1 > p1 ? e1 : p1, mn1 = e1 > p1 ? p1 : e1;
                        e0 = (d0 != upper) ? mx0 : mn0;
                        e1 = (d1 != upper) ? mx1 : mn1;
                    }
                }
            }
            const int x = (need - 1) & 127;
            const unsigned long long v0 = __shfl(e0, x & 63), v1 = __shfl(e1, x & 63);
            sel = (x < 64) ? v0 : v1;
            // finite logits have keys above zero, so the zero padding never matches
            fix_out(e0, true);
            fix_out(e1, true);
        }
        if (lane == 0) {
            THR(r, kk, 0) = (int)(uint32_t)(sel >> 32);
            THR(r, kk, 1) = (int)(0xFFFFFFFFu - (uint32_t)(sel & 0xFFFFFFFFull));
            THR(r, kk, 3) = (cnt > FCAP || need < 1 || need > cnt || fix_over) ? 1 : 0;
        }
    }
    lds_barrier();
    uint32_t tkey[NK];
    int tcut[NK];
    bool bad = degenerate;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
        tkey[kk] = (uint32_t)THR(rl, kk, 0);
        tcut[kk] = THR(rl, kk, 1);
        bad |= THR(rl, kk, 3) != 0;
    }
    if (w == 0 && grp == 0) {
        a.flags[row0 + rl] = bad ? 1 : 0;
        if (bad) a.flag_list[atomicAdd(a.flag_count, 1)] = (int32_t)(row0 + rl);
    }
    if (SEL && !bad) {  // the selected keys of the largest budget: count, reserve, write
        int c = 0;
        const float kf = opaque(key_to_float(tkey[NK - 1]));
        const int kc = opaque(tcut[NK - 1]);
#pragma unroll
        for (int t = 0; t < TILES; ++t) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = kw0 + 16 * tk(t) + 4 * grp + i;
                c += (int)(S[t][i] > kf) | ((int)(S[t][i] == kf) & (int)(j <= kc));
            }
            FW_TILE_FENCE();
        }
        int pos = c ? atomicAdd(&cntr[rl * 8 + 7], c) : 0;
        const float kx = opaque(kf);
        const int cx = opaque(kc);
#pragma unroll
        for (int t = 0; t < TILES; ++t) {
            FW_TILE_FENCE();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = kw0 + 16 * tk(t) + 4 * grp + i;
                if ((int)(S[t][i] > kx) | ((int)(S[t][i] == kx) & (int)(j <= cx))) {
                    const uint32_t u = ord_key(S[t][i]);
                    if (pos < a.kmax)
                        a.sel[(row0 + rl) * a.kmax + pos] =
                            ((unsigned long long)u << 32) | (0xFFFFFFFFu - (uint32_t)j);
                    ++pos;
                }
            }
        }
    }
    // tiers (2 bits per logit) and bf16 weights packed in pairs: from here
    // the lane keeps 3/4 fewer registers for its keys.  Word TB[t / 4] holds
    // tiles 4 (t / 4) .. + 3; key i of tile t sits at bit
    // 16 (i % 2) + 2 (2 (t % 4) + i / 2), so one shift brings the codes of a
    // pair of keys to the low bits of the two 16-bit halves.
    uint32_t TB[(TILES + 3) / 4];
    uint32_t P2[TILES][2];
    // thresholds as floats: ord_key order equals float order for finite
    // logits (both identify -0 with +0), and compares on S itself share no
    // work with the selection passes above
    float tf[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
        tf[kk] = opaque(key_to_float(tkey[kk]));
        tcut[kk] = opaque(tcut[kk]);
    }
    const float mL3 = -opaque(m) * LOG2E, il3 = opaque(inv_l);
    // The budgets' sets are nested: a key's tier is the number of sets that
    // leave it out.  Membership is one compare, logit >= threshold; the keys
    // for which the index decides (listed above) are corrected afterwards.
#pragma unroll
    for (int t = 0; t < TILES; ++t) {
        if ((t & 3) == 0) TB[t >> 2] = 0;
        float pv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float s = S[t][i];
            int tier = NK;
#pragma unroll
            for (int kk = 0; kk < NK; ++kk) tier -= (int)(s >= tf[kk]);
            TB[t >> 2] |= (uint32_t)tier << (16 * (i & 1) + 2 * (2 * (t & 3) + (i >> 1)));
            pv[i] = __builtin_amdgcn_exp2f(fmaf(s, LOG2E, mL3)) * il3;
        }
        // round to bf16 (nearest even) in pairs: the weights the tier
        // products and masses use
        P2[t][0] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){pv[0], pv[1]}, bf16x2));
        P2[t][1] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){pv[2], pv[3]}, bf16x2));
        FW_TILE_FENCE();
    }
    {
        // listed keys: the lane holding key j recomputes its tier with the
        // index rule (logit above the threshold, or equal and at most its index)
        const int nf = min(cntr[rl * 8 + 6], FIXCAP);
        int nmax = nf;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) nmax = max(nmax, __shfl_xor(nmax, off));
        for (int f = 0; f < nmax; ++f) {
            if (f < nf) {
                const unsigned long long e = fixl[rl * FIXCAP + f];
                const int j = (int)(0xFFFFFFFFu - (uint32_t)e);
                const int jj = j - kw0 - 4 * grp;  // 16 tk(t) + i for a key of this lane
                if (jj >= 0 && jj < 16 * TILES && (jj & 15) < 4) {
                    const float s = key_to_float((uint32_t)(e >> 32));
                    int tier = NK;
#pragma unroll
                    for (int kk = 0; kk < NK; ++kk)
                        tier -= (int)(s > tf[kk]) | ((int)(s == tf[kk]) & (int)(j <= tcut[kk]));
                    const int t = ((jj >> 4) - trot) & (TILES - 1), i = jj & 3;
                    const int sh = 16 * (i & 1) + 2 * (2 * (t & 3) + (i >> 1));
#pragma unroll
                    for (int x = 0; x < (TILES + 3) / 4; ++x)
                        if (x == (t >> 2)) TB[x] = (TB[x] & ~(3u << sh)) | ((uint32_t)tier << sh);
                }
            }
        }
    }
    lds_barrier();  // selection buffers are dead from here

    // ---- 4./5. tier products per DQ columns of d, then the epilogue -------
    const rsrc_t vres = make_rsrc(a.v + h * (int64_t)n * FD, (uint32_t)n * FD * 2);
    static_assert(VCR == 8, "V block rows are 8 chunks of 16 bytes");
    // load qq of a block, lane l: row 8 qq + l / 8, chunk position l % 8, which
    // holds chunk (l % 8) ^ (row % 8) of the row (conflict-free transposed reads)
    const uint32_t vvo = ((uint32_t)(kw0 + (lane >> 3)) * FD + 8 * ((lane & 7) ^ (lane >> 3))) * 2;
    unsigned char *vring = smem + L.ring + (size_t)w * RING;
    static_assert(DT == 4, "four 16-column tiles per pass");
    const int cq = rl & 3, cr = rl >> 2;
    // LDS byte address of this wave's ring, and the lane's transposed-read
    // offsets: row 4 grp + cr (= 4 (grp & 1) + cr mod 8), columns 16 dt + 4 cq
    // .. + 4, i.e. chunk 2 dt + cq / 2 at position chunk ^ (row mod 8)
    const uint32_t vra = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char *)vring;
    uint32_t vrd[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
        vrd[dt] = (uint32_t)(((4 * grp + cr) * DQ + ((2 * dt + (cq >> 1)) ^ (4 * (grp & 1) + cr)) * 8 + 4 * (cq & 1)) * 2);
    const bf16x8 ones = __builtin_bit_cast(bf16x8, (s16x8){0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80});
    const int64_t R = a.H * a.G;
    for (int pass = 0; pass < NPASS; ++pass) {
        // the tier operands below do not depend on the pass; an opaque zero
        // keeps them from being hoisted out of this loop for every block
        // at once (256 values), which would spill
        const uint32_t pz = opaque(0u);
        f32x4 acc[DT][NT], accm[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
            accm[tt] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) acc[dt][tt] = (f32x4){0.f, 0.f, 0.f, 0.f};
        }
        // V block b (32 keys x DQ columns, 2 DQ bytes per key, swizzled) in
        // ring slot b % VD, VD - 1 blocks ahead of the MFMAs
        constexpr int NB = TILES / 2;
        auto issue = [&](int b) {
#pragma unroll
            for (int qq = 0; qq < VLQ; ++qq)
                dma16(vres, vring + (b % VD) * (32 * DQ * 2) + qq * 1024, vvo,
                      (uint32_t)(((32 * ((b + trot / 2) & (NB - 1)) + (64 / VCR) * qq) * FD + DQ * pass) * 2));
        };
#pragma unroll
        for (int b = 0; b < VD - 1 && b < NB; ++b) issue(b);
#pragma unroll
        for (int blk = 0; blk < NB; ++blk) {
            wait_lds();  // the slot refilled next was read one block ago
            if (blk + VD - 1 < NB) issue(blk + VD - 1);
            const int after = (NB - 1 - blk < VD - 1) ? NB - 1 - blk : VD - 1;
            wait_vm(VLQ * after);
            // P^T operands: slots 0..3 = tile 2 blk, slots 4..7 = tile 2 blk + 1,
            // zero where the key is in another tier.  The nested sets' copies
            // N_kk (keys of tier <= kk) are masks of the packed pair; the tiers
            // are their differences, exact as 32-bit integers since each half
            // of a word is either the weight or zero in all of them
            uint32_t pw[NT][4];
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const int t = 2 * blk + hf;
#pragma unroll
                for (int pr = 0; pr < 2; ++pr) {
                    const uint32_t x = ((TB[t >> 2] ^ pz) >> (2 * (2 * (t & 3) + pr))) & 0x00030003u;
                    const uint32_t pp = P2[t][pr];
                    uint32_t prev = 0u;
#pragma unroll
                    for (int kk = 0; kk < NK; ++kk) {
                        const uint32_t nk = pp & codes_le(x, kk);
                        pw[kk][2 * hf + pr] = nk - prev;
                        prev = nk;
                    }
                    pw[NK][2 * hf + pr] = pp - prev;
                }
            }
            s16x8 pb[NT];
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) {
                typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                const u32x4 x = {pw[tt][0], pw[tt][1], pw[tt][2], pw[tt][3]};
                pb[tt] = __builtin_bit_cast(s16x8, x);
            }
            // V^T operands: transposed reads of rows 4 grp + cr (keys 0..15 of
            // the block) and 16 + 4 grp + cr (2048 bytes on), all eight in one
            // statement that also waits for them; the compiler would otherwise
            // drain every outstanding ring load before each transposed read
            s16x4 vt[DT][2];
            {
                const uint32_t slot = vra + (uint32_t)((blk % VD) * (32 * DQ * 2));
                asm volatile(
                    "ds_read_b64_tr_b16 %0, %8\n"
                    "ds_read_b64_tr_b16 %1, %8 offset:2048\n"
                    "ds_read_b64_tr_b16 %2, %9\n"
                    "ds_read_b64_tr_b16 %3, %9 offset:2048\n"
                    "ds_read_b64_tr_b16 %4, %10\n"
                    "ds_read_b64_tr_b16 %5, %10 offset:2048\n"
                    "ds_read_b64_tr_b16 %6, %11\n"
                    "ds_read_b64_tr_b16 %7, %11 offset:2048\n"
                    "s_waitcnt lgkmcnt(0)"
                    : "=&v"(vt[0][0]), "=&v"(vt[0][1]), "=&v"(vt[1][0]), "=&v"(vt[1][1]),
                      "=&v"(vt[2][0]), "=&v"(vt[2][1]), "=&v"(vt[3][0]), "=&v"(vt[3][1])
                    : "v"(slot + vrd[0]), "v"(slot + vrd[1]), "v"(slot + vrd[2]), "v"(slot + vrd[3])
                    : "memory");
            }
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const bf16x8 vbf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vt[dt][0], vt[dt][1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                for (int tt = 0; tt < NT; ++tt)
                    acc[dt][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        vbf, __builtin_bit_cast(bf16x8, pb[tt]), acc[dt][tt], 0, 0, 0);
            }
            // tier masses (first pass only): the same operands against a
            // block of ones
            if (pass == 0) {
#pragma unroll
                for (int tt = 0; tt < NT; ++tt)
                    accm[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, __builtin_bit_cast(bf16x8, pb[tt]), accm[tt], 0, 0, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // every lane of a row holds that row's masses over this wave's keys
        if (pass == 0 && grp == 0) {
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) WRED(tt, w, rl) = accm[tt][0];
        }
        lds_barrier();  // the rings are dead; partial sums overlay them
        // acc[dt][tt][i] = O^T[d = DQ pass + 16 dt + 4 grp + i][row rl] over this
        // wave's keys; stored [wave][tier][row][column], rows DQ + 4 floats
        // apart, so that the epilogue's column reads are contiguous
        constexpr int OP = DQ + 4;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int tt = 0; tt < NT; ++tt)
                *(f32x4 *)&opart[(((size_t)w * NT + tt) * FR + rl) * OP + 16 * dt + 4 * grp] = acc[dt][tt];
        lds_barrier();
        {
            // epilogue lane: row er, CPT columns from ec; derived from an opaque
            // copy of the thread index so that nothing here is hoisted out of
            // the pass loop (and spilled across the products)
            const int etid = opaque(tid);
            const int er = etid >> 5, ec = (etid & 31) * CPT;
            float M[NT];
            float mtot = 0.f;
#pragma unroll
            for (int tt = 0; tt < NT; ++tt) {
                float s = 0.f;
#pragma unroll
                for (int ww = 0; ww < FW; ++ww) s += WRED(tt, ww, er);
                M[tt] = s;
                mtot += s;
            }
            float T[NT][CPT];
#pragma unroll
            for (int tt = 0; tt < NT; ++tt)
#pragma unroll
                for (int c = 0; c < CPT; ++c) {
                    float s = 0.f;
#pragma unroll
                    for (int ww = 0; ww < FW; ++ww) s += opart[(((size_t)ww * NT + tt) * FR + er) * OP + ec + c];
                    T[tt][c] = s;
                }
            const float inv_tot = 1.0f / mtot;
            // outputs through a wave-uniform base (this tile's first row) and a
            // 32-bit byte offset: no per-lane 64-bit addresses to keep alive
            static_assert(CPT == 2, "two columns per lane and pass");
            const int col = DQ * pass + ec;
            const uint32_t eo = (uint32_t)((er * FD + col) * 4);
            if (a.o) {
                f32x2 ov;
#pragma unroll
                for (int c = 0; c < CPT; ++c) {
                    float s = 0.f;
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt) s += T[tt][c];
                    ov[c] = s * inv_tot;
                }
                *(f32x2 *)((char *)(a.o + row0 * FD) + eo) = ov;
            }
#pragma unroll
            for (int kk = 0; kk < NK; ++kk) {
                float km = 0.f, rm = 0.f;
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    if (tt <= kk) km += M[tt]; else rm += M[tt];
                }
                const float ikm = 1.0f / km, irm = (rm > 0.f) ? 1.0f / rm : 0.f;
                float ss = 0.f;
                f32x2 osv;
#pragma unroll
                for (int c = 0; c < CPT; ++c) {
                    float kt = 0.f, rt2 = 0.f;
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt) {
                        if (tt <= kk) kt += T[tt][c]; else rt2 += T[tt][c];
                    }
                    const float oS = kt * ikm;
                    osv[c] = oS;
                    if (rm > 0.f) {
                        const float diff = rt2 * irm - oS;
                        ss = fmaf(diff, diff, ss);
                    }
                }
                const int64_t plane = (int64_t)a.ks.perm[kk] * R + row0;
                if (a.o_s) *(f32x2 *)((char *)(a.o_s + plane * FD) + eo) = osv;
#pragma unroll
                for (int off = 1; off < 32; off <<= 1) ss += __shfl_xor(ss, off);
                if ((tid & 31) == 0) ssb[(pass * FR + er) * 4 + kk] = ss;
                if (pass == NPASS - 1 && (tid & 31) == 0) {
                    float st = ss;
                    for (int pp = 0; pp < NPASS - 1; ++pp) st += ssb[(pp * FR + er) * 4 + kk];
                    const uint32_t go = (uint32_t)er * 4u;
                    *(float *)((char *)(a.gap + plane) + go) = (rm > 0.f) ? (rm * inv_tot) * sqrtf(st) : 0.f;
                    *(float *)((char *)(a.dropped + plane) + go) = rm * inv_tot;
                }
            }
        }
        lds_barrier();
    }
#undef WRED
#undef THR
}

// ---------------------------------------------------------------------------
// rank-ordered indices: sort each row's selected keys (descending)
// ---------------------------------------------------------------------------
// Bitonic sorts of a row's kmax entries, padded with zeros (which sort last)
// to N = (threads) E; one workgroup per row, thread t holding entries
// t E .. t E + E - 1 in registers.  For partner distance s (a power of two):
// s < E pairs entries within a thread; E <= s < 64 E pairs threads of one wave
// (lane exchanges); larger s pairs waves through LDS.  The stages are
// unrolled, so every exchange has a fixed lane pattern.  An entry is
// ord_key(z) << 32 | (2^32 - 1 - key), so descending order is logit desc,
// then index asc.

template <int E, int T>
__device__ __forceinline__ void bitonic_rows(unsigned long long (&x)[E], unsigned long long *sb) {
    constexpr int N = T * E;
    const int t = threadIdx.x;
#pragma unroll
    for (int size = 2; size <= N; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride >= E; stride >>= 1) {
            const int m = stride / E;   // partner thread t ^ m
            // the larger of the pair goes to the lower position in a
            // descending block ((position & size) == 0), else the smaller
            const bool keep_max = (((t * E) & size) == 0) == ((t & m) == 0);
            unsigned long long y[E];
            if (m < 64) {
#pragma unroll
                for (int e = 0; e < E; ++e) y[e] = xlane64(x[e], m);
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) sb[t * E + e] = x[e];
                __syncthreads();
#pragma unroll
                for (int e = 0; e < E; ++e) y[e] = sb[(t ^ m) * E + e];
                __syncthreads();
            }
#pragma unroll
            for (int e = 0; e < E; ++e) x[e] = ((x[e] > y[e]) == keep_max) ? x[e] : y[e];
        }
#pragma unroll
        for (int s = E / 2; s >= 1; s >>= 1) {
            if (s < size) {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    if ((e & s) == 0) {
                        const bool desc = ((t * E + e) & size) == 0;
                        const unsigned long long a = x[e], b = x[e + s];
                        const bool sw = (a < b) == desc;
                        x[e] = sw ? b : a;
                        x[e + s] = sw ? a : b;
                    }
                }
            }
        }
    }
}

// T threads per row: one wave up to 1024 entries, four waves beyond
template <int E, int T>
__global__ void __launch_bounds__(T)
fused_sort_kernel(const unsigned long long *sel, const int32_t *flags, int kmax, int32_t *topk_idx) {
    __shared__ unsigned long long sb[T > 64 ? T * E : 1];
    const int64_t r = blockIdx.x;
    if (flags[r]) return;
    const int t = threadIdx.x;
    const unsigned long long *src = sel + r * kmax;
    unsigned long long x[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int i = t * E + e;
        x[e] = i < kmax ? src[i] : 0ull;
    }
    bitonic_rows<E, T>(x, sb);
    int32_t *dst = topk_idx + r * kmax;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int i = t * E + e;
        if (i < kmax) dst[i] = (int32_t)(0xFFFFFFFFu - (uint32_t)(x[e] & 0xFFFFFFFFull));
    }
}

__global__ void fused_clear_kernel(int32_t *flag_count) {
    if (threadIdx.x == 0) *flag_count = 0;
}

// ---------------------------------------------------------------------------
// fallback for listed rows: one workgroup per row, exact radix selection
// ---------------------------------------------------------------------------
template <int NK>
__global__ void __launch_bounds__(256)
fused_fixup_kernel(FusedArgs a, int32_t *topk_idx) {
    constexpr int NT = NK + 1;
    __shared__ float z[4096];
    __shared__ int hist[256];
    __shared__ int scan[256];
    __shared__ int sh[4];
    __shared__ float redf[256];
    __shared__ float acc_s[2][NT][FD + 1];   // [key half][tier][column]
    __shared__ float mass_s[2][NT];
    __shared__ float qs[FD];
    __shared__ unsigned long long sb[4096];   // weights and tiers, then the sort buffer
    const int tid = threadIdx.x;
    const int n = a.n;
    const int count = *a.flag_count;
    for (int li = blockIdx.x; li < count; li += gridDim.x) {
        const int64_t r = a.flag_list[li];
        const int64_t h = r / a.G;
        const float sc = a.scale ? a.scale[h] : (float)(1.0 / sqrt((double)FD));
        const uint16_t *qr = a.q + r * FD;
        const uint16_t *kh = a.k + h * (int64_t)n * FD;
        const uint16_t *vh = a.v + h * (int64_t)n * FD;
        for (int c = tid; c < FD; c += 256) qs[c] = bf16_bits_to_f32(qr[c]);
        __syncthreads();
        for (int j = tid; j < n; j += 256) {
            // the key row in 16-byte pieces
            const uint4 *kr = (const uint4 *)(kh + (int64_t)j * FD);
            float s = 0.f;
            for (int c8 = 0; c8 < FD / 8; ++c8) {
                const uint4 x = kr[c8];
                const uint32_t wd[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    s = fmaf(qs[8 * c8 + 2 * u], __uint_as_float(wd[u] << 16), s);
                    s = fmaf(qs[8 * c8 + 2 * u + 1], __uint_as_float(wd[u] & 0xFFFF0000u), s);
                }
            }
            z[j] = sc * s + (a.bias ? a.bias[j] : 0.f);
        }
        __syncthreads();
        float m = -INFINITY;
        for (int j = tid; j < n; j += 256) m = fmaxf(m, z[j]);
        m = block_reduce(m, redf, OpMax());
        float l = 0.f;
        for (int j = tid; j < n; j += 256) l += expf(z[j] - m);
        l = block_reduce(l, redf, OpSum());
        uint32_t key[NK];
        int64_t cut[NK];
        for (int kk = 0; kk < NK; ++kk) {
            int rem;
            radix_select_desc(z, n, a.ks.k[kk], hist, sh, &key[kk], &rem);
            cut[kk] = nth_tie(z, n, key[kk], rem, scan, sh);
        }
        // every key's weight and tier, then the tier sums: thread (column c,
        // key half hh) over the keys of its half
        float *pw = (float *)sb;
        int *tw = (int *)(pw + 4096);
        for (int j = tid; j < n; j += 256) {
            const uint32_t u = ord_key(z[j]);
            int tier = NK;
            for (int kk = NK - 1; kk >= 0; --kk)
                if (u > key[kk] || (u == key[kk] && j <= cut[kk])) tier = kk;
            pw[j] = expf(z[j] - m) / l;
            tw[j] = tier;
        }
        __syncthreads();
        {
            const int c = tid & (FD - 1), hh = tid / FD;
            const int j0 = hh * (n / 2), j1 = hh ? n : n / 2;
            float accl[NT], ml[NT];
            for (int tt = 0; tt < NT; ++tt) { accl[tt] = 0.f; ml[tt] = 0.f; }
            for (int j = j0; j < j1; ++j) {
                const float p = pw[j];
                const int tier = tw[j];
                const float vv = bf16_bits_to_f32(vh[(int64_t)j * FD + c]);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt)
                    if (tt == tier) { accl[tt] = fmaf(p, vv, accl[tt]); ml[tt] += p; }
            }
            for (int tt = 0; tt < NT; ++tt) {
                acc_s[hh][tt][c] = accl[tt];
                if (c == 0) mass_s[hh][tt] = ml[tt];
            }
        }
        __syncthreads();
        if (tid < FD) {
            for (int tt = 0; tt < NT; ++tt) acc_s[0][tt][tid] += acc_s[1][tt][tid];
        }
        if (tid == 0) {
            for (int tt = 0; tt < NT; ++tt) mass_s[0][tt] += mass_s[1][tt];
        }
        __syncthreads();
        if (tid < 64) {
            const int64_t R = a.H * a.G;
            float mtot = 0.f;
            for (int tt = 0; tt < NT; ++tt) mtot += mass_s[0][tt];
            for (int c = tid; c < FD; c += 64) {
                float s = 0.f;
                for (int tt = 0; tt < NT; ++tt) s += acc_s[0][tt][c];
                if (a.o) a.o[r * FD + c] = s / mtot;
            }
            for (int kk = 0; kk < NK; ++kk) {
                float km = 0.f, rm = 0.f;
                for (int tt = 0; tt < NT; ++tt) { if (tt <= kk) km += mass_s[0][tt]; else rm += mass_s[0][tt]; }
                float ss = 0.f;
                for (int c = tid; c < FD; c += 64) {
                    float kt = 0.f, rt2 = 0.f;
                    for (int tt = 0; tt < NT; ++tt) { if (tt <= kk) kt += acc_s[0][tt][c]; else rt2 += acc_s[0][tt][c]; }
                    const float oS = kt / km;
                    if (a.o_s) a.o_s[((int64_t)a.ks.perm[kk] * R + r) * FD + c] = oS;
                    if (rm > 0.f) { const float df = rt2 / rm - oS; ss = fmaf(df, df, ss); }
                }
                for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
                if (tid == 0) {
                    a.gap[(int64_t)a.ks.perm[kk] * R + r] = (rm > 0.f) ? (rm / mtot) * sqrtf(ss) : 0.f;
                    a.dropped[(int64_t)a.ks.perm[kk] * R + r] = rm / mtot;
                }
            }
        }
        if (topk_idx) {
            int sort_len = 1;
            while (sort_len < a.kmax) sort_len <<= 1;
            for (int i = tid; i < sort_len; i += 256) sb[i] = 0ull;
            __syncthreads();
            const int64_t chunk = (n + 255) / 256;
            const int64_t lo = tid * chunk, hi = (lo + chunk < n) ? lo + chunk : n;
            int c = 0;
            for (int64_t j = lo; j < hi; ++j) {
                const uint32_t u = ord_key(z[j]);
                c += (u > key[NK - 1]) || (u == key[NK - 1] && j <= cut[NK - 1]);
            }
            int total;
            int pos = block_exclusive_scan(c, scan, &total);
            for (int64_t j = lo; j < hi; ++j) {
                const uint32_t u = ord_key(z[j]);
                if ((u > key[NK - 1]) || (u == key[NK - 1] && j <= cut[NK - 1]))
                    sb[pos++] = ((unsigned long long)u << 32) | (0xFFFFFFFFu - (uint32_t)j);
            }
            __syncthreads();
            for (int size = 2; size <= sort_len; size <<= 1)
                for (int stride = size >> 1; stride > 0; stride >>= 1) {
                    for (int i = tid; i < sort_len / 2; i += 256) {
                        const int lo2 = 2 * stride * (i / stride) + (i % stride), hi2 = lo2 + stride;
                        const bool desc = (lo2 & size) == 0;
                        const unsigned long long x = sb[lo2], y = sb[hi2];
                        if (desc ? (x < y) : (x > y)) { sb[lo2] = y; sb[hi2] = x; }
                    }
                    __syncthreads();
                }
            for (int i = tid; i < a.kmax; i += 256)
                topk_idx[r * a.kmax + i] = (int32_t)(0xFFFFFFFFu - (uint32_t)(sb[i] & 0xFFFFFFFFull));
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
bool fused_topk_supported(const fw_rows &rows, const KsArg &ks) {
    return rows.dtype == FW_BF16 && rows.d == FD && (rows.n == 1024 || rows.n == 2048 || rows.n == 4096) &&
           rows.G % FR == 0 && ks.n >= 1 && ks.n <= 3;
}

size_t fused_topk_ws_bytes(const fw_rows &rows, int kmax) {
    const size_t R = (size_t)rows.H * rows.G;
    return align_up(R * 4, 256) * 2 + 256 + align_up(R * (size_t)kmax * 8, 256);
}

template <int TILES, int NK>
static void launch_fused_t(const FusedArgs &a, unsigned blocks, size_t lds, hipStream_t st) {
    if (a.bias) {
        if (a.sel) hipLaunchKernelGGL((topk_fused_kernel<TILES, NK, true, true>), dim3(blocks), dim3(FTH), lds, st, a);
        else hipLaunchKernelGGL((topk_fused_kernel<TILES, NK, true, false>), dim3(blocks), dim3(FTH), lds, st, a);
    } else {
        if (a.sel) hipLaunchKernelGGL((topk_fused_kernel<TILES, NK, false, true>), dim3(blocks), dim3(FTH), lds, st, a);
        else hipLaunchKernelGGL((topk_fused_kernel<TILES, NK, false, false>), dim3(blocks), dim3(FTH), lds, st, a);
    }
}

template <int NK>
static void launch_fused_nk(const FusedArgs &a, unsigned blocks, hipStream_t st) {
    const size_t lds = fused_lds(NK, a.n).total;
    switch (a.n) {
        case 1024: launch_fused_t<8, NK>(a, blocks, lds, st); break;
        case 2048: launch_fused_t<16, NK>(a, blocks, lds, st); break;
        default: launch_fused_t<32, NK>(a, blocks, lds, st); break;
    }
}

hipError_t launch_fused_topk(const fw_rows &rows, const KsArg &ks, float *o, float *o_s, float *gap,
                             float *dropped, int32_t *topk_idx, void *ws, hipStream_t st) {
    const size_t R = (size_t)rows.H * rows.G;
    const int kmax = ks.k[ks.n - 1];
    char *base = (char *)ws;
    FusedArgs a{};
    a.q = (const uint16_t *)rows.q;
    a.k = (const uint16_t *)rows.k;
    a.v = (const uint16_t *)rows.v;
    a.scale = rows.scale;
    a.bias = rows.bias;
    a.H = rows.H;
    a.G = rows.G;
    a.n = (int)rows.n;
    a.ks = ks;
    a.o = o;
    a.o_s = o_s;
    a.gap = gap;
    a.dropped = dropped;
    a.kmax = kmax;
    a.flags = (int32_t *)base;
    a.flag_list = (int32_t *)(base + align_up(R * 4, 256));
    a.flag_count = (int32_t *)(base + 2 * align_up(R * 4, 256));
    a.sel = topk_idx ? (unsigned long long *)(base + 2 * align_up(R * 4, 256) + 256) : nullptr;
    launch_fused_clear(a.flag_count, st);
    const unsigned blocks = (unsigned)(R / FR);
    switch (ks.n) {
        case 1: launch_fused_nk<1>(a, blocks, st); break;
        case 2: launch_fused_nk<2>(a, blocks, st); break;
        default: launch_fused_nk<3>(a, blocks, st); break;
    }
    launch_fused_finish(a, ks.n, topk_idx, st);
    return hipGetLastError();
}

void launch_fused_clear(int32_t *flag_count, hipStream_t st) {
    hipLaunchKernelGGL(fused_clear_kernel, dim3(1), dim3(64), 0, st, flag_count);
}

void launch_fused_finish(const FusedArgs &a, int nk, int32_t *topk_idx, hipStream_t st) {
    const size_t R = (size_t)a.H * a.G;
    if (topk_idx) {
        const dim3 g((unsigned)R), b(256);
        const unsigned long long *sel = a.sel;
        const int32_t *fl = a.flags;
        const dim3 w(64);
        if (a.kmax <= 64) hipLaunchKernelGGL((fused_sort_kernel<1, 64>), g, w, 0, st, sel, fl, a.kmax, topk_idx);
        else if (a.kmax <= 128) hipLaunchKernelGGL((fused_sort_kernel<2, 64>), g, w, 0, st, sel, fl, a.kmax, topk_idx);
        else if (a.kmax <= 256) hipLaunchKernelGGL((fused_sort_kernel<4, 64>), g, w, 0, st, sel, fl, a.kmax, topk_idx);
        else if (a.kmax <= 512) hipLaunchKernelGGL((fused_sort_kernel<8, 64>), g, w, 0, st, sel, fl, a.kmax, topk_idx);
        else if (a.kmax <= 1024) hipLaunchKernelGGL((fused_sort_kernel<16, 64>), g, w, 0, st, sel, fl, a.kmax, topk_idx);
        else if (a.kmax <= 2048) hipLaunchKernelGGL((fused_sort_kernel<8, 256>), g, b, 0, st, sel, fl, a.kmax, topk_idx);
        else hipLaunchKernelGGL((fused_sort_kernel<16, 256>), g, b, 0, st, sel, fl, a.kmax, topk_idx);
    }
    switch (nk) {
        case 1: hipLaunchKernelGGL(fused_fixup_kernel<1>, dim3(64), dim3(256), 0, st, a, topk_idx); break;
        case 2: hipLaunchKernelGGL(fused_fixup_kernel<2>, dim3(64), dim3(256), 0, st, a, topk_idx); break;
        default: hipLaunchKernelGGL(fused_fixup_kernel<3>, dim3(64), dim3(256), 0, st, a, topk_idx); break;
    }
}

}  // namespace fw
