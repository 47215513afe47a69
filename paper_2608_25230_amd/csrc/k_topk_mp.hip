// Multi-pass fused top-k forced-weight evaluation for bf16 rows with d = 128,
// n a multiple of 32 up to 4096 and 128 query rows per unit tile
// (Definition 2.1; the gap through Lemma 2.2's first form).
//
// One workgroup of eight waves takes 128 query rows of one key/value unit;
// each wave owns 16 rows and sees every key.  The unit's keys (and, in the
// last pass, its values) stream through a ring of LDS blocks of 32 keys that
// all eight waves read, so one read of K or V from L2 serves 128 rows.  The
// logits are recomputed on MFMA (16x16x32 bf16, fp32 accumulate) in every pass
// rather than held, which leaves the register file to the tier products:
//   A. range    every fourth block: each row's largest and smallest logit, the
//               range of its histogram
//   B. hist     every logit into one of 240 bins over that range (bins ordered
//               by logit, highest first; logits outside go to the end bins)
//   C. collect  a scan of the histogram gives, per budget, the bin holding the
//               k-th largest logit; that bin's logits are listed and ranked:
//               the exact k-th key (logit desc, index asc) of every budget
//   D. tiers    unnormalised weights exp(z - c), c the sampled maximum,
//               rounded to bf16 and split into disjoint tiers by rank
//               ([0, k_0), [k_0, k_1), ..., rest);
//               O^T_t += V^T P^T_t over all 128 columns on MFMA for every tier,
//               V read transposed from LDS (ds_read_b64_tr_b16), and the tier
//               masses from the same operands against a block of ones
// The epilogue forms o, o_S, the gap (1 - p(S)) ||m_{S^c} - m_S|| and the
// dropped mass of every budget, all ratios of tier sums and masses, so the
// softmax normaliser is never formed: it is the sum of the tier masses.  Rows whose selection degenerates (all
// sampled logits equal, non-finite values, threshold bins too full) are
// listed and recomputed by the exact fallback of the fused path.
#include "fw_internal.hpp"
#include "topk_fused.hpp"

namespace fw {

namespace {
constexpr int MW = 8;                // waves per workgroup
constexpr int MR = 16 * MW;          // rows per workgroup, 16 per wave
constexpr int MTH = 64 * MW;         // threads per workgroup
constexpr int MD = 128;              // head dimension
constexpr int KB = 32;               // keys per ring block
constexpr int NB = 240;              // histogram bins per row
constexpr int FIXC = 8;              // listed index-tie corrections per row
constexpr int SSTR = 4;              // pass A reads one block in SSTR
constexpr int KBYTES = KB * MD * 2;  // one block of keys (or values): 8 KiB
constexpr int BBYTES = KB * 4;       // the block's bias
constexpr int KSLOT = KBYTES + BBYTES;         // key ring slot: keys, bias
constexpr int KVSLOT = 2 * KBYTES + BBYTES;    // key/value ring slot: keys, bias, values
constexpr float MLOG2E = 1.4426950408889634f;

// LDS layout.  A few per-row counters and corrections persist; the rest, R,
// is shared in turn by each pass's ring and its working set, so that every
// ring keeps as many blocks in flight as the pass leaves room for (the
// unit's keys stream from the Infinity Cache or HBM, at microseconds of
// latency):
//   pass A  ring of 2 GA key slots
//   pass B  histograms (two rows per 32-bit word, 16-bit counts), ring of 2 GB
//   pass C  lists of threshold-bin logits (one pool per wave), ring of 2 GC
//   pass D  ring of 2 GD key/value slots
constexpr int L_FC = 0;                    // [MR] per-row correction counts
constexpr int L_FX = L_FC + MR * 4;        // [MR][FIXC] corrections (budget << 16 | key)
constexpr int L_R = L_FX + MR * FIXC * 4;
constexpr int L_TOTAL = 159232;            // bytes of LDS per workgroup (one per CU)
constexpr int R_BYTES = L_TOTAL - L_R;
constexpr int HIST_BYTES = (MR / 2) * NB * 4;
// ring batches: blocks per batch of each pass (a ring holds two batches)
constexpr int GA = 8, GB = 5, GC = 3, GD = 4;
constexpr int POOLW = ((R_BYTES - 2 * GC * KSLOT) / (8 * MW)) & ~1;   // list entries per wave
constexpr int ROWCAP = 128;                                           // listed logits per row
static_assert(L_R % 16 == 0 && HIST_BYTES % 16 == 0 && (8 * MW * POOLW) % 16 == 0, "alignment");
static_assert(2 * GA * KSLOT <= R_BYTES && HIST_BYTES + 2 * GB * KSLOT <= R_BYTES, "rings of A, B fit");
static_assert(8 * MW * POOLW + 2 * GC * KSLOT <= R_BYTES && 2 * GD * KVSLOT <= R_BYTES, "rings of C, D fit");

// reductions over the four lanes of a wave that share a row (l, l^16, l^32, l^48)
__device__ __forceinline__ float mp_max4(float v) {
    v = fmaxf(v, __shfl_xor(v, 16));
    return fmaxf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float mp_min4(float v) {
    v = fminf(v, __shfl_xor(v, 16));
    return fminf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float mp_sum4(float v) {
    v += __shfl_xor(v, 16);
    return v + __shfl_xor(v, 32);
}

// Histogram bin of logit z: (hi - z) / width rounded toward zero, clamped to
// [0, NB - 1].  A rounded affine map, non-increasing in z, so bins are ordered
// by logit, highest first.  Passes B and C evaluate it on the same operands
// and agree bit for bit.  A NaN logit lands in bin 0 (the row is then flagged
// by its non-finite normaliser), so the index is always in range.
__device__ __forceinline__ int mp_bin(float z, float bnw, float bmw) {
    return (int)__builtin_amdgcn_fmed3f(fmaf(z, bnw, bmw), 0.f, (float)(NB - 1));
}

// LDS updates inside the ring loops.  Written as inline assembly: the
// compiler cannot tell these addresses from the targets of the direct-to-LDS
// ring loads in flight and would otherwise wait for all of them (vmcnt(0))
// before every plain LDS store or atomic, draining the ring at each block.
// The memory clobber keeps them in program order with the other LDS accesses.
__device__ __forceinline__ void lds_add(uint32_t *p, uint32_t x) {
    const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint32_t *)p;
    asm volatile("ds_add_u32 %0, %1" ::"v"(a), "v"(x) : "memory");
}
__device__ __forceinline__ void lds_store64(unsigned long long *p, unsigned long long x) {
    const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned long long *)p;
    asm volatile("ds_write_b64 %0, %1" ::"v"(a), "v"(x) : "memory");
}

// Ring of direct-to-LDS block loads shared by the eight waves, in batches
// of G blocks: batch b sits in half b % 2 of a ring of 2 G slots.  At each
// batch every wave waits for its own loads of the batch (issued one batch
// earlier), the barrier makes every wave's loads visible and guarantees that
// every wave is done with the previous batch, whose half is refilled with the
// next batch while this one is read.  One barrier per batch leaves the waves
// free to drift apart inside it; `rot` rotates the order in which a wave
// takes the batch's blocks, so that the two waves sharing a SIMD are at
// different points of their work.
template <int G, class Issue, class Body>
__device__ __forceinline__ void mp_ring(int nb, int rot, Issue issue, Body body) {
    const int nbat = (nb + G - 1) / G;
    for (int t = 0; t < G && t < nb; ++t) issue(t);
    for (int b = 0; b < nbat; ++b) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        ring_barrier();
        const int nx = min(G, nb - (b + 1) * G);
        for (int t = 0; t < nx; ++t) issue((b + 1) * G + t);
        const int nc = min(G, nb - b * G);
        for (int t = 0; t < nc; ++t) body(b * G + (t + rot) % nc);   // rot < G, nc <= G
    }
}
}  // namespace

// ---------------------------------------------------------------------------
template <int NK, bool BIAS, bool SEL>
__global__ void __launch_bounds__(MTH, 1) topk_mp_kernel(FusedArgs a) {
    constexpr int NT = NK + 1;
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *rbase = smem + L_R;
    uint32_t *hist = (uint32_t *)rbase;                       // pass B: [MR / 2][NB]
    unsigned long long *lists = (unsigned long long *)rbase;  // pass C: [MW][POOLW]
    int *fcnt = (int *)(smem + L_FC);
    int *fixl = (int *)(smem + L_FX);

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int rl = lane & 15, grp = lane >> 4;
    const int n = a.n, nblk = n / KB;
    // workgroup -> (unit, row tile); the row tiles of a unit land on one XCD
    // (workgroups are dealt to the 8 XCDs round-robin) and share its L2
    const int64_t tpu = a.G / MR;
    int64_t h, rt;
    {
        const int64_t b = blockIdx.x;
        if ((a.H & 7) == 0) {
            const int64_t xcd = b & 7, s = b >> 3;
            h = (s / tpu) * 8 + xcd;
            rt = s % tpu;
        } else {
            h = b / tpu;
            rt = b % tpu;
        }
    }
    const int wr0 = 16 * w;                     // this wave's first row in the tile
    const int myr = wr0 + rl;                   // the row of this lane's logits, in the tile
    const int64_t row0 = h * a.G + rt * MR;     // the tile's first row
    const int64_t myrow = row0 + myr;
    const float sc = a.scale ? a.scale[h] : (float)(1.0 / sqrt((double)MD));

    // Q^T operand of this lane: row myrow, columns 8 grp + 32 s .. + 8
    bf16x8 qb[4];
    {
        const uint16_t *qr = a.q + myrow * MD + 8 * grp;
#pragma unroll
        for (int s = 0; s < 4; ++s) qb[s] = *(const bf16x8 *)(qr + 32 * s);
    }
    const rsrc_t kres = make_rsrc(a.k + h * (int64_t)n * MD, (uint32_t)n * MD * 2);
    const rsrc_t vres = make_rsrc(a.v + h * (int64_t)n * MD, (uint32_t)n * MD * 2);

    // Block loads.  Keys: wave w loads key rows 4 w .. 4 w + 3 of the block
    // (1 KiB contiguous); lane l takes row kr = 4 w + l / 16 and stores its
    // 16-byte chunk (l % 16) ^ (kr % 16) at chunk position l % 16 of the row, so
    // that the MFMA operand reads (16 rows, one chunk) hit distinct banks.
    const int kr = 4 * w + (lane >> 4);
    const uint32_t kvo = ((uint32_t)kr * MD + 8 * ((lane & 15) ^ (kr & 15))) * 2;
    // Values: two halves of 64 columns, each 32 rows of 128 bytes; wave w loads
    // rows 8 (w % 4) .. + 8 of half w / 4, lane l row 8 (w % 4) + l / 8 and
    // chunk (l % 8) ^ (l / 8) at chunk position l % 8 (conflict-free transposed
    // reads).
    const uint32_t vvo = ((uint32_t)(8 * (w & 3) + (lane >> 3)) * MD + 64 * (w >> 2) +
                          8 * ((lane & 7) ^ (lane >> 3))) * 2;
    // Bias: wave w loads the block's biases 4 w .. 4 w + 3 with lanes 0..3.
    const uint32_t bvo = (uint32_t)(4 * w + (lane & 3)) * 4;
    auto issue_k = [&](unsigned char *slot, int blk) {
        dma16(kres, slot + 1024 * w, kvo, (uint32_t)blk * KBYTES);
        if (BIAS) {
            const rsrc_t bres = make_rsrc(a.bias, (uint32_t)n * 4);
            if (lane < 4) dma4(bres, slot + KBYTES + 16 * w, bvo, (uint32_t)blk * BBYTES);
        }
    };
    auto issue_kv = [&](unsigned char *slot, int blk) {
        issue_k(slot, blk);
        dma16(vres, slot + KBYTES + BBYTES + 4096 * (w >> 2) + 1024 * (w & 3), vvo, (uint32_t)blk * KBYTES);
    };

    // MFMA operand offsets: key tile t of a slot at 4096 t, row rl, chunk
    // 4 s + grp at chunk position (4 s + grp) ^ rl
    uint32_t kro[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) kro[s] = (uint32_t)(rl * 256 + (((4 * s + grp) ^ rl) * 16));
    // z[t][e]: the logit of this lane's row against key 16 t + 4 grp + e of
    // the block (S^T = K Q^T, lane l holds column l % 16, rows 4 (l / 16) ..)
    auto logits = [&](const unsigned char *slot, float (&z)[2][4]) {
        // the two tiles' accumulation chains interleaved
        f32x4 ac[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int t = 0; t < 2; ++t)
                ac[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8 *)(slot + 4096 * t + kro[s]), qb[s],
                                                                ac[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const f32x4 acc = ac[t];
            if (BIAS) {
                const f32x4 bj = *(const f32x4 *)(slot + KBYTES + (16 * t + 4 * grp) * 4);
#pragma unroll
                for (int e = 0; e < 4; ++e) z[t][e] = sc * acc[e] + bj[e];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) z[t][e] = sc * acc[e];
            }
        }
    };

    // ---- A. range ----------------------------------------------------------
    float zmx = -INFINITY, zmn = INFINITY;
    {
        const int na = (nblk + SSTR - 1) / SSTR;
        auto slot = [&](int i) { return rbase + (i % (2 * GA)) * KSLOT; };
        mp_ring<GA>(na, 0, [&](int i) { issue_k(slot(i), i * SSTR); },
                [&](int i) {
                    float z[2][4];
                    logits(slot(i), z);
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            zmx = fmaxf(zmx, z[t][e]);
                            zmn = fminf(zmn, z[t][e]);
                        }
                });
    }
    zmx = mp_max4(zmx);
    zmn = mp_min4(zmn);
    const float range = zmx - zmn;
    bool bad = !(range > 0.f) || !(range < INFINITY);
    const float inv_w = bad ? 0.f : (float)NB / range;
    const float bnw = -inv_w, bmw = bad ? 0.f : zmx * inv_w;
    const float c2 = bad ? 0.f : zmx * MLOG2E;   // the weights' exponent reference, in log2 units

    // ---- B. histogram --------------------------------------------------------
    // Rows 2 p and 2 p + 1 share word p NB + bin: 16-bit counts (n <= 4096)
    // in the low and the high half, so each lane adds its own constant.
    ring_barrier();   // every wave is done with pass A's ring, which the histograms overlay
    for (int e = lane; e < 8 * NB; e += 64) hist[(wr0 >> 1) * NB + e] = 0u;   // this wave's rows only
    uint32_t *hword = hist + (myr >> 1) * NB;
    const uint32_t hinc = (myr & 1) ? 0x10000u : 1u;
    {
        auto slot = [&](int i) { return rbase + HIST_BYTES + (i % (2 * GB)) * KSLOT; };
        mp_ring<GB>(nblk, (w >> 2) * (GB / 2), [&](int i) { issue_k(slot(i), i); },
            [&](int i) {
                float z[2][4];
                logits(slot(i), z);
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) lds_add(&hword[mp_bin(z[t][e], bnw, bmw)], hinc);
            });
    }

    // ---- scan: the threshold bin of every budget, per row -----------------
    // Row r of this wave: lane L holds bins 4 L .. 4 L + 3 (L < NB / 4), from
    // the half of the row-pair words that holds row r.  A budget equal to n
    // keeps every key and needs no threshold.
    int tb[NK], need[NK], cntb[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) { tb[kk] = -1; need[kk] = 0; cntb[kk] = 0; }
    for (int r = 0; r < 16; ++r) {
        typedef int i32x4 __attribute__((ext_vector_type(4)));
        int hv[4] = {0, 0, 0, 0};
        if (lane < NB / 4) {
            const i32x4 x = *(const i32x4 *)(hist + ((wr0 + r) >> 1) * NB + 4 * lane);
            const int sh = 16 * (r & 1);
            hv[0] = (x[0] >> sh) & 0xFFFF; hv[1] = (x[1] >> sh) & 0xFFFF;
            hv[2] = (x[2] >> sh) & 0xFFFF; hv[3] = (x[3] >> sh) & 0xFFFF;
        }
        const int c = hv[0] + hv[1] + hv[2] + hv[3];
        int incl = c;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off);
            if (lane >= off) incl += y;
        }
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
            const int kv = a.ks.k[kk];
            if (kv >= n) continue;   // wave-uniform
            const unsigned long long bal = __ballot(incl >= kv);
            const int f = bal ? __ffsll((long long)bal) - 1 : 0;
            int bsel = -1, nd = 0, ct = 0;
            if (lane == f && bal) {
                int cum = incl - c;
                bool found = false;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const bool here = !found && cum + hv[b] >= kv;
                    bsel = here ? 4 * lane + b : bsel;
                    nd = here ? kv - cum : nd;
                    ct = here ? hv[b] : ct;
                    found |= here;
                    cum += hv[b];
                }
            }
            const int bs = __builtin_amdgcn_readlane(bsel, f);
            const int ns = __builtin_amdgcn_readlane(nd, f);
            const int cs = __builtin_amdgcn_readlane(ct, f);
            if (rl == r) { tb[kk] = bs; need[kk] = ns; cntb[kk] = cs; }
        }
    }
    // One list per row in its wave's pool: every logit of the row's threshold
    // bins (a budget equal to n has none), rows packed one after another.
    // rtot is the row's number of such logits (the bins' counts, each bin
    // once), pbase its first entry.  A row already left to the fallback takes
    // no room and lists nothing.
    int rtot = 0;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
        bool first = tb[kk] >= 0;
#pragma unroll
        for (int k2 = 0; k2 < kk; ++k2) first &= tb[k2] != tb[kk];
        if (first) rtot += cntb[kk];
        if (tb[kk] < 0 && a.ks.k[kk] < n) bad = true;   // no threshold bin found
    }
    bad |= rtot > ROWCAP;
    int pbase;
    {
        const int tot = bad ? 0 : rtot;
        int incl = tot;   // exclusive prefix over the wave's 16 rows (each group of 16 lanes holds them all)
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            const int y = __shfl_up(incl, o, 16);
            if (rl >= o) incl += y;
        }
        pbase = incl - tot;
        bad |= incl > POOLW;
    }
    if (bad) {
        rtot = 0;
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) tb[kk] = -2;   // matches no bin: pass C lists nothing
    }

    // ---- C. collect the threshold bins' logits ----------------------------
    // entry = ord_key(z) << 32 | bin << 16 | (0xFFFF - key): within a bin,
    // larger entries rank first (logit desc, then index asc).  Positions come
    // from a running count held by the row's four lanes and an exclusive
    // prefix over them, with no atomics.
    unsigned long long *pool = lists + (size_t)w * POOLW;
    unsigned long long *prow = pool + pbase;
    int rc = 0;
    ring_barrier();   // every wave's scan is done: the pools overlay the histograms
    {
        auto slot = [&](int i) { return rbase + 8 * MW * POOLW + (i % (2 * GC)) * KSLOT; };
        mp_ring<GC>(nblk, 0, [&](int i) { issue_k(slot(i), i); },
            [&](int i) {
                float z[2][4];
                logits(slot(i), z);
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    int bin[4];
                    bool hit[4];
                    int nh = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        bin[e] = mp_bin(z[t][e], bnw, bmw);
                        bool hh = false;
#pragma unroll
                        for (int kk = 0; kk < NK; ++kk) hh |= bin[e] == tb[kk];
                        hit[e] = hh;
                        nh += (int)hh;
                    }
                    int sc4 = nh;   // inclusive prefix over the row's lanes l, l+16, l+32, l+48
                    {
                        const int y1 = __shfl_up(sc4, 16);
                        if (grp >= 1) sc4 += y1;
                        const int y2 = __shfl_up(sc4, 32);
                        if (grp >= 2) sc4 += y2;
                    }
                    const int total = __shfl(sc4, 48 + rl);
                    int pos = rc + sc4 - nh;
                    rc += total;
                    if (__ballot(nh > 0)) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            if (hit[e]) {
                                const uint32_t j = (uint32_t)(i * KB + 16 * t + 4 * grp + e);
                                if (pos < rtot)
                                    lds_store64(&prow[pos], ((unsigned long long)ord_key(z[t][e]) << 32) |
                                                                ((uint32_t)bin[e] << 16) | (0xFFFFu - j));
                                ++pos;
                            }
                        }
                    }
                }
            });
    }
    bad |= rc != rtot;   // pass C must list exactly the logits the histogram counted
    if (grp == 0) fcnt[myr] = 0;   // rows skipped below keep no corrections
    ring_barrier();   // every wave is done with the key ring; lists complete

    // ---- exact k-th key of every budget, per row ---------------------------
    // Row r's list holds c <= 128 entries: lane L takes entries L and L + 64,
    // and a bitonic network over the 128 slots (zeros past c, below every
    // entry) sorts them descending, that is by logit desc, then index asc,
    // with each bin's entries contiguous (bins run from the highest logits).
    // A budget's key is then the entry need - 1 places after the start of its
    // threshold bin, which follows the listed entries of the higher listed
    // bins.  Entries of that bin equal to it in logit but with a larger index
    // are outside the set although their logit reaches the threshold: they are
    // listed as corrections for the tier products (budget << 16 | key).
    float tz[NK];
    int cut[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) { tz[kk] = -INFINITY; cut[kk] = n; }
    for (int r = 0; r < 16; ++r) {
        const int row = wr0 + r;
        if (__builtin_amdgcn_readlane((int)bad, r)) continue;   // wave-uniform: the fallback recomputes the row
        const int c = __builtin_amdgcn_readlane(rtot, r);
        const int rb = __builtin_amdgcn_readlane(pbase, r);
        int rtb[NK], rneed[NK], rcnt[NK];
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
            rtb[kk] = __builtin_amdgcn_readlane(tb[kk], r);
            rneed[kk] = __builtin_amdgcn_readlane(need[kk], r);
            rcnt[kk] = __builtin_amdgcn_readlane(cntb[kk], r);
        }
        const unsigned long long *lp = pool + rb;
        unsigned long long e0 = lane < c ? lp[lane] : 0ull;
        unsigned long long e1 = lane + 64 < c ? lp[lane + 64] : 0ull;
        // slots L (e0) and L + 64 (e1); the larger of a pair goes to the lower
        // slot in a descending block ((slot & size) == 0), else the smaller
#pragma unroll
        for (int size = 2; size <= 128; size <<= 1) {
#pragma unroll
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                if (stride == 64) {   // size 128: slots L and L + 64, descending
                    const bool sw = e0 < e1;
                    const unsigned long long t0 = e0;
                    e0 = sw ? e1 : e0;
                    e1 = sw ? t0 : e1;
                } else {
                    const unsigned long long y0 = xlane64(e0, stride), y1 = xlane64(e1, stride);
                    const bool lo = (lane & stride) == 0;
                    const bool k0 = ((lane & size) == 0) == lo, k1 = (((lane + 64) & size) == 0) == lo;
                    e0 = ((e0 > y0) == k0) ? e0 : y0;
                    e1 = ((e1 > y1) == k1) ? e1 : y1;
                }
            }
        }
        const uint32_t b0 = ((uint32_t)e0 >> 16) & 0xFFFFu, b1 = ((uint32_t)e1 >> 16) & 0xFFFFu;
        bool fail = false;
        int xk0 = -1, xk1 = -1;   // the smallest budget each entry is a correction for
        const int j0 = (int)(0xFFFFu - ((uint32_t)e0 & 0xFFFFu)), j1 = (int)(0xFFFFu - ((uint32_t)e1 & 0xFFFFu));
#pragma unroll
        for (int kk = NK - 1; kk >= 0; --kk) {
            if (a.ks.k[kk] >= n) continue;   // keeps every key
            // the threshold bin starts after the listed entries of the higher
            // listed bins (each distinct bin counted once)
            int start = 0;
#pragma unroll
            for (int k2 = 0; k2 < NK; ++k2) {
                bool first = rtb[k2] >= 0 && rtb[k2] < rtb[kk];
#pragma unroll
                for (int k3 = 0; k3 < k2; ++k3) first &= rtb[k3] != rtb[k2];
                if (first) start += rcnt[k2];
            }
            const int pos = start + rneed[kk] - 1;
            if (rneed[kk] < 1 || pos >= c) { fail = true; continue; }
            const int fl = pos & 63;
            const unsigned long long sel = pos < 64 ? e0 : e1;
            const uint32_t shi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(sel >> 32), fl);
            const uint32_t slo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)sel, fl);
            if ((int)((slo >> 16) & 0xFFFFu) != rtb[kk]) { fail = true; continue; }
            const int ct = (int)(0xFFFFu - (slo & 0xFFFFu));
            if (rl == r) {
                tz[kk] = key_to_float(shi);
                cut[kk] = ct;
            }
            if (lane < c && (uint32_t)(e0 >> 32) == shi && (int)b0 == rtb[kk] && j0 > ct) xk0 = kk;
            if (lane + 64 < c && (uint32_t)(e1 >> 32) == shi && (int)b1 == rtb[kk] && j1 > ct) xk1 = kk;
        }
        const unsigned long long bx0 = __ballot(xk0 >= 0), bx1 = __ballot(xk1 >= 0);
        const int p0 = __popcll(bx0 & ((1ull << lane) - 1ull));
        const int p1 = __popcll(bx0) + __popcll(bx1 & ((1ull << lane) - 1ull));
        if (xk0 >= 0 && p0 < FIXC) fixl[row * FIXC + p0] = (xk0 << 16) | j0;
        if (xk1 >= 0 && p1 < FIXC) fixl[row * FIXC + p1] = (xk1 << 16) | j1;
        const int nfix = __popcll(bx0) + __popcll(bx1);
        fail |= nfix > FIXC;
        if (rl == r) bad |= fail;
        if (lane == 0) fcnt[row] = min(nfix, FIXC);
    }

    // ---- D. tier products --------------------------------------------------
    f32x4 acc[NT][8], accm[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        accm[tt] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) acc[tt][dt] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }
    const bf16x8 ones =
        __builtin_bit_cast(bf16x8, (s16x8){0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80, 0x3F80});
    // transposed-read offsets inside one 64-column half of a value block: row
    // 4 grp + cr (its chunk positions swizzled by row % 8 = 4 (grp & 1) + cr),
    // columns 16 dt + 4 cq .. + 4
    const int cq = rl & 3, cr = rl >> 2;
    uint32_t vrd[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
        vrd[dt] = (uint32_t)(((4 * grp + cr) * 64 + ((2 * dt + (cq >> 1)) ^ (4 * (grp & 1) + cr)) * 8 + 4 * (cq & 1)) * 2);
    const float mc2 = -c2;
    int selpos = 0;
    auto kvslot = [&](int i) { return rbase + (i % (2 * GD)) * KVSLOT; };
    ring_barrier();   // every wave's rank phase is done with the pools
    mp_ring<GD>(nblk, (w >> 2) * (GD / 2), [&](int i) { issue_kv(kvslot(i), i); },
            [&](int i) {
                unsigned char *slot = kvslot(i);
                float z[2][4];
                logits(slot, z);
                // P^T operands per tier: slots 0..3 keys 4 grp .. + 4 of tile 0,
                // slots 4..7 the same keys of tile 1 (the value operand below
                // follows the same key order)
                uint32_t pw[NT][4];
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    float p[4];
                    bool in[NK][4];   // in[kk][e]: the logit reaches budget kk's threshold
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        p[e] = __builtin_amdgcn_exp2f(fmaf(z[t][e], MLOG2E, mc2));
#pragma unroll
                        for (int kk = 0; kk < NK; ++kk) in[kk][e] = z[t][e] >= tz[kk];
                    }
                    // tier tt < NK: in budget tt's set but not in budget tt - 1's
                    // (thresholds are non-increasing); tier NK: in none.  The
                    // conditions are lane masks, combined on the scalar unit.
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
                        for (int pr = 0; pr < 2; ++pr) {
                            bool c0, c1;
                            if (tt == 0) {
                                c0 = in[0][2 * pr];
                                c1 = in[0][2 * pr + 1];
                            } else if (tt < NK) {
                                c0 = in[tt][2 * pr] && !in[tt - 1][2 * pr];
                                c1 = in[tt][2 * pr + 1] && !in[tt - 1][2 * pr + 1];
                            } else {
                                c0 = !in[NK - 1][2 * pr];
                                c1 = !in[NK - 1][2 * pr + 1];
                            }
                            const f32x2 pp = {c0 ? p[2 * pr] : 0.f, c1 ? p[2 * pr + 1] : 0.f};
                            pw[tt][2 * t + pr] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pp, bf16x2));
                        }
                    if (SEL) {
                        // the selected keys of the largest budget (exact rule),
                        // listed in the row's order of arrival: positions from a
                        // running count held by the row's four lanes and an
                        // exclusive prefix over them, as in pass C
                        bool in[4];
                        int nh = 0;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int j = i * KB + 16 * t + 4 * grp + e;
                            in[e] = (z[t][e] > tz[NK - 1]) || (z[t][e] == tz[NK - 1] && j <= cut[NK - 1]);
                            nh += (int)in[e];
                        }
                        int sc4 = nh;
                        {
                            const int y1 = __shfl_up(sc4, 16);
                            if (grp >= 1) sc4 += y1;
                            const int y2 = __shfl_up(sc4, 32);
                            if (grp >= 2) sc4 += y2;
                        }
                        int pos = selpos + sc4 - nh;
                        selpos += __shfl(sc4, 48 + rl);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            if (in[e]) {
                                const int j = i * KB + 16 * t + 4 * grp + e;
                                if (pos < a.kmax)
                                    a.sel[myrow * a.kmax + pos] =
                                        ((unsigned long long)ord_key(z[t][e]) << 32) | (0xFFFFFFFFu - (uint32_t)j);
                                ++pos;
                            }
                        }
                    }
                }
                bf16x8 pb[NT];
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                    const u32x4 x = {pw[tt][0], pw[tt][1], pw[tt][2], pw[tt][3]};
                    pb[tt] = __builtin_bit_cast(bf16x8, x);
                }
                // V^T operands of both 64-column halves: transposed reads of rows
                // 4 grp + cr (keys 0..15) and 16 + 4 grp + cr (2048 bytes on) of
                // each half, all issued at once; the second half's wait comes
                // after the first half's products.  The operands pass through the
                // wait statements so that no product is scheduled before its wait.
                const uint32_t va =
                    (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char *)(slot + KBYTES + BBYTES);
                s16x4 vt[2][4][2];
                asm volatile(
                    "ds_read_b64_tr_b16 %0, %16\n"
                    "ds_read_b64_tr_b16 %1, %16 offset:2048\n"
                    "ds_read_b64_tr_b16 %2, %17\n"
                    "ds_read_b64_tr_b16 %3, %17 offset:2048\n"
                    "ds_read_b64_tr_b16 %4, %18\n"
                    "ds_read_b64_tr_b16 %5, %18 offset:2048\n"
                    "ds_read_b64_tr_b16 %6, %19\n"
                    "ds_read_b64_tr_b16 %7, %19 offset:2048\n"
                    "ds_read_b64_tr_b16 %8, %16 offset:4096\n"
                    "ds_read_b64_tr_b16 %9, %16 offset:6144\n"
                    "ds_read_b64_tr_b16 %10, %17 offset:4096\n"
                    "ds_read_b64_tr_b16 %11, %17 offset:6144\n"
                    "ds_read_b64_tr_b16 %12, %18 offset:4096\n"
                    "ds_read_b64_tr_b16 %13, %18 offset:6144\n"
                    "ds_read_b64_tr_b16 %14, %19 offset:4096\n"
                    "ds_read_b64_tr_b16 %15, %19 offset:6144\n"
                    "s_waitcnt lgkmcnt(8)"
                    : "=&v"(vt[0][0][0]), "=&v"(vt[0][0][1]), "=&v"(vt[0][1][0]), "=&v"(vt[0][1][1]),
                      "=&v"(vt[0][2][0]), "=&v"(vt[0][2][1]), "=&v"(vt[0][3][0]), "=&v"(vt[0][3][1]),
                      "=&v"(vt[1][0][0]), "=&v"(vt[1][0][1]), "=&v"(vt[1][1][0]), "=&v"(vt[1][1][1]),
                      "=&v"(vt[1][2][0]), "=&v"(vt[1][2][1]), "=&v"(vt[1][3][0]), "=&v"(vt[1][3][1])
                    : "v"(va + vrd[0]), "v"(va + vrd[1]), "v"(va + vrd[2]), "v"(va + vrd[3])
                    : "memory");
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    if (hf == 1)
                        asm volatile("s_waitcnt lgkmcnt(0)"
                                     : "+v"(vt[1][0][0]), "+v"(vt[1][0][1]), "+v"(vt[1][1][0]), "+v"(vt[1][1][1]),
                                       "+v"(vt[1][2][0]), "+v"(vt[1][2][1]), "+v"(vt[1][3][0]), "+v"(vt[1][3][1])
                                     :
                                     : "memory");
#pragma unroll
                    for (int dt = 0; dt < 4; ++dt) {
                        const bf16x8 vb = __builtin_bit_cast(
                            bf16x8, __builtin_shufflevector(vt[hf][dt][0], vt[hf][dt][1], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                        for (int tt = 0; tt < NT; ++tt)
                            acc[tt][4 * hf + dt] =
                                __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, pb[tt], acc[tt][4 * hf + dt], 0, 0, 0);
                    }
                }
#pragma unroll
                for (int tt = 0; tt < NT; ++tt)
                    accm[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[tt], accm[tt], 0, 0, 0);
            });

    // ---- corrections: listed keys whose logit equals a threshold logit but
    // whose index is past that budget's cut sit one tier too low above --------
    {
        int nfx = min(fcnt[myr], FIXC);
        int nmax = nfx;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) nmax = max(nmax, __shfl_xor(nmax, off));
        for (int f = 0; f < nmax; ++f) {
            if (f < nfx && !bad) {
                const int fe = fixl[myr * FIXC + f];
                const int j = fe & 0xFFFF, fk = fe >> 16;
                // its logit is the threshold logit of budget fk
                float zj = 0.f;
#pragma unroll
                for (int kk = 0; kk < NK; ++kk)
                    if (kk == fk) zj = tz[kk];
                int tfast = NK, ttrue = NK;
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    tfast -= (int)(zj >= tz[kk]);
                    ttrue -= (int)((zj > tz[kk]) || (zj == tz[kk] && j <= cut[kk]));
                }
                if (tfast != ttrue) {
                    const f32x2 pp = {__builtin_amdgcn_exp2f(fmaf(zj, MLOG2E, mc2)), 0.f};
                    const uint32_t pbits = __builtin_bit_cast(uint32_t, __builtin_convertvector(pp, bf16x2));
                    const float pr = __uint_as_float(pbits << 16);
                    const uint16_t *vj = a.v + (h * (int64_t)n + j) * MD + 4 * grp;
#pragma unroll
                    for (int dt = 0; dt < 8; ++dt) {
                        const s16x4 vv = *(const s16x4 *)(vj + 16 * dt);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float x = pr * bf16_bits_to_f32((uint16_t)vv[e]);
#pragma unroll
                            for (int tt = 0; tt < NT; ++tt) {
                                if (tt == tfast) acc[tt][dt][e] -= x;
                                if (tt == ttrue) acc[tt][dt][e] += x;
                            }
                        }
                    }
#pragma unroll
                    for (int tt = 0; tt < NT; ++tt) {
                        if (tt == tfast) accm[tt][0] -= pr;
                        if (tt == ttrue) accm[tt][0] += pr;
                    }
                }
            }
        }
    }
    // ---- epilogue ------------------------------------------------------------
    // acc[tt][dt][e] = O^T_tt[column 16 dt + 4 grp + e][row myr]; accm[tt][0]
    // = the tier's mass of that row
    float M[NT];
    float mtot = 0.f;
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        M[tt] = accm[tt][0];
        mtot += M[tt];
    }
    // a non-finite logit (or weight) anywhere in the row shows in the masses
    bad |= !(mtot > 0.f) || !(mtot < INFINITY);
    const float inv_tot = 1.0f / mtot;
    const int64_t R = a.H * a.G;
    float *orow = a.o ? a.o + myrow * MD + 4 * grp : nullptr;
    if (orow) {
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            f32x4 ov;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float s = 0.f;
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) s += acc[tt][dt][e];
                ov[e] = s * inv_tot;
            }
            *(f32x4 *)(orow + 16 * dt) = ov;
        }
    }
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
        float km = 0.f, rm = 0.f;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
            if (tt <= kk) km += M[tt]; else rm += M[tt];
        }
        const float ikm = 1.0f / km, irm = (rm > 0.f) ? 1.0f / rm : 0.f;
        const int64_t plane = (int64_t)a.ks.perm[kk] * R + myrow;
        float *osrow = a.o_s ? a.o_s + plane * MD + 4 * grp : nullptr;
        float ss = 0.f;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            f32x4 osv;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float kt = 0.f, rt2 = 0.f;
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    if (tt <= kk) kt += acc[tt][dt][e]; else rt2 += acc[tt][dt][e];
                }
                const float oS = kt * ikm;
                osv[e] = oS;
                const float diff = rt2 * irm - oS;
                ss = fmaf(diff, diff, ss);
            }
            if (osrow) *(f32x4 *)(osrow + 16 * dt) = osv;
        }
        ss = mp_sum4(ss);
        if (grp == 0) {
            a.gap[plane] = (rm > 0.f) ? (rm * inv_tot) * sqrtf(ss) : 0.f;
            a.dropped[plane] = rm * inv_tot;
        }
    }
    if (grp == 0) {
        a.flags[myrow] = bad ? 1 : 0;
        if (bad) a.flag_list[atomicAdd(a.flag_count, 1)] = (int32_t)myrow;
    }
}

// ---------------------------------------------------------------------------
bool mp_topk_supported(const fw_rows &rows, const KsArg &ks) {
    return rows.dtype == FW_BF16 && rows.d == MD && rows.n >= KB && rows.n <= 4096 && rows.n % KB == 0 &&
           rows.G % MR == 0 && ks.n >= 1 && ks.n <= 3;
}

template <int NK>
static void launch_mp_nk(const FusedArgs &a, unsigned blocks, hipStream_t st) {
    const size_t lds = L_TOTAL;
    if (a.bias) {
        if (a.sel) hipLaunchKernelGGL((topk_mp_kernel<NK, true, true>), dim3(blocks), dim3(MTH), lds, st, a);
        else hipLaunchKernelGGL((topk_mp_kernel<NK, true, false>), dim3(blocks), dim3(MTH), lds, st, a);
    } else {
        if (a.sel) hipLaunchKernelGGL((topk_mp_kernel<NK, false, true>), dim3(blocks), dim3(MTH), lds, st, a);
        else hipLaunchKernelGGL((topk_mp_kernel<NK, false, false>), dim3(blocks), dim3(MTH), lds, st, a);
    }
}

hipError_t launch_mp_topk(const fw_rows &rows, const KsArg &ks, float *o, float *o_s, float *gap,
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
    const unsigned blocks = (unsigned)(R / MR);
    switch (ks.n) {
        case 1: launch_mp_nk<1>(a, blocks, st); break;
        case 2: launch_mp_nk<2>(a, blocks, st); break;
        default: launch_mp_nk<3>(a, blocks, st); break;
    }
    launch_fused_finish(a, ks.n, topk_idx, st);
    return hipGetLastError();
}

}  // namespace fw
