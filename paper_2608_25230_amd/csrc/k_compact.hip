// ContourKV allocation and ragged per-unit storage (Section 4, "ContourKV"
// and "Setup and measured memory").
//
// One threshold tau over every unit's non-floor scores: the quota = budget -
// H*floor largest entries in the order (score desc, unit asc, position asc)
// are kept, plus each unit's last `floor` positions.  tau is found by a
// device-wide radix select (four 8-bit passes over order-preserving keys);
// entries equal to tau are taken in (unit, position) order.  Kept rows are
// then gathered unit after unit, positions ascending, as bit copies.
//
// With a per-unit cap (budget enforcement), each unit first finds its
// (cap - floor)-th best non-floor key in the order (score desc, position asc)
// by a radix select of its own; only keys up to that one are candidates for
// the shared threshold.
#include "fw_internal.hpp"

namespace fw {

namespace {
struct SelState {
    uint32_t prefix, pmask;
    int64_t rem;
    uint32_t hist[256];
};

struct CompactLayout {
    SelState *sel;
    int64_t *cgt, *ceq, *take;
    uint32_t *ckey;  // per unit: key of its last candidate (cap only)
    int64_t *ccut;   // per unit: position of its last candidate among equal keys
    size_t bytes;
};

CompactLayout compact_layout(int64_t H, void *ws) {
    CompactLayout L{};
    size_t off = 0;
    char *base = (char *)ws;
    auto take = [&](size_t bytes) -> void * {
        off = align_up(off, 256);
        void *p = base ? base + off : nullptr;
        off += bytes;
        return p;
    };
    L.sel = (SelState *)take(sizeof(SelState));
    L.cgt = (int64_t *)take((size_t)H * 8);
    L.ceq = (int64_t *)take((size_t)H * 8);
    L.take = (int64_t *)take((size_t)H * 8);
    L.ckey = (uint32_t *)take((size_t)H * 4);
    L.ccut = (int64_t *)take((size_t)H * 8);
    L.bytes = align_up(off, 256);
    return L;
}
// Whether non-floor key j of unit h (order key u) is offered to the shared
// threshold: every key without a cap, else the keys up to the unit's last
// candidate in the order (key desc, position asc).
__device__ __forceinline__ bool offered(const uint32_t *ckey, const int64_t *ccut, int64_t h, int64_t j,
                                        uint32_t u) {
    if (!ckey) return true;
    const uint32_t k = ckey[h];
    return u > k || (u == k && j <= ccut[h]);
}
}  // namespace

// Per unit (one workgroup): its capnf-th best non-floor key (capnf < nf) by a
// radix select over order keys, then the position cut among equal keys
// (ascending positions).  capnf = 0 offers no key.
__global__ void __launch_bounds__(256)
unit_cap_kernel(const float *__restrict__ imp, int64_t n, int64_t nf, int64_t capnf, uint32_t *ckey,
                int64_t *ccut) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_prefix, s_mask;
    __shared__ int64_t s_rem;
    __shared__ int scan[256];
    const int64_t h = blockIdx.x;
    const int t = threadIdx.x;
    const float *r = imp + h * n;
    if (capnf == 0) {
        if (t == 0) {
            ckey[h] = 0xFFFFFFFFu;
            ccut[h] = -1;
        }
        return;
    }
    if (t == 0) {
        s_prefix = 0;
        s_mask = 0;
        s_rem = capnf;
    }
    for (int shift = 24; shift >= 0; shift -= 8) {
        hist[t] = 0;
        __syncthreads();
        const uint32_t prefix = s_prefix, mask = s_mask;
        for (int64_t j = t; j < nf; j += 256) {
            const uint32_t u = ord_key(r[j]);
            if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (t == 0) {
            int64_t cum = 0;
            int b = 0;
            for (int bb = 255; bb >= 0; --bb) {
                if (cum + (int64_t)hist[bb] >= s_rem) { b = bb; break; }
                cum += hist[bb];
            }
            s_prefix |= (uint32_t)b << shift;
            s_mask |= 255u << shift;
            s_rem -= cum;
        }
        __syncthreads();
    }
    // the s_rem-th key equal to the cut key, positions ascending
    const uint32_t key = s_prefix;
    const int64_t need = s_rem;
    const int64_t chunk = (nf + 255) / 256;
    const int64_t lo = t * chunk, hi = (lo + chunk < nf) ? lo + chunk : nf;
    int c = 0;
    for (int64_t j = lo; j < hi; ++j) c += ord_key(r[j]) == key;
    int tot;
    const int before = block_exclusive_scan(c, scan, &tot);
    if (before < need && need <= before + c) {
        int64_t seen = before;
        for (int64_t j = lo; j < hi; ++j)
            if (ord_key(r[j]) == key && ++seen == need) {
                ckey[h] = key;
                ccut[h] = j;
                break;
            }
    }
}

// SnapKV's pooling of a window score: the largest score within kernel / 2
// positions on either side (positions outside the unit ignored).
__global__ void __launch_bounds__(256)
maxpool_kernel(const float *__restrict__ r, int64_t H, int64_t n, int half, float *out) {
    const int64_t total = H * n;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
        const int64_t h = e / n, j = e % n;
        const int64_t lo = j - half < 0 ? 0 : j - half, hi = j + half + 1 < n ? j + half + 1 : n;
        float m = r[h * n + lo];
        for (int64_t i = lo + 1; i < hi; ++i) m = fmaxf(m, r[h * n + i]);
        out[e] = m;
    }
}

__global__ void sel_init_kernel(SelState *s, int64_t quota) {
    const int t = threadIdx.x;
    if (t < 256) s->hist[t] = 0;
    if (t == 0) {
        s->prefix = 0;
        s->pmask = 0;
        s->rem = quota;
    }
}

// histogram of the next 8-bit digit over non-floor entries matching the prefix.
// Block b reads slice b / H of unit b % H (the grid is a multiple of H), so
// positions come without a division per entry; each wave counts into its own
// copy of the bins (fewer lanes contend for one LDS word), summed at the end.
__global__ void __launch_bounds__(256)
sel_hist_kernel(const float *__restrict__ imp, int64_t H, int64_t n, int64_t nf, int shift,
                SelState *s, const uint32_t *ckey, const int64_t *ccut) {
    __shared__ uint32_t hw[4][256];
    const int t = threadIdx.x, w = t >> 6;
#pragma unroll
    for (int i = 0; i < 4; ++i) hw[i][t] = 0;
    __syncthreads();
    const uint32_t prefix = s->prefix, pmask = s->pmask;
    const int64_t hh = blockIdx.x % H;
    const int64_t nsl = gridDim.x / H, sl = blockIdx.x / H;
    const float *row = imp + hh * n;
    for (int64_t j = sl * 256 + t; j < nf; j += nsl * 256) {
        const uint32_t u = ord_key(row[j]);
        if ((u & pmask) == prefix && offered(ckey, ccut, hh, j, u)) atomicAdd(&hw[w][(u >> shift) & 255u], 1u);
    }
    __syncthreads();
    const uint32_t c = hw[0][t] + hw[1][t] + hw[2][t] + hw[3][t];
    if (c) atomicAdd(&s->hist[t], c);
}

// choose the digit holding the rem-th largest; clear the histogram
__global__ void sel_pick_kernel(SelState *s, int shift) {
    if (threadIdx.x == 0) {
        int64_t cum = 0;
        int b = 0;
        for (int bb = 255; bb >= 0; --bb) {
            if (cum + (int64_t)s->hist[bb] >= s->rem) { b = bb; break; }
            cum += s->hist[bb];
        }
        s->prefix |= (uint32_t)b << shift;
        s->pmask |= 255u << shift;
        s->rem -= cum;
    }
    __syncthreads();
    if (threadIdx.x < 256) s->hist[threadIdx.x] = 0;
}

// per unit: entries above tau and equal to tau among the non-floor positions
// (16-byte loads of four scores where the row allows them)
__global__ void __launch_bounds__(256)
unit_counts_kernel(const float *__restrict__ imp, int64_t n, int64_t nf, const SelState *s,
                   int64_t quota, int64_t *cgt, int64_t *ceq, const uint32_t *ckey, const int64_t *ccut) {
    __shared__ int64_t r1[256], r2[256];
    const int64_t h = blockIdx.x;
    const int t = threadIdx.x;
    const uint32_t key = s->prefix;
    const float *row = imp + h * n;
    int64_t a = 0, b = 0;
    auto one = [&](int64_t j, float x) {
        const uint32_t u = ord_key(x);
        const bool o = offered(ckey, ccut, h, j, u);
        a += o && (u > key);
        b += o && (u == key);
    };
    if (quota > 0) {
        int64_t j0 = 0;
        if ((n & 3) == 0) {
            const int64_t nv = nf / 4;   // whole groups of four non-floor positions
            for (int64_t g = t; g < nv; g += 256) {
                const float4 y = *(const float4 *)(row + 4 * g);
                one(4 * g, y.x);
                one(4 * g + 1, y.y);
                one(4 * g + 2, y.z);
                one(4 * g + 3, y.w);
            }
            j0 = 4 * nv;
        }
        for (int64_t j = j0 + t; j < nf; j += 256) one(j, row[j]);
    }
    a = block_reduce(a, r1, OpSum());
    b = block_reduce(b, r2, OpSum());
    if (t == 0) {
        cgt[h] = a;
        ceq[h] = b;
    }
}

// ties taken per unit, offsets, tau and the bytes held (one workgroup).  The
// units take the remaining ties in unit order: unit h takes
// clamp(rem - (ties of the units before it), 0, its ties), so both the ties
// taken and the offsets are prefix sums, formed 256 units at a time.
__device__ __forceinline__ int64_t block_excl_scan64(int64_t v, int64_t *buf, int64_t *total) {
    const int t = threadIdx.x, nt = blockDim.x;
    buf[t] = v;
    __syncthreads();
    for (int s2 = 1; s2 < nt; s2 <<= 1) {
        const int64_t add = (t >= s2) ? buf[t - s2] : 0;
        __syncthreads();
        buf[t] += add;
        __syncthreads();
    }
    const int64_t incl = buf[t];
    *total = buf[nt - 1];
    __syncthreads();
    return incl - v;
}

__global__ void __launch_bounds__(256)
unit_offsets_kernel(int64_t H, int64_t hpl, int64_t n, int64_t f, int64_t quota, const SelState *s,
                    const int64_t *cgt, const int64_t *ceq, int64_t *take, int64_t *offsets,
                    float *tau, int64_t *bytes_held, int64_t row_bytes) {
    __shared__ int64_t buf[256];
    __shared__ int64_t red[256];
    const int t = threadIdx.x;
    const int64_t rem = s->rem;
    int64_t eq_run = 0, acc = 0;   // ties and kept entries of the chunks before
    for (int64_t h0 = 0; h0 < H; h0 += 256) {
        const int64_t h = h0 + t;
        const int64_t e = (h < H && quota > 0) ? ceq[h] : 0;
        int64_t etot;
        const int64_t ebefore = eq_run + block_excl_scan64(e, buf, &etot);
        int64_t tk = 0;
        if (h < H && quota > 0) {
            const int64_t left = rem - ebefore;
            tk = left <= 0 ? 0 : (left < e ? left : e);
        }
        const int64_t c = (h < H) ? f + (quota > 0 ? cgt[h] : 0) + tk : 0;
        int64_t ctot;
        const int64_t cbefore = acc + block_excl_scan64(c, buf, &ctot);
        if (h < H) {
            take[h] = tk;
            offsets[h] = cbefore;
        }
        eq_run += etot;
        acc += ctot;
    }
    if (t == 0) offsets[H] = acc;
    if (t == 0 && tau) *tau = (quota > 0) ? key_to_float(s->prefix) : INFINITY;
    if (bytes_held) {
        __threadfence_block();
        __syncthreads();   // offsets of every unit are written
        int64_t padded = 0;
        for (int64_t l = t; l < H / hpl; l += 256) {
            int64_t mx = 0;
            for (int64_t h = l * hpl; h < (l + 1) * hpl; ++h) {
                const int64_t cc = offsets[h + 1] - offsets[h];
                mx = cc > mx ? cc : mx;
            }
            padded += mx * hpl;
        }
        padded = block_reduce(padded, red, OpSum());
        if (t == 0) {
            bytes_held[0] = acc * row_bytes;
            bytes_held[1] = padded * row_bytes;
            bytes_held[2] = H * n * row_bytes;
        }
    }
}

// per unit: kept positions ascending, and the dropped score mass.  The unit's
// scores are read in tiles of 16 consecutive positions per thread (16-byte
// loads: a wave reads whole lines), and one scan per tile places them.  Each
// thread's count of plain keeps (floor, or offered above the threshold key)
// and of offered keys equal to it share one word (16 bits each: a tile holds
// 4096 positions), and ties are kept in position order while the unit's
// quota of them lasts, so the number of ties kept before a thread follows
// from the ties before it.
__device__ __forceinline__ int keep_block_scan(int v, int *wsum, int *total) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6, nw = blockDim.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int before = 0, tot = 0;
    for (int i = 0; i < nw; ++i) {
        const int s = wsum[i];
        before += i < w ? s : 0;
        tot += s;
    }
    __syncthreads();   // wsum is reused by the next tile
    *total = tot;
    return before + x - v;
}

__global__ void __launch_bounds__(256)
unit_keep_kernel(const float *__restrict__ imp, int64_t n, int64_t f, int64_t quota,
                 const SelState *s, const int64_t *take, const int64_t *offsets, int32_t *kept_pos,
                 float *dropped, const uint32_t *ckey, const int64_t *ccut) {
    constexpr int PER = 16;
    __shared__ int wsum[4];
    __shared__ double red[256];
    const int64_t h = blockIdx.x;
    const int t = threadIdx.x;
    const uint32_t key = s->prefix;
    const int64_t tk = take[h];
    const int64_t nf = n - f;
    const float *row = imp + h * n;
    const bool vec = (n & 3) == 0;
    int64_t out = offsets[h];
    int64_t eq_run = 0;   // offered keys equal to the threshold key before this tile
    double dm = 0.0;
    for (int64_t base = 0; base < n; base += (int64_t)PER * 256) {
        const int64_t j0 = base + (int64_t)PER * t;
        float x[PER];
        if (vec && j0 + PER <= n) {
#pragma unroll
            for (int q = 0; q < PER / 4; ++q) {
                const float4 y = *(const float4 *)(row + j0 + 4 * q);
                x[4 * q] = y.x; x[4 * q + 1] = y.y; x[4 * q + 2] = y.z; x[4 * q + 3] = y.w;
            }
        } else {
#pragma unroll
            for (int e = 0; e < PER; ++e) x[e] = (j0 + e < n) ? row[j0 + e] : 0.f;
        }
        // 0: not kept, 1: kept, 2: an offered key equal to the threshold key
        uint32_t cls[PER];
        int cplain = 0, ctie = 0;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            const int64_t j = j0 + e;
            uint32_t c = 0;
            if (j < n) {
                if (j >= nf) {
                    c = 1;
                } else if (quota > 0) {
                    const uint32_t u = ord_key(x[e]);
                    if (offered(ckey, ccut, h, j, u)) c = u > key ? 1u : (u == key ? 2u : 0u);
                }
            }
            cls[e] = c;
            cplain += c == 1;
            ctie += c == 2;
        }
        int tot;
        const int pre = keep_block_scan(cplain | (ctie << 16), wsum, &tot);
        const int64_t rem = tk - eq_run;   // ties still to keep
        const int64_t tie_before = pre >> 16;
        int64_t tied_kept = rem <= 0 ? 0 : (tie_before < rem ? tie_before : rem);
        int64_t o = out + (pre & 0xFFFF) + tied_kept;
        int64_t tie_rank = eq_run + tie_before;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            bool keep = cls[e] == 1;
            if (cls[e] == 2) keep = tie_rank++ < tk;
            if (keep) kept_pos[o++] = (int32_t)(j0 + e);
            else if (j0 + e < n) dm += (double)x[e];
        }
        const int64_t tile_ties = tot >> 16;
        out += (tot & 0xFFFF) + (rem <= 0 ? 0 : (tile_ties < rem ? tile_ties : rem));
        eq_run += tile_ties;
    }
    dm = block_reduce(dm, red, OpSum());
    if (t == 0 && dropped) dropped[h] = (float)dm;
}

// gather kept rows: 16-byte pieces.  Block b copies part b % per of unit
// b / per, so each thread knows its unit without a search; one wave covers
// four rows of up to 256 bytes (16 lanes per row) per step.
__global__ void __launch_bounds__(256)
gather_rows_kernel(const char *__restrict__ k, const char *__restrict__ v, int64_t H, int64_t n,
                   int64_t row_bytes, const int64_t *offsets, const int32_t *kept_pos, char *k_out,
                   char *v_out, int per) {
    const int64_t h = blockIdx.x / per;
    const int part = blockIdx.x % per;
    const int64_t pieces = row_bytes / 16;
    const int64_t r0 = offsets[h], r1 = offsets[h + 1];
    const int64_t nwork = (r1 - r0) * pieces;
    const char *kh = k + h * n * row_bytes, *vh = v + h * n * row_bytes;
    for (int64_t w = (int64_t)part * blockDim.x + threadIdx.x; w < nwork; w += (int64_t)per * blockDim.x) {
        const int64_t row = r0 + w / pieces, pc = w % pieces;
        const int64_t src = (int64_t)kept_pos[row] * row_bytes + pc * 16;
        const int64_t dst = row * row_bytes + pc * 16;
        *(uint4 *)(k_out + dst) = *(const uint4 *)(kh + src);
        *(uint4 *)(v_out + dst) = *(const uint4 *)(vh + src);
    }
}

// same, any row size (byte copies), for rows that are not 16-byte multiples
__global__ void __launch_bounds__(256)
gather_bytes_kernel(const char *__restrict__ k, const char *__restrict__ v, int64_t H, int64_t n,
                    int64_t row_bytes, const int64_t *offsets, const int32_t *kept_pos, char *k_out,
                    char *v_out, int64_t total) {
    const int64_t nwork = total * row_bytes;
    for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < nwork;
         w += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = w / row_bytes, b = w % row_bytes;
        int64_t lo = 0, hi = H;
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) / 2;
            if (offsets[mid] <= row) lo = mid; else hi = mid;
        }
        const int64_t src = (lo * n + kept_pos[row]) * row_bytes + b;
        k_out[row * row_bytes + b] = k[src];
        v_out[row * row_bytes + b] = v[src];
    }
}

size_t compact_ws_bytes(int64_t H, int64_t n) {
    (void)n;
    return compact_layout(H, nullptr).bytes;
}

hipError_t launch_compact(int dtype, const void *k, const void *v, int64_t H, int64_t hpl, int64_t n,
                          int64_t d, const float *importance, int64_t budget, int floor, int64_t cap,
                          int64_t *offsets, int32_t *kept_pos, void *k_out, void *v_out, float *tau,
                          float *dropped, int64_t *bytes_held, void *ws, hipStream_t st) {
    CompactLayout L = compact_layout(H, ws);
    const int64_t f = floor < n ? floor : n;
    const int64_t nf = n - f;
    const int64_t quota = budget - H * f;
    // the per-unit candidate cut, when a cap leaves some non-floor key out
    const uint32_t *ckey = nullptr;
    const int64_t *ccut = nullptr;
    if (cap > 0 && cap - f < nf) {
        hipLaunchKernelGGL(unit_cap_kernel, dim3((unsigned)H), dim3(256), 0, st, importance, n, nf, cap - f, L.ckey,
                           L.ccut);
        ckey = L.ckey;
        ccut = L.ccut;
    }
    const int64_t elem = (dtype == FW_BF16) ? 2 : 4;
    const int64_t row_bytes = d * elem;
    hipLaunchKernelGGL(sel_init_kernel, dim3(1), dim3(256), 0, st, L.sel, quota);
    if (quota > 0) {
        // slices per unit so that the grid holds about 4096 blocks (a multiple of H)
        const int64_t per = (nf + 255) / 256;
        int64_t nsl = 4096 / H;
        if (nsl > per) nsl = per;
        if (nsl < 1) nsl = 1;
        const unsigned blocks = (unsigned)(H * nsl);
        for (int shift = 24; shift >= 0; shift -= 8) {
            hipLaunchKernelGGL(sel_hist_kernel, dim3(blocks), dim3(256), 0, st, importance, H, n, nf,
                               shift, L.sel, ckey, ccut);
            hipLaunchKernelGGL(sel_pick_kernel, dim3(1), dim3(256), 0, st, L.sel, shift);
        }
    }
    hipLaunchKernelGGL(unit_counts_kernel, dim3((unsigned)H), dim3(256), 0, st, importance, n, nf,
                       L.sel, quota, L.cgt, L.ceq, ckey, ccut);
    hipLaunchKernelGGL(unit_offsets_kernel, dim3(1), dim3(256), 0, st, H, hpl, n, f, quota, L.sel,
                       L.cgt, L.ceq, L.take, offsets, tau, bytes_held, 2 * row_bytes);
    hipLaunchKernelGGL(unit_keep_kernel, dim3((unsigned)H), dim3(256), 0, st, importance, n, f, quota,
                       L.sel, L.take, offsets, kept_pos, dropped, ckey, ccut);
    if (budget > 0) {
        if (row_bytes % 16 == 0) {
            // blocks per unit: about the unit's average share of 16 K blocks
            const int64_t work = budget * (row_bytes / 16);
            int64_t per = (work + 255) / 256 / H;
            per = per < 1 ? 1 : (per > 1024 ? 1024 : per);
            if (H * per > (int64_t)1 << 30) per = 1;
            hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)(H * per)), dim3(256), 0, st, (const char *)k,
                               (const char *)v, H, n, row_bytes, offsets, kept_pos, (char *)k_out,
                               (char *)v_out, (int)per);
        } else {
            const int64_t work = budget * row_bytes;
            const unsigned blocks = (unsigned)((work + 255) / 256 < 65536 ? (work + 255) / 256 : 65536);
            hipLaunchKernelGGL(gather_bytes_kernel, dim3(blocks), dim3(256), 0, st, (const char *)k,
                               (const char *)v, H, n, row_bytes, offsets, kept_pos, (char *)k_out,
                               (char *)v_out, budget);
        }
    }
    return hipGetLastError();
}

hipError_t launch_maxpool(const float *scores, int64_t H, int64_t n, int kernel, float *out, hipStream_t st) {
    const int64_t total = H * n;
    const unsigned blocks = (unsigned)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
    hipLaunchKernelGGL(maxpool_kernel, dim3(blocks), dim3(256), 0, st, scores, H, n, kernel / 2, out);
    return hipGetLastError();
}

}  // namespace fw
