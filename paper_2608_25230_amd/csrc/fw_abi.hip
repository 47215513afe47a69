// C ABI of libfw: argument validation, workspace layout and launch order.
// No entry point allocates device memory, synchronises or copies to the host.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "fw_internal.hpp"

// Scratch space of fw_dense_topk_noalloc: one copy per GPU, allocated with the
// code object and held until the process ends.  In host code this name only
// stands in for the symbol; kernels and copies use the per-device address
// taken from hipGetSymbolAddress below, never the name itself.
static __device__ __align__(256) unsigned char scratch[FW_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512] = "";

fw_status fail(fw_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

fw_status hip_status(hipError_t e, const char *where) {
    if (e == hipSuccess) return FW_OK;
    return fail(FW_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

// Sequential carve-out of the caller's workspace in 256-byte aligned pieces.
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *b) : base((char *)b) {}
    template <typename T> T *take(size_t count) {
        off = fw::align_up(off, 256);
        T *p = base ? (T *)(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
    size_t size() const { return fw::align_up(off, 256); }
};

fw_status check_rows(const fw_rows *rows, bool need_v) {
    if (!rows) return fail(FW_E_NULL, "rows is NULL");
    if (rows->dtype != FW_F32 && rows->dtype != FW_BF16)
        return fail(FW_E_DTYPE, "unknown dtype %d", (int)rows->dtype);
    if (!rows->q || !rows->k) return fail(FW_E_NULL, "rows->q or rows->k is NULL");
    if (need_v && !rows->v) return fail(FW_E_NULL, "rows->v is NULL");
    if (rows->H < 1 || rows->G < 1 || rows->n < 1)
        return fail(FW_E_SHAPE, "H, G, n must be >= 1 (H=%lld G=%lld n=%lld)", (long long)rows->H,
                    (long long)rows->G, (long long)rows->n);
    if (rows->d < 1 || rows->d > 256) return fail(FW_E_SHAPE, "d must be in [1, 256], got %lld", (long long)rows->d);
    if (rows->n > (1ll << 30)) return fail(FW_E_SHAPE, "n must be <= 2^30");
    if (rows->H > (1ll << 31) / rows->G) return fail(FW_E_SHAPE, "H*G must be < 2^31");
    const double hgn = (double)rows->H * (double)rows->G * (double)rows->n;
    if (hgn >= 1099511627776.0) return fail(FW_E_SHAPE, "H*G*n must be < 2^40");
    return FW_OK;
}

fw_status check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (need && !ws) return fail(FW_E_WORKSPACE, "workspace is NULL, %zu bytes needed", need);
    if (ws_bytes < need) return fail(FW_E_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
    return FW_OK;
}

// ---------------------------------------------------------------------------
// fw_dense_topk
// ---------------------------------------------------------------------------
fw_status parse_ks(const fw_rows *rows, const int32_t *ks, int32_t n_ks, fw::KsArg *out) {
    if (!ks) return fail(FW_E_NULL, "ks is NULL");
    if (n_ks < 1 || n_ks > FW_MAX_KS) return fail(FW_E_SHAPE, "n_ks must be in [1, %d]", FW_MAX_KS);
    int idx[FW_MAX_KS];
    for (int i = 0; i < n_ks; ++i) {
        if (ks[i] < 1 || ks[i] > rows->n)
            return fail(FW_E_SHAPE, "ks[%d] = %d outside [1, n=%lld]", i, ks[i], (long long)rows->n);
        idx[i] = i;
    }
    std::sort(idx, idx + n_ks, [&](int a, int b) { return ks[a] < ks[b]; });
    out->n = n_ks;
    for (int t = 0; t < n_ks; ++t) {
        if (t && ks[idx[t]] == ks[idx[t - 1]]) return fail(FW_E_SHAPE, "ks must be distinct");
        out->k[t] = ks[idx[t]];
        out->perm[t] = idx[t];
    }
    for (int t = n_ks; t < FW_MAX_KS; ++t) { out->k[t] = 0; out->perm[t] = 0; }
    return FW_OK;
}

struct DenseTopkWs {
    float *z, *row_m, *row_l;
    uint32_t *thr_key;
    int32_t *thr_cut;
    size_t bytes;
};

DenseTopkWs dense_topk_layout(const fw_rows *rows, int n_ks, void *ws) {
    Carve c(ws);
    const size_t R = (size_t)rows->H * rows->G;
    DenseTopkWs w;
    w.z = c.take<float>(R * rows->n);
    w.row_m = c.take<float>(R);
    w.row_l = c.take<float>(R);
    w.thr_key = c.take<uint32_t>(R * n_ks);
    w.thr_cut = c.take<int32_t>(R * n_ks);
    w.bytes = c.size();
    return w;
}

// ---------------------------------------------------------------------------
// argument checks of the other entry points
// ---------------------------------------------------------------------------
fw_status check_best_subset(const fw_rows *rows, int32_t k) {
    fw_status s = check_rows(rows, true);
    if (s != FW_OK) return s;
    if (k < 1 || k > rows->n) return fail(FW_E_SHAPE, "k = %d outside [1, n=%lld]", k, (long long)rows->n);
    if (rows->n > 64) return fail(FW_E_UNSUPPORTED, "exhaustive enumeration needs n <= 64 (n=%lld)", (long long)rows->n);
    if (fw::binom((int)rows->n, k) >= (1ull << 31))
        return fail(FW_E_UNSUPPORTED, "C(n=%lld, k=%d) must be < 2^31", (long long)rows->n, k);
    if (!fw::best_subset_plannable(rows->n, k))
        return fail(FW_E_UNSUPPORTED, "no enumeration plan fits for n=%lld, k=%d", (long long)rows->n, k);
    return FW_OK;
}

fw_status check_swap(const fw_rows *rows, int32_t k, int32_t max_iters) {
    fw_status s = check_rows(rows, true);
    if (s != FW_OK) return s;
    if (k < 1 || k > rows->n) return fail(FW_E_SHAPE, "k = %d outside [1, n=%lld]", k, (long long)rows->n);
    if (max_iters < 0 || max_iters > 4096) return fail(FW_E_SHAPE, "max_iters must be in [0, 4096]");
    if (rows->n > 64 && rows->H * rows->G > 65535)
        return fail(FW_E_UNSUPPORTED, "rows longer than 64 keys: at most 65535 rows per call");
    return FW_OK;
}

fw_status check_compact(int32_t dtype, const void *k, const void *v, int64_t H, int64_t hpl, int64_t n,
                        int64_t d, const float *importance, int64_t budget, int32_t floor, int64_t cap) {
    if (dtype != FW_F32 && dtype != FW_BF16) return fail(FW_E_DTYPE, "unknown dtype %d", (int)dtype);
    if (!k || !v || !importance) return fail(FW_E_NULL, "k, v and importance are required");
    if (H < 1 || n < 1 || d < 1 || d > 4096) return fail(FW_E_SHAPE, "need H >= 1, n >= 1, 1 <= d <= 4096");
    if (n > (1ll << 30) || (double)H * (double)n >= 1099511627776.0) return fail(FW_E_SHAPE, "H*n too large");
    if (hpl < 1 || H % hpl != 0) return fail(FW_E_SHAPE, "heads_per_layer must divide H");
    if (floor < 0) return fail(FW_E_SHAPE, "recency_floor must be >= 0");
    const int64_t f = floor < n ? floor : n;
    if (cap < 0 || (cap > 0 && cap < f))
        return fail(FW_E_SHAPE, "cap must be 0 (none) or >= min(recency_floor, n), got %lld", (long long)cap);
    const int64_t per_cell = (cap > 0 && cap < n) ? cap : n;
    if (budget < H * f || budget > H * per_cell)
        return fail(FW_E_SHAPE, "budget_entries %lld outside [H*floor, H*min(cap, n)] = [%lld, %lld]",
                    (long long)budget, (long long)(H * f), (long long)(H * per_cell));
    if (budget >= (1ll << 31)) return fail(FW_E_SHAPE, "budget_entries must be < 2^31");
    return FW_OK;
}

fw_status check_pool(const fw_rows *rows, int32_t n_budgets, const int32_t *s, const int32_t *extra,
                     int32_t max_swaps) {
    fw_status st = check_rows(rows, true);
    if (st != FW_OK) return st;
    if (!s || !extra) return fail(FW_E_NULL, "s and extra are required");
    if (n_budgets < 1 || n_budgets > FW_POOL_MAX_BUDGETS)
        return fail(FW_E_SHAPE, "n_budgets must be in [1, %d]", FW_POOL_MAX_BUDGETS);
    for (int b = 0; b < n_budgets; ++b) {
        if (s[b] < 1 || extra[b] < 0 || (int64_t)s[b] + extra[b] > rows->n)
            return fail(FW_E_SHAPE, "budget %d: need 1 <= s, 0 <= extra, s + extra <= n (s=%d extra=%d n=%lld)", b,
                        s[b], extra[b], (long long)rows->n);
        if (s[b] + extra[b] > 64) return fail(FW_E_UNSUPPORTED, "budget %d: s + extra = %d > 64 pool keys", b, s[b] + extra[b]);
    }
    if (max_swaps < 0 || max_swaps > 4096) return fail(FW_E_SHAPE, "max_swaps must be in [0, 4096]");
    if (rows->n > 8192) return fail(FW_E_UNSUPPORTED, "n = %lld > 8192 for the candidate-set search", (long long)rows->n);
    if (!fw::pool_plannable(rows->n, (int)rows->d, n_budgets, s, extra))
        return fail(FW_E_UNSUPPORTED, "no enumeration plan for these budgets within the limits");
    return FW_OK;
}

}  // namespace

extern "C" {

const char *fw_last_error(void) { return g_err; }
const char *fw_version(void) { return "libfw 0.1 (gfx950)"; }

size_t dense_topk_ws_bytes(const fw_rows *rows, const fw::KsArg &k) {
    if (fw::mp_topk_supported(*rows, k) || fw::fused_topk_supported(*rows, k))
        return fw::fused_topk_ws_bytes(*rows, k.k[k.n - 1]);
    return dense_topk_layout(rows, k.n, nullptr).bytes;
}

size_t fw_dense_topk_workspace_size(const fw_rows *rows, const int32_t *ks, int32_t n_ks) {
    fw::KsArg k;
    if (check_rows(rows, true) != FW_OK || parse_ks(rows, ks, n_ks, &k) != FW_OK) return 0;
    return dense_topk_ws_bytes(rows, k);
}

}  // extern "C"

namespace {

fw_status check_dense_topk(const fw_rows *rows, const int32_t *ks, int32_t n_ks, const float *gap,
                           const float *dropped, const int32_t *topk_idx, fw::KsArg *k) {
    fw_status s = check_rows(rows, true);
    if (s != FW_OK) return s;
    if ((s = parse_ks(rows, ks, n_ks, k)) != FW_OK) return s;
    if (!gap || !dropped) return fail(FW_E_NULL, "gap and dropped are required");
    if (topk_idx && k->k[k->n - 1] > 16384) return fail(FW_E_UNSUPPORTED, "topk_idx needs kmax <= 16384");
    return FW_OK;
}

// Launches of fw_dense_topk once the arguments and the workspace are checked.
fw_status dense_topk_launch(const fw_rows *rows, const fw::KsArg &k, float *o, float *o_s, float *gap,
                            float *dropped, int32_t *topk_idx, void *ws, hipStream_t st) {
    const int kmax = k.k[k.n - 1];
    const int n_ks = k.n;
    if (fw::mp_topk_supported(*rows, k))
        return hip_status(fw::launch_mp_topk(*rows, k, o, o_s, gap, dropped, topk_idx, ws, st), "fw_dense_topk");
    if (fw::fused_topk_supported(*rows, k))
        return hip_status(fw::launch_fused_topk(*rows, k, o, o_s, gap, dropped, topk_idx, ws, st),
                          "fw_dense_topk");
    const DenseTopkWs w = dense_topk_layout(rows, n_ks, ws);
    const int64_t H = rows->H, G = rows->G, n = rows->n;
    const int d = (int)rows->d;
    hipError_t e = fw::launch_scores(rows->dtype, rows->q, rows->k, rows->scale, rows->bias, H, G, n,
                                     d, w.z, st);
    if (e == hipSuccess)
        e = fw::launch_select(w.z, H * G, n, k, w.row_m, w.row_l, w.thr_key, w.thr_cut, topk_idx,
                              kmax, st);
    if (e == hipSuccess)
        e = fw::launch_tiers(rows->dtype, rows->v, w.z, w.row_m, w.row_l, w.thr_key, w.thr_cut, H,
                             G, n, d, k, o, o_s, gap, dropped, st);
    return hip_status(e, "fw_dense_topk");
}

// Per-device address of `scratch`, taken once per device with that device
// current (every GPU holds its own copy at its own address).
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchDevices];

fw_status scratch_address(hipStream_t st, void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "fw_dense_topk_noalloc: hipGetDevice");
    if (st) {
        int sdev = -1;
        if ((e = hipStreamGetDevice(st, &sdev)) != hipSuccess)
            return hip_status(e, "fw_dense_topk_noalloc: hipStreamGetDevice");
        if (sdev != dev)
            return fail(FW_E_UNSUPPORTED, "stream belongs to device %d but device %d is current", sdev, dev);
    }
    if (dev < 0 || dev >= kScratchDevices)
        return fail(FW_E_UNSUPPORTED, "device %d is beyond the %d devices the scratch table holds", dev,
                    kScratchDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
            return hip_status(e, "fw_dense_topk_noalloc: hipGetSymbolAddress");
        if (!p) return fail(FW_E_HIP, "fw_dense_topk_noalloc: no device address for the scratch array");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return FW_OK;
}

}  // namespace

extern "C" {

fw_status fw_dense_topk(const fw_rows *rows, const int32_t *ks, int32_t n_ks, float *o, float *o_s,
                        float *gap, float *dropped, int32_t *topk_idx, void *ws, size_t ws_bytes,
                        fw_stream stream) {
    fw::KsArg k;
    fw_status s = check_dense_topk(rows, ks, n_ks, gap, dropped, topk_idx, &k);
    if (s != FW_OK) return s;
    if ((s = check_ws(ws, ws_bytes, dense_topk_ws_bytes(rows, k))) != FW_OK) return s;
    return dense_topk_launch(rows, k, o, o_s, gap, dropped, topk_idx, ws, (hipStream_t)stream);
}

fw_status fw_dense_topk_noalloc(const fw_rows *rows, const int32_t *ks, int32_t n_ks, float *o, float *o_s,
                                float *gap, float *dropped, int32_t *topk_idx, fw_stream stream) {
    fw::KsArg k;
    fw_status s = check_dense_topk(rows, ks, n_ks, gap, dropped, topk_idx, &k);
    if (s != FW_OK) return s;
    const size_t need = dense_topk_ws_bytes(rows, k);
    if (need > FW_NOALLOC_SCRATCH_BYTES)
        return fail(FW_E_UNSUPPORTED,
                    "fw_dense_topk_noalloc: this call needs %zu bytes of scratch, more than the %zu the "
                    "library holds per device (use fw_dense_topk with a workspace)",
                    need, (size_t)FW_NOALLOC_SCRATCH_BYTES);
    hipStream_t st = (hipStream_t)stream;
    void *ws = nullptr;
    if ((s = scratch_address(st, &ws)) != FW_OK) return s;
    return dense_topk_launch(rows, k, o, o_s, gap, dropped, topk_idx, ws, st);
}

// ---------------------------------------------------------------------------
size_t fw_best_subset_workspace_size(const fw_rows *rows, int32_t k) {
    if (check_best_subset(rows, k) != FW_OK) return 0;
    return fw::best_subset_ws_bytes(rows->n, k);
}

fw_status fw_best_subset(const fw_rows *rows, int32_t k, int32_t *best_idx, float *best_gap,
                         float *topk_gap, float *closed, float *dropped_topk, int32_t *topk_idx,
                         void *ws, size_t ws_bytes, fw_stream stream) {
    fw_status s = check_best_subset(rows, k);
    if (s != FW_OK) return s;
    if (!best_idx || !best_gap) return fail(FW_E_NULL, "best_idx and best_gap are required");
    if ((s = check_ws(ws, ws_bytes, fw::best_subset_ws_bytes(rows->n, k))) != FW_OK) return s;
    hipError_t e = fw::launch_best_subset(*rows, k, best_idx, best_gap, topk_gap, closed,
                                          dropped_topk, topk_idx, ws, (hipStream_t)stream);
    return hip_status(e, "fw_best_subset");
}

// ---------------------------------------------------------------------------
size_t fw_pool_subset_workspace_size(const fw_rows *rows, int32_t n_budgets, const int32_t *s,
                                     const int32_t *extra) {
    if (check_pool(rows, n_budgets, s, extra, 0) != FW_OK) return 0;
    return fw::pool_ws_bytes(*rows, n_budgets, s, extra);
}

fw_status fw_pool_subset(const fw_rows *rows, int32_t n_budgets, const int32_t *s, const int32_t *extra,
                         int32_t max_swaps, int32_t fw_iters, int32_t *pool_idx, int32_t *best_idx,
                         int32_t *bal_idx, int32_t *geo_idx, int32_t *n_swaps, float *stats, float flat_threshold,
                         float *cell_median, uint8_t *cell_flat, void *ws, size_t ws_bytes, fw_stream stream) {
    fw_status st = check_pool(rows, n_budgets, s, extra, max_swaps);
    if (st != FW_OK) return st;
    if (fw_iters < 0 || fw_iters > 4096) return fail(FW_E_SHAPE, "fw_iters must be in [0, 4096]");
    if (!best_idx || !stats) return fail(FW_E_NULL, "best_idx and stats are required");
    if ((st = check_ws(ws, ws_bytes, fw::pool_ws_bytes(*rows, n_budgets, s, extra))) != FW_OK) return st;
    hipError_t e = fw::launch_pool(*rows, n_budgets, s, extra, max_swaps, fw_iters, pool_idx, best_idx, bal_idx,
                                   geo_idx, n_swaps, stats, flat_threshold, cell_median, cell_flat, ws,
                                   (hipStream_t)stream);
    return hip_status(e, "fw_pool_subset");
}

// ---------------------------------------------------------------------------
size_t fw_swap_workspace_size(const fw_rows *rows, int32_t k, int32_t max_iters) {
    if (check_swap(rows, k, max_iters) != FW_OK) return 0;
    return fw::swap_ws_bytes(*rows, k, max_iters);
}

fw_status fw_swap(const fw_rows *rows, int32_t k, int32_t max_iters, int32_t *s_idx, float *gap_traj,
                  int32_t *n_swaps, float *dropped, void *ws, size_t ws_bytes, fw_stream stream) {
    fw_status s = check_swap(rows, k, max_iters);
    if (s != FW_OK) return s;
    if (!s_idx || !gap_traj || !n_swaps) return fail(FW_E_NULL, "s_idx, gap_traj and n_swaps are required");
    if ((s = check_ws(ws, ws_bytes, fw::swap_ws_bytes(*rows, k, max_iters))) != FW_OK) return s;
    hipError_t e = fw::launch_swap(*rows, k, max_iters, s_idx, gap_traj, n_swaps, dropped, ws,
                                   (hipStream_t)stream);
    return hip_status(e, "fw_swap");
}

// ---------------------------------------------------------------------------
size_t fw_dropped_mass_curve_workspace_size(const fw_rows *rows) {
    if (check_rows(rows, false) != FW_OK) return 0;
    return fw::curve_ws_bytes(*rows);
}

fw_status fw_dropped_mass_curve(const fw_rows *rows, float *importance, float *curve, int32_t *order,
                                void *ws, size_t ws_bytes, fw_stream stream) {
    fw_status s = check_rows(rows, false);
    if (s != FW_OK) return s;
    if (!importance || !curve) return fail(FW_E_NULL, "importance and curve are required");
    if ((s = check_ws(ws, ws_bytes, fw::curve_ws_bytes(*rows))) != FW_OK) return s;
    hipError_t e = fw::launch_curve(*rows, importance, curve, order, ws, (hipStream_t)stream);
    return hip_status(e, "fw_dropped_mass_curve");
}

// ---------------------------------------------------------------------------
size_t fw_ragged_compact_workspace_size(int64_t H, int64_t n, int64_t d, int64_t budget_entries) {
    if (H < 1 || n < 1 || d < 1 || budget_entries < 0) return 0;
    return fw::compact_ws_bytes(H, n);
}

fw_status fw_ragged_compact(int32_t dtype, const void *k, const void *v, int64_t H, int64_t heads_per_layer,
                            int64_t n, int64_t d, const float *importance, int64_t budget_entries,
                            int32_t recency_floor, int64_t cap, int64_t *offsets, int32_t *kept_pos,
                            void *k_out, void *v_out, float *tau, float *dropped, int64_t *bytes_held, void *ws,
                            size_t ws_bytes, fw_stream stream) {
    fw_status s = check_compact(dtype, k, v, H, heads_per_layer, n, d, importance, budget_entries,
                                recency_floor, cap);
    if (s != FW_OK) return s;
    if (!offsets || !kept_pos || !k_out || !v_out)
        return fail(FW_E_NULL, "offsets, kept_pos, k_out and v_out are required");
    if ((s = check_ws(ws, ws_bytes, fw::compact_ws_bytes(H, n))) != FW_OK) return s;
    hipError_t e = fw::launch_compact(dtype, k, v, H, heads_per_layer, n, d, importance,
                                      budget_entries, recency_floor, cap, offsets, kept_pos, k_out, v_out,
                                      tau, dropped, bytes_held, ws, (hipStream_t)stream);
    return hip_status(e, "fw_ragged_compact");
}

fw_status fw_maxpool_scores(const float *scores, int64_t H, int64_t n, int32_t kernel, float *out,
                            fw_stream stream) {
    if (!scores || !out) return fail(FW_E_NULL, "scores and out are required");
    if (H < 1 || n < 1 || (double)H * (double)n >= 1099511627776.0) return fail(FW_E_SHAPE, "need H, n >= 1, H*n < 2^40");
    if (kernel < 1 || kernel % 2 == 0 || kernel > 1023) return fail(FW_E_SHAPE, "kernel must be odd, 1..1023");
    if (scores == out && kernel > 1) return fail(FW_E_SHAPE, "out must not alias scores");
    return hip_status(fw::launch_maxpool(scores, H, n, kernel, out, (hipStream_t)stream), "fw_maxpool_scores");
}

// ---------------------------------------------------------------------------
size_t fw_group_vote_workspace_size(const fw_rows *rows, int32_t s, int32_t group_size) {
    (void)rows;
    (void)s;
    (void)group_size;
    return 0;
}

fw_status fw_group_vote(const fw_rows *rows, int32_t s, int32_t group_size, int32_t *vote_idx, float *es_vote,
                        float *es_top, float *dropped, void *ws, size_t ws_bytes, fw_stream stream) {
    (void)ws;
    (void)ws_bytes;
    fw_status st = check_rows(rows, true);
    if (st != FW_OK) return st;
    if (group_size < 1 || rows->G % group_size != 0)
        return fail(FW_E_SHAPE, "group_size must divide G (G=%lld group_size=%d)", (long long)rows->G, group_size);
    if (s < 1 || s > rows->n) return fail(FW_E_SHAPE, "s must be in [1, n=%lld], got %d", (long long)rows->n, s);
    if (s > 256) return fail(FW_E_UNSUPPORTED, "s = %d > 256", s);
    if (!fw::vote_supported(*rows, s, group_size))
        return fail(FW_E_UNSUPPORTED, "n, d and the group size need more than 160 KiB of LDS");
    if (!vote_idx || !es_vote || !es_top) return fail(FW_E_NULL, "vote_idx, es_vote and es_top are required");
    hipError_t e = fw::launch_vote(*rows, s, group_size, vote_idx, es_vote, es_top, dropped, (hipStream_t)stream);
    return hip_status(e, "fw_group_vote");
}

}  // extern "C"

