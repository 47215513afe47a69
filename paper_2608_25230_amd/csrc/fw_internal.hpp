// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include "fw_common.hpp"

namespace fw {

// Budgets of one fw_dense_topk call, sorted ascending; perm[t] is the
// caller's position of the t-th smallest budget.
struct KsArg {
    int n;
    int k[FW_MAX_KS];
    int perm[FW_MAX_KS];
};

// k_topk.hip
hipError_t launch_scores(int dtype, const void *q, const void *k, const float *scale,
                         const float *bias, int64_t H, int64_t G, int64_t n, int d, float *z,
                         hipStream_t st);
hipError_t launch_select(const float *z, int64_t R, int64_t n, const KsArg &ks, float *row_m,
                         float *row_l, uint32_t *thr_key, int32_t *thr_cut, int32_t *topk_idx,
                         int kmax, hipStream_t st);
hipError_t launch_tiers(int dtype, const void *v, const float *z, const float *row_m,
                        const float *row_l, const uint32_t *thr_key, const int32_t *thr_cut,
                        int64_t H, int64_t G, int64_t n, int d, const KsArg &ks, float *o,
                        float *o_s, float *gap, float *dropped, hipStream_t st);

// k_topk_fused.hip -- one-kernel path for bf16, d = 128, n in {1024, 2048, 4096}
bool fused_topk_supported(const fw_rows &rows, const KsArg &ks);
size_t fused_topk_ws_bytes(const fw_rows &rows, int kmax);
hipError_t launch_fused_topk(const fw_rows &rows, const KsArg &ks, float *o, float *o_s, float *gap,
                             float *dropped, int32_t *topk_idx, void *ws, hipStream_t st);

// k_topk_mp.hip -- multi-pass one-kernel path for bf16, d = 128, n a multiple
// of 32 up to 4096, 128 rows per unit tile (same workspace as the fused path)
bool mp_topk_supported(const fw_rows &rows, const KsArg &ks);
hipError_t launch_mp_topk(const fw_rows &rows, const KsArg &ks, float *o, float *o_s, float *gap,
                          float *dropped, int32_t *topk_idx, void *ws, hipStream_t st);

// k_subset.hip -- exhaustive best subset (float64)
size_t best_subset_ws_bytes(int64_t n, int k);
bool best_subset_plannable(int64_t n, int k);
hipError_t launch_best_subset(const fw_rows &rows, int k, int32_t *best_idx, float *best_gap,
                              float *topk_gap, float *closed, float *dropped_topk,
                              int32_t *topk_idx, void *ws, hipStream_t st);

// k_pool.hip -- candidate-set search (ES_pool, pool balancing, certificate)
bool pool_plannable(int64_t N, int d, int nb, const int32_t *s, const int32_t *extra);
size_t pool_ws_bytes(const fw_rows &rows, int nb, const int32_t *s, const int32_t *extra);
hipError_t launch_pool(const fw_rows &rows, int nb, const int32_t *s, const int32_t *extra, int max_swaps,
                       int fw_iters, int32_t *pool_idx, int32_t *best_idx, int32_t *bal_idx, int32_t *geo_idx,
                       int32_t *n_swaps, float *stats,
                       float flat_threshold, float *cell_median, uint8_t *cell_flat, void *ws, hipStream_t st);

// k_vote.hip -- group vote
bool vote_supported(const fw_rows &rows, int s, int gs);
hipError_t launch_vote(const fw_rows &rows, int s, int gs, int32_t *vote_idx, float *es_vote, float *es_top,
                       float *dropped, hipStream_t st);

// k_swap.hip -- swap rule
size_t swap_ws_bytes(const fw_rows &rows, int k, int max_iters);
hipError_t launch_swap(const fw_rows &rows, int k, int max_iters, int32_t *s_idx, float *gap_traj,
                       int32_t *n_swaps, float *dropped, void *ws, hipStream_t st);

// k_curve.hip -- window importance and dropped-mass curve
size_t curve_ws_bytes(const fw_rows &rows);
hipError_t launch_curve(const fw_rows &rows, float *importance, float *curve, int32_t *order,
                        void *ws, hipStream_t st);

// k_window.hip -- window importance on MFMA (bf16, d = 128, 16..64 rows)
bool window_mfma_supported(const fw_rows &rows);
void launch_window_mfma(const fw_rows &rows, float *part_m, float *part_l, float *row_m, float *row_il,
                        float *importance, hipStream_t st);

// k_compact.hip -- global allocation and ragged compaction
size_t compact_ws_bytes(int64_t H, int64_t n);
hipError_t launch_compact(int dtype, const void *k, const void *v, int64_t H, int64_t hpl,
                          int64_t n, int64_t d, const float *importance, int64_t budget,
                          int floor, int64_t cap, int64_t *offsets, int32_t *kept_pos, void *k_out,
                          void *v_out, float *tau, float *dropped, int64_t *bytes_held, void *ws,
                          hipStream_t st);
hipError_t launch_maxpool(const float *scores, int64_t H, int64_t n, int kernel, float *out, hipStream_t st);

}  // namespace fw
