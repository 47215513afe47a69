/*
 * fw.h -- C ABI of libfw: forced-weight subset evaluation over attention rows
 * on AMD Instinct MI355X (gfx950).
 *
 * The operations follow "Trust the Mass: Forced Weights in KV-Cache Eviction"
 * (arXiv 2608.25230).  An instance (Definition 2.1) is one attention query row:
 * weights p = softmax(z), z_j = scale * <q, k_j> + bias_j, values v_j, dense
 * output mu = sum_j p_j v_j.  A kept set S with mass p(S) gives the forced
 * output m_S = sum_{j in S} (p_j / p(S)) v_j, the gap es(S) = ||m_S - mu||_2 and
 * the dropped mass 1 - p(S).
 *
 * Conventions shared by every entry point
 *   - All array pointers are DEVICE pointers to contiguous row-major buffers
 *     unless marked "host".  The caller owns every buffer; the library keeps
 *     no pointer after a call returns and no call allocates device memory:
 *     scratch space is the caller's workspace, sized by the matching
 *     fw_*_workspace_size() query (which returns 0 for invalid arguments),
 *     or, for fw_dense_topk_noalloc, a static per-device array.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default
 *     stream).  No call synchronises the device or copies device data to the
 *     host; results are valid once the stream reaches them.
 *   - Validation happens before anything is enqueued: on any error status no
 *     output has been written.  fw_last_error() returns a thread-local message
 *     describing the last failure of the calling thread.
 *   - Rows are grouped in units of H key/value sets with G query rows each
 *     (grouped-query attention: the G rows of unit h share k[h], v[h]); row r
 *     = h*G + g, R = H*G rows in total.
 *   - Ties: the top-k set ranks keys by logit descending, then key index
 *     ascending.  Equal-error best subsets resolve to the lexicographically
 *     smallest ascending index tuple; equal swaps to the smallest (out, in).
 *   - Results are bitwise repeatable across calls on the same device.
 */
#ifndef FW_H
#define FW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fw_status {
    FW_OK = 0,
    FW_E_NULL = 1,        /* a required pointer is NULL                       */
    FW_E_SHAPE = 2,       /* a size is out of range or inconsistent           */
    FW_E_DTYPE = 3,       /* unknown element type                             */
    FW_E_UNSUPPORTED = 4, /* valid request this build does not handle         */
    FW_E_WORKSPACE = 5,   /* workspace NULL or smaller than the size query    */
    FW_E_HIP = 6          /* the HIP runtime reported an error at launch      */
} fw_status;

typedef enum fw_dtype {
    FW_F32 = 0,  /* IEEE float32                        */
    FW_BF16 = 1  /* bfloat16 (upper half of a float32)  */
} fw_dtype;

/* A hipStream_t, passed opaquely so that C callers need no HIP headers. */
typedef void *fw_stream;

/* A batch of attention rows (Definition 2.1 in attention form).
 *   q     [H][G][d]  query rows, element type `dtype`
 *   k, v  [H][n][d]  keys and values of each unit, element type `dtype`;
 *                    v may be NULL for fw_dropped_mass_curve
 *   scale [H] float32 logit scale per unit, or NULL for 1/sqrt(d)
 *   bias  [n] float32 additive logit bias shared by every row, or NULL
 * Limits: H, G >= 1; 1 <= n <= 2^30; 1 <= d <= 256; H*G*n < 2^40.
 * The paper's worked examples (a given p) are reached with q = 0 and
 * bias = log p. */
typedef struct fw_rows {
    int32_t dtype;
    const void *q;
    const void *k;
    const void *v;
    int64_t H, G, n, d;
    const float *scale;
    const float *bias;
} fw_rows;

#define FW_MAX_KS 8

/* ---------------------------------------------------------------------------
 * fw_dense_topk -- top-k forced-weight evaluation of every row
 * (Definition 2.1; the gap is evaluated through Lemma 2.2's first form
 * es(S) = (1 - p(S)) * ||m_{S^c} - m_S|| so that it stays accurate when the
 * dropped mass is small).
 *   ks        host [n_ks] budgets, each 1 <= k <= n, 1 <= n_ks <= FW_MAX_KS,
 *             pairwise distinct, any order; outputs follow this order
 *   o         [H][G][d] float32 dense output mu, or NULL
 *   o_s       [n_ks][H][G][d] float32 forced output of each top-k set, or NULL
 *   gap       [n_ks][H][G] float32 ||o_s - o||_2 (required)
 *   dropped   [n_ks][H][G] float32 dropped mass 1 - p(S) (required)
 *   topk_idx  [H][G][kmax] int32 top-kmax keys in rank order (logit
 *             descending, index ascending), kmax = max(ks); or NULL.  The
 *             top-k set of a smaller budget is the first k entries.
 * Errors: FW_E_NULL (rows, q, k, v, gap, dropped or ks NULL), FW_E_SHAPE,
 * FW_E_DTYPE, FW_E_WORKSPACE, FW_E_UNSUPPORTED (topk_idx with kmax > 16384),
 * FW_E_HIP.
 * ------------------------------------------------------------------------- */
size_t fw_dense_topk_workspace_size(const fw_rows *rows, const int32_t *ks, int32_t n_ks);
fw_status fw_dense_topk(const fw_rows *rows, const int32_t *ks, int32_t n_ks,
                        float *o, float *o_s, float *gap, float *dropped,
                        int32_t *topk_idx, void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_dense_topk_noalloc -- fw_dense_topk for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same operation, arguments, outputs, kernels and
 * results as fw_dense_topk, without the workspace arguments.  Its scratch
 * space is a static device array of FW_NOALLOC_SCRATCH_BYTES bytes that the
 * library holds on every GPU it runs on until the process ends; the call
 * allocates nothing, and it clears what must start at zero with a kernel (no
 * memset).  `stream` must belong to the current device.
 * Calls on one GPU share that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (several streams or host threads)
 * race and must be serialised by the caller.
 * Errors: those of fw_dense_topk other than FW_E_WORKSPACE; FW_E_UNSUPPORTED
 * when the call needs more scratch than FW_NOALLOC_SCRATCH_BYTES (the size
 * fw_dense_topk_workspace_size reports for the same arguments) or when the
 * stream belongs to another device; FW_E_HIP when the device or the scratch
 * address cannot be queried.
 * ------------------------------------------------------------------------- */
#define FW_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
fw_status fw_dense_topk_noalloc(const fw_rows *rows, const int32_t *ks, int32_t n_ks,
                                float *o, float *o_s, float *gap, float *dropped,
                                int32_t *topk_idx, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_best_subset -- exact best kept set of size k by exhaustive enumeration
 * (Section 2.2, Definition 2.5 with every key of the row as the candidate
 * set), with the top-k comparison and the closed fraction
 * c = 1 - ES(k)/es(A*_k) (0 when es(A*_k) = 0).  Arithmetic is float64.
 *   k             budget, 1 <= k <= n
 *   best_idx      [H][G][k] int32 best set, ascending (required)
 *   best_gap      [H][G] float32 ES(k) (required)
 *   topk_gap      [H][G] float32 es of the top-k set, or NULL
 *   closed        [H][G] float32 closed fraction, or NULL
 *   dropped_topk  [H][G] float32 dropped mass of the top-k set, or NULL
 *   topk_idx      [H][G][k] int32 top-k set in rank order, or NULL
 * Errors: FW_E_UNSUPPORTED when n > 64 or C(n, k) >= 2^31; FW_E_NULL,
 * FW_E_SHAPE, FW_E_DTYPE, FW_E_WORKSPACE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
size_t fw_best_subset_workspace_size(const fw_rows *rows, int32_t k);
fw_status fw_best_subset(const fw_rows *rows, int32_t k, int32_t *best_idx, float *best_gap,
                         float *topk_gap, float *closed, float *dropped_topk, int32_t *topk_idx,
                         void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_pool_subset -- the candidate-set search of Section 2.2 (Definition 2.5
 * and the appendix's enumeration protocol) on rows of any length, with the
 * per-row certificate statistics of Section 2.3 and the appendix's absolute
 * forms, for up to FW_POOL_MAX_BUDGETS budgets per call (the row's weights,
 * dense output and key deviations are formed once for all of them).  Per row
 * and budget (s, extra), with the full row's masses p and dense output mu:
 *   - the candidate set: the top-mass set A*_s (logit desc, index asc) and
 *     the `extra` keys outside it of largest single-key error
 *     p_j ||v_j - mu|| (error desc, index asc);
 *   - ES_pool: the least es over the s-subsets of the candidate set, by
 *     exhaustive enumeration (ties to the lexicographically smallest
 *     ascending index tuple);
 *   - the balancing selector drawing from the candidate set: from A*_s, the
 *     (kept, dropped) pool swap that most decreases es (ties to the smallest
 *     (out, in)), strict decrease only, at most max_swaps swaps;
 *   - the free-weight side (Section 2.1's ef(A) = dist(mu, conv{v_j : j in
 *     A}) and EF(s); the appendix's penalty estimate): the Frank-Wolfe
 *     estimate EF_FW of EF(s) over the candidate set's values, from the key
 *     nearest mu (ties to the lower index), each step toward the vertex of
 *     least <v_j, x - mu> (ties to the lower index) with the exact line
 *     search, stopping at a non-positive duality gap, at a vertex that would
 *     be the (s+1)-th key of the support, or after fw_iters steps; the
 *     geometric set A^geo_s (the support padded to s keys with top-mass keys
 *     in rank order), its es, and pi_hat = ES_pool / EF_FW.
 * Arithmetic is float64 throughout.
 *   n_budgets      1 <= n_budgets <= FW_POOL_MAX_BUDGETS
 *   s, extra       host [n_budgets]: 1 <= s[b], 0 <= extra[b],
 *                  s[b] + extra[b] <= min(64, n); pools dropping more than
 *                  4 keys need a plannable enumeration of C(s + extra, s)
 *                  subsets (every pool of at most 24 keys is, and the
 *                  paper's (4, 24), (8, 12), (16, 6), (32, 4)); n <= 8192
 *   max_swaps      0 <= max_swaps <= 4096
 *   fw_iters       0 <= fw_iters <= 4096 Frank-Wolfe steps at most
 * With P_b = s[b] + extra[b], the budgets' lists are concatenated per row in
 * the caller's budget order:
 *   pool_idx       [H][G][sum_b P_b] int32: per budget, A*_s in rank order,
 *                  then the extra keys in error order, or NULL
 *   best_idx       [H][G][sum_b s[b]] int32: per budget, the ES_pool argmin,
 *                  ascending (required)
 *   bal_idx        [H][G][sum_b s[b]] int32: per budget, the balancing set,
 *                  ascending, or NULL
 *   geo_idx        [H][G][sum_b s[b]] int32: per budget, the geometric set,
 *                  ascending, or NULL
 *   n_swaps        [n_budgets][H][G] int32 balancing swaps applied, or NULL
 *   stats          [n_budgets][H][G][FW_POOL_NSTATS] float32 (required),
 *                  columns FW_POOL_* below
 *   flat_threshold, cell_median [n_budgets][H], cell_flat [n_budgets][H]
 *                  uint8: per budget and unit, the median of the rows'
 *                  dropped mass of A*_s (the mean of the two middle values
 *                  for even G) and whether it exceeds flat_threshold (a flat
 *                  cell at s = 8, threshold 0.25); either may be NULL
 * kappa and pi values are num/den, 1 when both are 0 and +inf when only den
 * is.
 * Errors: FW_E_UNSUPPORTED when a pool or its enumeration is out of the
 * limits above; FW_E_NULL, FW_E_SHAPE, FW_E_DTYPE, FW_E_WORKSPACE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
#define FW_POOL_MAX_BUDGETS 4
#define FW_POOL_NSTATS 16
#define FW_POOL_ES_TOP 0     /* es(A*_s)                                  */
#define FW_POOL_ES_POOL 1    /* ES_pool(s)                                */
#define FW_POOL_ES_BAL 2     /* es of the balancing set                   */
#define FW_POOL_KAPPA 3      /* kappa_hat = es(A*_s) / ES_pool            */
#define FW_POOL_C_HAT 4      /* c_hat = 1 - ES_pool / es(A*_s), 0 if es=0 */
#define FW_POOL_KAPPA_BAL 5  /* es(A_bal) / ES_pool                       */
#define FW_POOL_DROPPED 6    /* dropped mass of A*_s                      */
#define FW_POOL_PHI 7        /* Phi = ||g_{A*_s}|| (Lemma 2.2)            */
#define FW_POOL_DIAM 8       /* D = max_j ||v_j - mu||                    */
#define FW_POOL_SIGMA 9      /* sigma, sigma^2 = sum_j p_j ||v_j - mu||^2 */
#define FW_POOL_BOUND_DIAM 10 /* 2 D pbar (Lemma 2.2)                     */
#define FW_POOL_BOUND_VAR 11  /* sqrt(pbar / (1 - pbar)) sigma            */
#define FW_POOL_EF_FW 12      /* EF_FW(s): Frank-Wolfe estimate of EF(s)  */
#define FW_POOL_ES_GEO 13     /* es of the geometric set A^geo_s          */
#define FW_POOL_PI_HAT 14     /* pi_hat = ES_pool / EF_FW                 */
#define FW_POOL_FW_STEPS 15   /* Frank-Wolfe steps taken                  */
size_t fw_pool_subset_workspace_size(const fw_rows *rows, int32_t n_budgets, const int32_t *s,
                                     const int32_t *extra);
fw_status fw_pool_subset(const fw_rows *rows, int32_t n_budgets, const int32_t *s, const int32_t *extra,
                         int32_t max_swaps, int32_t fw_iters, int32_t *pool_idx, int32_t *best_idx,
                         int32_t *bal_idx, int32_t *geo_idx, int32_t *n_swaps, float *stats, float flat_threshold,
                         float *cell_median, uint8_t *cell_flat, void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_group_vote -- the group vote of Section 2.1: deployment keeps one set
 * per key/value head for the group of query rows that share it; the vote
 * keeps the s keys of largest mass summed over the group's rows (ties to the
 * lower index).  Each unit's G rows are ordered (query head) x (position),
 * G = group_size x T; the group of position t is the group_size rows
 * qh*T + t.  Per row, its forced-weight error under the vote's set and under
 * its own top-mass set (logit desc, index asc), from float64 sums.
 *   s           1 <= s <= min(n, 256)
 *   group_size  query heads per key/value head, dividing G
 *   vote_idx    [H][T][s] int32 the vote's keys by summed mass, descending
 *               (required)
 *   es_vote     [H][G] float32 es of the vote's set (required)
 *   es_top      [H][G] float32 es of the row's own top-mass set (required)
 *   dropped     [H][G] float32 the row's dropped mass under the vote's set,
 *               1 - p(vote), or NULL
 * The workspace query returns 0: no workspace is used (ws may be NULL).
 * Errors: FW_E_UNSUPPORTED when n, d and the group size need more than
 * 160 KiB of LDS (n <= 8192 always fits at d <= 256 and group_size <= 16);
 * FW_E_NULL, FW_E_SHAPE, FW_E_DTYPE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
size_t fw_group_vote_workspace_size(const fw_rows *rows, int32_t s, int32_t group_size);
fw_status fw_group_vote(const fw_rows *rows, int32_t s, int32_t group_size, int32_t *vote_idx, float *es_vote,
                        float *es_top, float *dropped, void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_swap -- the balancing selector of Section 2.1 ("swap rule"): start at
 * the top-k set and repeatedly apply the single (kept i, dropped j) swap that
 * most decreases es, over the full neighbourhood, accepting only a strict
 * decrease, for at most max_iters swaps.  Rows with n <= 64 run in float64;
 * longer rows evaluate swaps in float32 and report gaps from a float64 sum.
 *   k          budget, 1 <= k <= n
 *   max_iters  0 <= max_iters <= 4096
 *   s_idx      [H][G][k] int32 final set, ascending (required)
 *   gap_traj   [H][G][max_iters+1] float32 es after 0, 1, ... swaps; NaN
 *              after the last accepted swap (required)
 *   n_swaps    [H][G] int32 swaps applied (required)
 *   dropped    [H][G] float32 dropped mass of the final set, or NULL
 * Errors: FW_E_NULL, FW_E_SHAPE, FW_E_DTYPE, FW_E_WORKSPACE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
size_t fw_swap_workspace_size(const fw_rows *rows, int32_t k, int32_t max_iters);
fw_status fw_swap(const fw_rows *rows, int32_t k, int32_t max_iters, int32_t *s_idx,
                  float *gap_traj, int32_t *n_swaps, float *dropped,
                  void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_dropped_mass_curve -- observation-window importance and the per-unit
 * dropped-mass curve (Section 4, "ContourKV": r_j = mean over the G window
 * rows of the softmax weight p_{g,j}; Definition 2.1's least achievable
 * dropped mass as a function of the budget).  v is not read.
 *   importance [H][n] float32 r (required)
 *   curve      [H][n+1] float32 curve[k] = sum of all but the k largest r,
 *              accumulated from the smallest upward; curve[n] = 0 (required)
 *   order      [H][n] int32 keys by r descending, index ascending, or NULL
 * Errors: FW_E_NULL, FW_E_SHAPE, FW_E_DTYPE, FW_E_WORKSPACE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
size_t fw_dropped_mass_curve_workspace_size(const fw_rows *rows);
fw_status fw_dropped_mass_curve(const fw_rows *rows, float *importance, float *curve,
                                int32_t *order, void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_ragged_compact -- ContourKV allocation and ragged per-unit storage
 * (Section 4, "ContourKV" and "Setup and measured memory"): one score and
 * one threshold tau shared by all H units; each unit keeps its last
 * recency_floor positions plus its non-floor keys of score >= tau, tau set
 * so that exactly budget_entries entries are kept in total (floor included;
 * ties at tau resolve by unit, then position, ascending).  With cap > 0 the
 * budget is enforced per unit (Section 4: enforcement caps every head):
 * each unit offers only its cap - floor best non-floor keys (score desc,
 * position asc) to the shared threshold, so no unit keeps more than cap.
 * Kept rows are gathered, positions ascending within a unit, unit after
 * unit.
 *   dtype, k, v        [H][n][d] keys/values to compact (bit copies)
 *   heads_per_layer    units per layer (divides H), for the padded layout
 *   importance         [H][n] float32 score r (e.g. fw_dropped_mass_curve,
 *                      or its fw_maxpool_scores pooling)
 *   budget_entries     H*min(floor,n) <= budget_entries <= H*min(cap,n)
 *   cap                0 (no per-unit cap) or min(floor, n) <= cap
 *   offsets            [H+1] int64 exclusive prefix of kept counts (required)
 *   kept_pos           [budget_entries] int32 kept positions (required)
 *   k_out, v_out       [budget_entries][d] gathered rows (required)
 *   tau                [1] float32 threshold (score of the last non-floor
 *                      pick; +inf when no non-floor entry is kept), or NULL
 *   dropped            [H] float32 score mass of the evicted keys, or NULL
 *   bytes_held         [3] int64: K+V bytes held ragged, with every layer
 *                      padded to its widest unit, and as a full cache under a
 *                      mask; or NULL
 * Errors: FW_E_NULL, FW_E_SHAPE, FW_E_DTYPE, FW_E_WORKSPACE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
size_t fw_ragged_compact_workspace_size(int64_t H, int64_t n, int64_t d, int64_t budget_entries);
fw_status fw_ragged_compact(int32_t dtype, const void *k, const void *v, int64_t H,
                            int64_t heads_per_layer, int64_t n, int64_t d,
                            const float *importance, int64_t budget_entries,
                            int32_t recency_floor, int64_t cap, int64_t *offsets, int32_t *kept_pos,
                            void *k_out, void *v_out, float *tau, float *dropped,
                            int64_t *bytes_held, void *ws, size_t ws_bytes, fw_stream stream);

/* ---------------------------------------------------------------------------
 * fw_maxpool_scores -- SnapKV's pooling of an observation-window score, as
 * the appendix's audit runs it (kernel 7): out[h][j] = max of scores[h][i]
 * over |i - j| <= kernel / 2, positions outside [0, n) ignored.
 *   scores, out  [H][n] float32 (out must not alias scores unless kernel = 1)
 *   kernel       odd, 1 <= kernel <= 1023
 * Errors: FW_E_NULL, FW_E_SHAPE, FW_E_HIP.
 * ------------------------------------------------------------------------- */
fw_status fw_maxpool_scores(const float *scores, int64_t H, int64_t n, int32_t kernel, float *out,
                            fw_stream stream);

/* Thread-local description of the calling thread's last error ("" if none). */
const char *fw_last_error(void);
/* Library version string. */
const char *fw_version(void);

#ifdef __cplusplus
}
#endif
#endif /* FW_H */
