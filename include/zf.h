/*
 * zf.h -- C ABI of the ZenFlow selective-update hot path on MI355X (gfx950).
 *
 * For each bf16 weight gradient G of shape n x m (n output features = rows,
 * m input channels = columns, PyTorch [out, in] row-major layout):
 *
 *   zf_colnorm          s_j = sum_i G_ij^2, one score per input channel
 *                       (paper, Gradient Selection: "Lightweight Proxy for
 *                       Gradient Ranking" -- per-column squared norms).
 *   zf_topk_select      the k = round(ratio*m) columns with the largest score
 *                       (Gradient Selection; ratio = the "topk_ratio"
 *                       hyperparameter of the Evaluation section).
 *   zf_adam_selected    in-place Adam/AdamW step of the selected columns'
 *                       fp32 master weight and moments, with the bf16 weight
 *                       write-back (Asynchronous Offloading Workflow: the
 *                       GPU-side selective optimizer; Implementation:
 *                       "Selective GPU-side Optimizer").
 *   zf_pack_accumulate  the unselected columns gathered into a contiguous
 *                       fp32 buffer and summed over an interval of S steps
 *                       (Asynchronous Offloading Workflow: unimportant
 *                       gradients accumulated over several iterations;
 *                       Convergence Analysis: the S-step rule).
 *   zf_unpack           the accumulated buffer scattered back to a dense
 *                       n x m fp32 matrix, times a scale (1/S gives the mean
 *                       of the Convergence Analysis update).
 *   zf_update_fused     zf_adam_selected + zf_pack_accumulate in one pass
 *                       over G.
 *
 * plus a batched "plan" that runs each of these over many matrices in one
 * launch per kernel.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.   Every pointer argument is a DEVICE pointer unless marked HOST.
 *           The caller owns all memory.  Only zf_plan_create allocates
 *           (its device tables and workspace, freed by zf_plan_destroy).
 * Streams.  Work is enqueued on `stream` (a hipStream_t; NULL = the null
 *           stream); calls return without synchronising.  Device-side
 *           faults surface at the caller's next synchronisation.
 * Layouts.  Every matrix of a call is stored in one of two layouts
 *           (zf_layout).  ZF_LAYOUT_ROW_MAJOR is PyTorch's [out, in]: G, W
 *           (bf16, passed as uint16_t bit patterns) and the dense unpack
 *           output are [n][ld >= m]; the compact optimizer states P (master),
 *           M (first moment), V (second moment) are [n][ld_state >= k], slot
 *           r of a row belonging to column sel_idx[r]; the accumulation
 *           buffer A is [n][ld_acc >= m-k], slot u belonging to column
 *           unsel_idx[u].  ZF_LAYOUT_CHANNEL_MAJOR stores each of these
 *           transposed, so that an input channel is one contiguous row (the
 *           paper reorganises gradients column-major for channel access,
 *           Implementation, "Fully Segmented Gradient Selection"): G, W and
 *           the unpack output are [m][ld >= n], P/M/V are [k][ld_state >= n]
 *           (row r = column sel_idx[r]), A is [m-k][ld_acc >= n] (row u =
 *           column unsel_idx[u]).  Results are identical in both layouts.
 * Selection.  sel_idx[k] and unsel_idx[m-k] are ascending column indices;
 *           sel_mask[ceil(m/64)] has bit b of word w set iff column 64w+b is
 *           selected (bits at columns >= m are 0); sel_prefix[ceil(m/64)]
 *           counts the selected columns with index < 64w.
 * Errors.   Arguments are validated on the host before anything is
 *           enqueued; on any error nothing is enqueued.  ZF_EINVAL: a NULL
 *           pointer where the sizes require data, n, m or k out of range,
 *           ld < width, a pointer not aligned to its element size, ratio
 *           outside [0, 1] or NaN, step < 1, step_in_interval outside
 *           [1, accum_interval], invalid hyperparameters, or the gradient
 *           overlapping an output.  ZF_EWORKSPACE: workspace too small.
 *           ZF_EHIP: a HIP call failed (zf_last_hip_error() gives its code,
 *           per thread).  ZF_ENOMEM: a plan's device allocation failed.
 *           Sizes n = 0 or m = 0 are valid and enqueue no work, except that
 *           zf_colnorm with n = 0 writes zeros to its m scores.  Limits:
 *           n, m < 2^30; in the row-major layout the update and unpack
 *           kernels address 8-row blocks through 32-bit offsets, so a row
 *           stride times 8 must stay below 2 GiB.
 * Threads.  Entry points are reentrant.  Calls that share an output buffer,
 *           a workspace or a plan must be ordered by the caller.
 */
#ifndef ZF_H
#define ZF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void* zf_stream; /* a hipStream_t */

typedef enum zf_layout {
  ZF_LAYOUT_ROW_MAJOR = 0,
  ZF_LAYOUT_CHANNEL_MAJOR = 1
} zf_layout;

typedef enum zf_status {
  ZF_OK = 0,
  ZF_EINVAL = 1,
  ZF_EWORKSPACE = 2,
  ZF_EHIP = 3,
  ZF_ENOMEM = 4
} zf_status;

/* HOST struct.  Adam (Kingma & Ba) with decoupled weight decay (AdamW); the
 * paper fine-tunes with AdamW, weight decay 0 and lr 1e-5 (Experimental
 * Setup).  Requirements: lr, eps finite and >= 0; 0 <= beta1, beta2 < 1;
 * weight_decay finite and >= 0. */
typedef struct zf_adam_hparams {
  double lr;
  double beta1;
  double beta2;
  double eps;
  double weight_decay;
} zf_adam_hparams;

/* HOST struct of DEVICE pointers describing one selection (see Selection
 * above).  The selection of an n x m matrix depends on m and k only. */
typedef struct zf_selection {
  int32_t* sel_idx;    /* [k]           */
  int32_t* unsel_idx;  /* [m - k]       */
  uint64_t* sel_mask;  /* [ceil(m/64)]  */
  int32_t* sel_prefix; /* [ceil(m/64)]  */
} zf_selection;

/* Where the states of the selected columns come from in an Adam step.
 * ZF_STATES_INPLACE: P/M/V already hold the states of the selected columns.
 * ZF_STATES_REMAP:   the selection was just refreshed; a column that was
 *                    selected before reads its (p, m, v) from the previous
 *                    compact states at its previous slot, a newly selected
 *                    column starts with m = v = 0 and p from the init source.
 *                    The previous states must not alias the new ones.
 * ZF_STATES_INIT:    every selected column is new (first step).
 * Init source for p: the fp32 full master [n][ld_init] when init_master is
 * not NULL, else the widened bf16 weight W.  This is the swap-in of the
 * selective optimizer's states when its subset changes (Zero-stall
 * Pipeline, "Swapping out/in"). */
typedef enum zf_state_mode {
  ZF_STATES_INPLACE = 0,
  ZF_STATES_REMAP = 1,
  ZF_STATES_INIT = 2
} zf_state_mode;

/* HOST struct of DEVICE pointers; fields unused by the chosen mode may be
 * NULL.  prev_mask / prev_prefix describe the previous selection of the same
 * matrix (same m); the prev_* states are compact states of that selection
 * (as many slots as it has columns) with row stride ld_prev, in the call's
 * layout; init_master is a full fp32 n x m master in the call's layout with
 * row stride ld_init. */
typedef struct zf_state_source {
  const uint64_t* prev_mask;
  const int32_t* prev_prefix;
  const float* prev_master;
  const float* prev_exp_avg;
  const float* prev_exp_avg_sq;
  int64_t ld_prev;
  const float* init_master;
  int64_t ld_init;
} zf_state_source;

/* Text for a status code (static storage). */
const char* zf_status_string(int status);

/* HIP error code of the last ZF_EHIP returned on this thread (0 if none). */
int zf_last_hip_error(void);

/* Number of selected columns for a ratio: floor(ratio*m + 1/2) computed in
 * double, clamped to [0, m] (reading: round half up).  Returns -1 when ratio
 * is outside [0, 1] or NaN, or m < 0.  Pure host function. */
int64_t zf_k_from_ratio(double ratio, int64_t m);

/* ---- a1: column scores ------------------------------------------------- */

/* Workspace bytes zf_colnorm needs for an n x m gradient in `layout` (0 for
 * the channel-major layout). */
size_t zf_colnorm_workspace_bytes(int64_t n, int64_t m, int32_t layout);

/* norms_sq[j] = sum over i < n of G[i][j]^2 (fp32 result; squares summed in
 * fp64, deterministic order), for j < m.
 * grad: bf16 in `layout` with row stride ld_grad; norms_sq: [m] fp32 output;
 * ws: device workspace of at least zf_colnorm_workspace_bytes(n, m, layout)
 * bytes (may be NULL if that is 0), contents overwritten. */
zf_status zf_colnorm(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                     int32_t layout, float* norms_sq, void* ws, size_t ws_bytes,
                     zf_stream stream);

/* ---- a2: selection ------------------------------------------------------ */

/* Selects the k = zf_k_from_ratio(ratio, m) columns with the largest score.
 * Order: larger score first; equal scores (-0.0 equals +0.0) go to the lower
 * column index.  NaN scores give an unspecified (but valid) selection.
 * norms_sq: [m] fp32 input; out: HOST struct of the four output arrays;
 * k_out: HOST, optional, receives k. */
zf_status zf_topk_select(const float* norms_sq, int64_t m, double ratio,
                         const zf_selection* out, int64_t* k_out, zf_stream stream);

/* ---- a3 + a4: selective Adam and bf16 write-back ------------------------ */

/* For every row i < n and selected slot r < k (column j = sel_idx[r]):
 *   g = G[i][j]; states (p, m, v) per `mode` (see zf_state_mode);
 *   m' = B1*m + C1*g;  v' = B2*v + C2*(g*g);
 *   u  = (m'*IB1) / (sqrt(v'*IB2) + EPS);
 *   p  = p - WD*p (only if weight_decay != 0);  p' = p - LR*u;
 *   P/M/V[i][r] = p', m', v';  W[i][j] = bf16_round_nearest_even(p')
 * with B1 = beta1, C1 = 1-beta1, B2 = beta2, C2 = 1-beta2, LR = lr,
 * WD = lr*weight_decay, IB1 = 1/(1-beta1^step), IB2 = 1/(1-beta2^step), each
 * computed in double on the host and rounded once to fp32; every device
 * operation is one fp32 IEEE operation (no contraction, correctly rounded
 * sqrt and division).  Unselected columns of W are not touched.
 * step: 1-based step counter used for bias correction.
 * sel: HOST struct; all four arrays are read and must describe one
 * consistent selection (as zf_topk_select writes it). */
zf_status zf_adam_selected(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                           int32_t layout, const zf_selection* sel, int64_t k,
                           float* master, float* exp_avg, float* exp_avg_sq, int64_t ld_state,
                           uint16_t* weight, int64_t ld_weight,
                           const zf_adam_hparams* hp, int64_t step,
                           int32_t mode, const zf_state_source* src, zf_stream stream);

/* ---- a5: accumulation of the unselected columns ------------------------- */

/* For every row i < n and unselected slot u < m-k (column j = unsel_idx[u]):
 *   A[i][u] = G[i][j]              if step_in_interval == 1 (overwrite),
 *   A[i][u] = A[i][u] + G[i][j]    otherwise (one fp32 addition).
 * step_in_interval: 1-based position inside the accumulation interval of
 * accum_interval (= S) steps.  sel: HOST struct; all four arrays are read
 * and must describe one consistent selection. */
zf_status zf_pack_accumulate(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                             int32_t layout, const zf_selection* sel, int64_t k,
                             float* acc, int64_t ld_acc,
                             int64_t step_in_interval, int64_t accum_interval,
                             zf_stream stream);

/* zf_adam_selected and zf_pack_accumulate for the same step, one pass over G.
 * Arguments as in those two calls. */
zf_status zf_update_fused(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                          int32_t layout, const zf_selection* sel, int64_t k,
                          float* master, float* exp_avg, float* exp_avg_sq, int64_t ld_state,
                          uint16_t* weight, int64_t ld_weight,
                          const zf_adam_hparams* hp, int64_t step,
                          int32_t mode, const zf_state_source* src,
                          float* acc, int64_t ld_acc,
                          int64_t step_in_interval, int64_t accum_interval,
                          zf_stream stream);

/* ---- a6: hand-over ------------------------------------------------------ */

/* out[i][j] = +0.0 for selected j, scale * A[i][u] for the unselected column
 * j = unsel_idx[u] (one fp32 multiply; scale 1 copies bits).
 * acc: [n][ld_acc]; out: [n][ld_out] fp32 dense.  sel: HOST struct; sel_mask
 * and sel_prefix are read. */
zf_status zf_unpack(const float* acc, int64_t ld_acc, const zf_selection* sel, int64_t k,
                    int64_t n, int64_t m, int32_t layout, float scale, float* out,
                    int64_t ld_out, zf_stream stream);

/* ---- batched plans ------------------------------------------------------ */

/* HOST struct describing one matrix of a batch.  Pointers as in the single
 * calls; fields of a stage that the caller never runs may be NULL.  k must
 * equal zf_k_from_ratio(ratio, m) for the ratio the caller selects with
 * (zf_plan_create takes k as given). */
typedef struct zf_matrix {
  int64_t n, m, k;
  int32_t layout; /* zf_layout; every matrix of a plan uses the same one */
  const uint16_t* grad;
  int64_t ld_grad;
  uint16_t* weight;
  int64_t ld_weight;
  float* master;
  float* exp_avg;
  float* exp_avg_sq;
  int64_t ld_state;
  float* acc;
  int64_t ld_acc;
  float* norms_sq;
  zf_selection sel;
  float* unpacked;
  int64_t ld_unpacked;
  zf_state_source src;
} zf_matrix;

typedef struct zf_plan zf_plan;

/* Validates nmats >= 1 descriptors (HOST array, copied), computes the launch
 * geometry and allocates the plan's device tables and column-score
 * workspace (synchronous upload on the null stream).  *out receives the plan
 * (HOST handle). */
zf_status zf_plan_create(const zf_matrix* mats, int32_t nmats, zf_plan** out);

/* Frees a plan and its device memory (synchronises the device first). */
void zf_plan_destroy(zf_plan* plan);

/* Device bytes a plan holds (tables + workspace). */
size_t zf_plan_device_bytes(const zf_plan* plan);

/* zf_colnorm over every matrix of the plan (one workspace shared by the
 * plan: do not run two colnorm calls of one plan concurrently). */
zf_status zf_plan_colnorm(zf_plan* plan, zf_stream stream);

/* zf_topk_select over every matrix, k taken from the descriptors. */
zf_status zf_plan_topk_select(zf_plan* plan, zf_stream stream);

/* zf_adam_selected (do_adam != 0) and/or zf_pack_accumulate (do_pack != 0)
 * over every matrix; both together is zf_update_fused. */
zf_status zf_plan_update(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                         int32_t mode, int64_t step_in_interval, int64_t accum_interval,
                         int32_t do_adam, int32_t do_pack, zf_stream stream);

/* zf_unpack over every matrix into its `unpacked` buffer. */
zf_status zf_plan_unpack(zf_plan* plan, float scale, zf_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* ZF_H */
