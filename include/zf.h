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
 * launch per kernel, and, on a plan, the statistics of Zen-auto (the
 * adaptive accumulation interval) fused into the update pass
 * (zf_plan_update_zen).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.   Every pointer argument is a DEVICE pointer unless marked HOST.
 *           The caller owns all memory; the library allocates no device
 *           memory.  Workspaces and a plan's device tables live in buffers
 *           the caller provides, sized by the *_workspace_bytes and
 *           zf_plan_query calls.  The only allocation the library makes is
 *           the host-side plan handle (zf_plan_create, freed by
 *           zf_plan_destroy).
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
 *           Row-major update steps with the states in place (and pack-only
 *           calls) run a kernel with 16-byte accesses when G is 16-byte
 *           aligned with ld % 8 == 0 and A, P/M/V and the hand-over output
 *           (those the call uses) are 16-byte aligned with ld % 4 == 0;
 *           otherwise a per-column kernel.  The results are identical.
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
 *           per thread).  ZF_ENOMEM: the plan's host handle could not be
 *           allocated.
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
 * row stride ld_init.
 *
 * Full-state store (the offloaded optimizer's states of every column; paper,
 * Zero-stall Pipeline, "Swapping out/in": the selective optimizer's states
 * are swapped out to the host and back in).  store_* are full fp32 n x m
 * master / first / second moment arrays in the call's layout with row
 * stride ld_store, in device memory or in pinned host memory that the
 * kernels access in place.  When store_master is not NULL it replaces the
 * init source: in ZF_STATES_INIT and ZF_STATES_REMAP a newly selected column
 * reads (p, m, v) from its column of the store (swap-in), and in
 * ZF_STATES_REMAP a column that was selected before but no longer is writes
 * its previous compact (p, m, v) to its column of the store (swap-out), so
 * the prev_* states are then required even when k = 0.  The store must not
 * overlap any other buffer of the call.
 *
 * Owed deferred update (read by zf_plan_update_pending only, else may be
 * NULL): pend_acc holds the packed sums of the accumulation interval that
 * ended just before a refresh, under the previous selection (which has k
 * columns as well), in the layout of the packed buffer with row stride
 * ld_pend ([n][ld_pend >= m-k],
 * channel-major [m-k][ld_pend >= n]; slot u' = the u'-th column, in
 * ascending order, that the previous selection left unselected). */
typedef struct zf_state_source {
  const uint64_t* prev_mask;
  const int32_t* prev_prefix;
  const float* prev_master;
  const float* prev_exp_avg;
  const float* prev_exp_avg_sq;
  int64_t ld_prev;
  const float* init_master;
  int64_t ld_init;
  float* store_master;
  float* store_exp_avg;
  float* store_exp_avg_sq;
  int64_t ld_store;
  const float* pend_acc;
  int64_t ld_pend;
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

/* For callers that cannot allocate device memory or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): zf_colnorm with its workspace in an array of
 * ZF_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on,
 * from the first call on that GPU until the process ends.  Arguments and
 * results as in zf_colnorm.  Allocates nothing: the first call on a GPU
 * only looks up that array's device address.  ZF_EWORKSPACE (nothing
 * enqueued) when zf_colnorm_workspace_bytes(n, m, layout) exceeds
 * ZF_STATIC_SCRATCH_BYTES (row-major: ceil(n / rows per block) * m * 8
 * bytes, 4-15 MiB for the Llama-2 shapes; channel-major needs none).  Every
 * call on one GPU shares that GPU's array: calls that may overlap on one
 * GPU (other streams, other host threads) race and must be ordered by the
 * caller.  Nothing in the array needs to start at zero; each call writes
 * every part it reads. */
#define ZF_STATIC_SCRATCH_BYTES (32u << 20)
zf_status zf_colnorm_noalloc(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                             int32_t layout, float* norms_sq, zf_stream stream);

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

/* zf_update_fused for the last step of an accumulation interval with the
 * hand-over (zf_unpack) fused in: the same Adam step of the selected
 * columns, and for every unselected slot u (column j = unsel_idx[u]):
 *   out[i][j] = scale * G[i][j]                  if step_in_interval == 1,
 *   out[i][j] = scale * (A[i][u] + G[i][j])      otherwise
 * (the same two fp32 operations, in the same order, as zf_pack_accumulate
 * followed by zf_unpack), out[i][j] = +0.0 for selected j.  The packed
 * buffer A is only read: it keeps the sums of the interval's earlier steps
 * (the next interval overwrites it).  This moves 8 bytes per unselected
 * element less than the two separate passes (A is neither written nor read
 * back).  out: fp32 n x m in `layout` with row stride ld_out, disjoint from
 * every other buffer of the call.  Other arguments as in zf_update_fused. */
zf_status zf_update_fused_handover(const uint16_t* grad, int64_t n, int64_t m, int64_t ld_grad,
                                   int32_t layout, const zf_selection* sel, int64_t k,
                                   float* master, float* exp_avg, float* exp_avg_sq,
                                   int64_t ld_state, uint16_t* weight, int64_t ld_weight,
                                   const zf_adam_hparams* hp, int64_t step, int32_t mode,
                                   const zf_state_source* src, const float* acc, int64_t ld_acc,
                                   int64_t step_in_interval, int64_t accum_interval, float scale,
                                   float* out, int64_t ld_out, zf_stream stream);

/* ---- a6: hand-over ------------------------------------------------------ */

/* out[i][j] = +0.0 for selected j, scale * A[i][u] for the unselected column
 * j = unsel_idx[u] (one fp32 multiply; scale 1 copies bits).
 * acc: [n][ld_acc]; out: [n][ld_out] fp32 dense.  sel: HOST struct; sel_mask
 * and sel_prefix are read. */
zf_status zf_unpack(const float* acc, int64_t ld_acc, const zf_selection* sel, int64_t k,
                    int64_t n, int64_t m, int32_t layout, float scale, float* out,
                    int64_t ld_out, zf_stream stream);

/* ---- deferred update of the unselected columns (offloaded optimizer) ---- */

/* HOST function (host pointers only; no device work): one Adam/AdamW step
 * of every unselected column with the accumulation interval's mean gradient,
 * on the offloaded optimizer's states (paper, Asynchronous Offloading
 * Workflow: the accumulated unimportant gradients are applied by the CPU
 * optimizer; Convergence Analysis: the delayed coordinates move by the mean
 * of the S accumulated gradients; Implementation, "Concurrent CPU-side
 * Optimizer").  For every unselected slot u (column j = unsel_idx[u]) and
 * row i:
 *   g = acc[i][u] * scale;  (p, m, v) = state column j;  the element
 *   sequence of zf_adam_selected with the constants of step `step`;
 *   state column j = (p', m', v');  weight_cols[i][u] = bf16_rne(p').
 * acc: packed sums [n][ld_acc >= m-k] (channel-major: [m-k][ld_acc >= n]),
 *   e.g. a host copy of the device buffer zf_pack_accumulate fills;
 * unsel_idx: [m-k] strictly ascending column indices in [0, m);
 * master / exp_avg / exp_avg_sq: full n x m fp32 states with row stride
 *   ld_state in `layout`, updated in place at the unselected columns only;
 * weight_cols: bf16 output [n][ld_wcols >= m-k] (channel-major [m-k][..]);
 * scale: fp32 factor of the sums (1/S for the mean), finite;
 * step: the offloaded optimizer's own 1-based step counter;
 * nthreads: worker threads (0 = all hardware threads); the call returns
 *   when every thread has finished.
 * ZF_EINVAL (nothing written) for invalid sizes, strides, hyperparameters,
 * indices that are not strictly ascending in [0, m), or overlapping
 * buffers.  Results are bit-identical to the device's element sequence. */
zf_status zf_host_adam_unselected(const float* acc, int64_t ld_acc, const int32_t* unsel_idx,
                                  int64_t n, int64_t m, int64_t k, int32_t layout, float scale,
                                  float* master, float* exp_avg, float* exp_avg_sq,
                                  int64_t ld_state, uint16_t* weight_cols, int64_t ld_wcols,
                                  const zf_adam_hparams* hp, int64_t step, int32_t nthreads);

/* Write-back of the deferred update: W[i][unsel_idx[u]] = weight_cols[i][u]
 * for every unselected slot u and row i; selected columns of W are not
 * touched.  weight_cols: bf16 [n][ld_wcols >= m-k] (channel-major
 * [m-k][ld_wcols >= n]) in device memory or pinned host memory (read in
 * place); weight: bf16 n x m in `layout`.  sel: HOST struct; sel_mask and
 * sel_prefix are read (the selection the columns were updated under). */
zf_status zf_scatter_weights(const uint16_t* weight_cols, int64_t ld_wcols,
                             const zf_selection* sel, int64_t k, int64_t n, int64_t m,
                             int32_t layout, uint16_t* weight, int64_t ld_weight,
                             zf_stream stream);

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
  float* sel_sq; /* Zen-auto only: [k] fp32 (else NULL)     */
  float* acc_sq; /* Zen-auto only: [m - k] fp32 (else NULL) */
  const uint16_t* weight_cols; /* deferred update only: bf16 [n][m-k] / cm [m-k][n] */
  int64_t ld_weight_cols;
  uint16_t* acc_first; /* optional: bf16 in the gradient's shape (channel-major
                          [m][ld >= n], row j = channel j; row-major [n][ld >= m]) */
  int64_t ld_acc_first;
} zf_matrix;

typedef struct zf_plan zf_plan;

/* First-step stage of the packed buffer (acc_first).
 * On the first step of an interval the packed values are the widened
 * gradient itself, so every one of them is exactly a bf16.  When a
 * descriptor gives acc_first (a bf16 array in the gradient's shape: element
 * (i, j) at the place of G's element (i, j)),
 * zf_plan_update (do_pack) and zf_plan_update_handover keep that step's
 * values there, as the gradient's bf16 bits (2 bytes per element written
 * instead of 4), and the interval's second step reads them from there
 * instead of from acc (2 bytes read instead of 4) and writes its fp32 sums
 * to acc as usual.  The rule is stateless: with acc_first,
 * step_in_interval == 1 writes the unselected channels' rows of acc_first
 * and not acc; step_in_interval == 2 reads those rows.  A refresh step may
 * instead run zf_plan_colnorm_stage (scores plus every channel's row of the
 * stage, in one pass over G) and then zf_plan_update with do_pack = 0: the
 * stage then holds what the packing would have written.  Every result (acc
 * from the second step on, the hand-over, W, the states) is bit-identical
 * to a plan without it.  acc_first must overlap no other buffer and be
 * 2-byte aligned (channel-major: 16-byte aligned with ld % 8 == 0 for the
 * vector path; row-major: always 16-byte aligned with ld % 8 == 0).  In the
 * channel-major layout zf_plan_update_zen follows the same rule, and the
 * separate hand-over of an interval that ended after its first step reads
 * the stage: zf_plan_unpack_first instead of zf_plan_unpack.  Row-major
 * plans with a stage reject zf_plan_update_zen (its refresh statistics
 * read the packed buffer); the offloaded optimizer's calls
 * (zf_plan_update_pending, zf_plan_update_zen_pending) reject any plan with
 * a stage (ZF_EINVAL). */

/* Device bytes a plan over these descriptors needs (its descriptor tables
 * and its workspaces: column-score partials of row-major matrices,
 * Zen-auto partials).  Validates the descriptors as zf_plan_create does;
 * no device work.  mats: HOST array of nmats >= 1 descriptors;
 * device_bytes: HOST, receives the size.  ZF_EINVAL also when one of the
 * plan's launches would need more than 2^32 - 1 work-items, the limit of a
 * dispatch (channel-major: a set of more than about 34 G parameters, whose
 * update grid covers 2048 or 4096 rows of a channel per 256-thread block);
 * such a set is split over several plans. */
zf_status zf_plan_query(const zf_matrix* mats, int32_t nmats, size_t* device_bytes);

/* Builds a plan in caller-provided device memory: validates nmats >= 1
 * descriptors (HOST array, copied into the plan), computes the launch
 * geometry and enqueues, on `stream`, the upload of the descriptor tables
 * to the start of device_mem (the rest is the plan's workspace).  The
 * upload is stream-ordered: launches of the plan on `stream`, or on a
 * stream ordered after it, see the tables.  device_mem: at least
 * zf_plan_query's bytes, 256-byte aligned, owned by the caller, not
 * touched by anything else while the plan is used.  *out receives the plan
 * (a HOST handle, the only memory the library allocates).  ZF_EWORKSPACE
 * when device_bytes is too small; nothing is enqueued on any error. */
zf_status zf_plan_create(const zf_matrix* mats, int32_t nmats, void* device_mem,
                         size_t device_bytes, zf_stream stream, zf_plan** out);

/* Frees the plan's host handle.  No device call and no synchronisation:
 * the caller frees device_mem once the plan's launches have completed. */
void zf_plan_destroy(zf_plan* plan);

/* Device bytes the plan uses of its device_mem (tables + workspace). */
size_t zf_plan_device_bytes(const zf_plan* plan);

/* zf_colnorm over every matrix of the plan (one workspace shared by the
 * plan: do not run two colnorm calls of one plan concurrently). */
zf_status zf_plan_colnorm(zf_plan* plan, zf_stream stream);

/* zf_plan_colnorm that also copies the gradient to the descriptor's
 * acc_first (descriptors without one: scores only), in the same pass over
 * G: on a refresh step that starts an interval, the
 * packing of whichever channels the selection leaves unselected, done
 * before the selection is known (2 bytes per element written for every
 * channel instead of 2 read + 2 written for each unselected one in the
 * update).  Needs a plan with a stage (ZF_EINVAL otherwise). */
zf_status zf_plan_colnorm_stage(zf_plan* plan, zf_stream stream);

/* zf_plan_colnorm that also writes, for every channel, scale times its
 * widened gradient row to its row of the descriptor's `unpacked` buffer,
 * in the same pass over G (channel-major plans): on a refresh step that is
 * a one-step interval (handed over at once), the hand-over of whichever
 * channels the selection leaves unselected, done before the selection is
 * known; zf_plan_update_adam_handover then completes the step.  The
 * results equal those of zf_plan_colnorm followed by
 * zf_plan_update_handover with step_in_interval 1, bit for bit (4 bytes per
 * element written for every channel instead of 2 read + 4 written for each
 * unselected one in the update).  scale finite. */
zf_status zf_plan_colnorm_handover(zf_plan* plan, float scale, zf_stream stream);

/* zf_topk_select over every matrix, k taken from the descriptors. */
zf_status zf_plan_topk_select(zf_plan* plan, zf_stream stream);

/* zf_adam_selected (do_adam != 0) and/or zf_pack_accumulate (do_pack != 0)
 * over every matrix; both together is zf_update_fused. */
zf_status zf_plan_update(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                         int32_t mode, int64_t step_in_interval, int64_t accum_interval,
                         int32_t do_adam, int32_t do_pack, zf_stream stream);

/* After zf_plan_colnorm_handover and the selection: the Adam step of the
 * selected channels (zf_adam_selected, mode as there) and +0.0 in their rows
 * of `unpacked`; the unselected channels are not touched (their hand-over
 * rows are already written, the packed buffer is not needed for a one-step
 * interval).  Channel-major plans without a full-state store. */
zf_status zf_plan_update_adam_handover(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                       int32_t mode, zf_stream stream);

/* zf_plan_unpack for an interval that ended after its first step on a plan
 * whose every descriptor gives acc_first: the unselected channels' rows
 * are scale times their widened stage rows (the first step's values),
 * selected rows +0.0.  Channel-major plans; ZF_EINVAL for a row-major plan
 * or when a descriptor has no stage. */
zf_status zf_plan_unpack_first(zf_plan* plan, float scale, zf_stream stream);

/* zf_unpack over every matrix into its `unpacked` buffer. */
zf_status zf_plan_unpack(zf_plan* plan, float scale, zf_stream stream);

/* zf_update_fused_handover over every matrix (out = its `unpacked` buffer):
 * the last step of an interval in one pass, Adam + final accumulation +
 * hand-over.  With step_in_interval == 1 the packed buffer is not used
 * (out = scale * G at the unselected columns), so descriptors may then
 * leave it NULL. */
zf_status zf_plan_update_handover(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                  int32_t mode, int64_t step_in_interval, int64_t accum_interval,
                                  float scale, zf_stream stream);

/* Deferred packing: the unselected part of each step's gradient is left
 * where it was written (the caller keeps the gradients of the interval's
 * steps resident and unchanged until the interval ends: S buffers per
 * matrix), the interval's earlier steps run the Adam part alone
 * (zf_plan_update with do_pack = 0), and its last step, with
 * length = n_earlier + 1 >= 2, runs this call: the Adam step of the
 * selected channels (states in place, zf_adam_selected) and, in every
 * matrix's `unpacked` buffer,
 *   out[i][j] = scale * (((g_1[i][j] + g_2[i][j]) + ...) + g[i][j])
 * at the unselected channels (g_s the gradient of the interval's s-th step,
 * g this step's; the additions in step order, each one fp32 operation),
 * +0.0 at the selected ones: bit for bit what zf_pack_accumulate over the
 * interval followed by zf_unpack (or zf_plan_update_handover on the last
 * step) gives, with the packed buffer never written.  Each step's gradient
 * is read once, at its unselected channels, when the interval ends (2 bytes
 * per element per step, instead of the packed buffer's 8 per step).
 * earlier: HOST array of n_earlier (1..15) plans over the same matrices in
 * the same order (same n, m, k; channel-major: the same access path), in
 * step order, whose descriptors' grad is the gradient of that step; only
 * those gradients are read.  They must not overlap what this step writes.
 * Both layouts, plans without a full-state store; `unpacked` required;
 * scale finite.  Row-major: two launches, the Adam-only pass and a
 * hand-over pass (the 16-byte kernels when the plan runs the 16-byte update
 * and every earlier gradient has 16-byte rows, else the per-column ones);
 * the hand-over pass reads every element of each step's gradient, since
 * the selected columns share their cache lines.  ZF_EINVAL (nothing
 * enqueued) on a mismatch or when an earlier gradient's row stride does
 * not fit the plan's row blocks.  The kernels read the earlier plans'
 * device tables when they run: those plans' device memory (and their
 * gradients) must stay valid until this call's work on `stream` is done. */
zf_status zf_plan_update_handover_deferred(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                           const zf_plan* const* earlier, int32_t n_earlier,
                                           float scale, zf_stream stream);

/* zf_scatter_weights over every matrix (weight_cols of each descriptor). */
zf_status zf_plan_scatter_weights(zf_plan* plan, zf_stream stream);

/* The refresh step of the offloaded optimizer while the host is still
 * applying the deferred update of the interval that ended at the previous
 * step (paper, Zero-stall Pipeline: the GPU does not wait for the CPU-side
 * optimizer).  zf_plan_update with do_adam = do_pack = 1, mode
 * ZF_STATES_REMAP and step_in_interval = 1 against the full-state store,
 * except that a column entering the selection (selected now, unselected in
 * src.prev_mask) first takes the deferred step that its store column still
 * owes, then this step's Adam:
 *   g' = pend_acc[i][u'] * pend_scale  (u' its slot under the previous
 *        selection);  (p, m, v) = its store column;  the element sequence
 *        of zf_adam_selected with the constants of pend_step and g';
 *   then g = G[i][j] and the constants of `step` as in zf_adam_selected.
 * The results equal, bit for bit, those of zf_host_adam_unselected (same
 * pend_acc, pend_scale, pend_step) landing in the store before a plain
 * refresh.  The entering columns' store columns are only read: the caller
 * must not write them before this call has completed, and the write-back
 * of that host update must skip the columns the refresh selected
 * (zf_plan_scatter_weights_skip_prev).  Every descriptor needs the store,
 * the previous selection and states, the packed buffer and pend_acc, which
 * must not overlap any buffer the call writes.  pend_step >= 1; pend_scale
 * finite.  Zen-auto: zf_plan_update_zen_pending. */
zf_status zf_plan_update_pending(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                 int64_t accum_interval, int64_t pend_step, float pend_scale,
                                 zf_stream stream);

/* zf_plan_scatter_weights, except that every column set in the
 * descriptor's src.prev_mask is left untouched: the write-back of a
 * deferred update issued after the refresh that zf_plan_update_pending
 * ran, on a plan whose sel is the selection the update ran under and whose
 * src.prev_mask is the refreshed selection (the columns that entered it
 * already hold the selective optimizer's weights). */
zf_status zf_plan_scatter_weights_skip_prev(zf_plan* plan, zf_stream stream);

/* ---- Zen-auto: adaptive accumulation interval ---------------------------- */

/* Totals of one Zen-auto step over a whole plan, as written to DEVICE memory
 * by zf_plan_update_zen (40 bytes, 8-byte aligned). */
typedef struct zf_zen_totals {
  double sum_sel;  /* sum over every selected channel of sqrt(sel_sq)    */
  double sum_acc;  /* sum over every unselected channel of sqrt(acc_sq)  */
  int64_t k_total; /* selected channels of the plan                      */
  int64_t u_total; /* unselected channels of the plan                    */
  int32_t trigger; /* 1: hand the accumulated buffers over after this step */
  int32_t pad;
} zf_zen_totals;

/* The fused update (zf_plan_update with do_adam = do_pack = 1, same
 * arguments and results) that also measures what Zen-auto compares (paper,
 * Zero-stall Pipeline, "Hyperparameter Auto-tuning": the unimportant part's
 * average accumulated channel norm against the important part's average
 * channel norm; the deferred update is triggered once they are comparable):
 *   sel_sq[r] = sum_i g_ij^2 for the selected channel j = sel_idx[r], g this
 *               step's gradient (the important part, applied at once);
 *   acc_sq[u] = sum_i A_iu^2 over the accumulated column of slot u after
 *               this step's accumulation (the unimportant part);
 * each summed in fp64 (exact squares) in a fixed order and rounded once to
 * fp32.  Then, over every matrix of the plan, in fp64:
 *   sum_sel = sum of sqrt(sel_sq), sum_acc = sum of sqrt(acc_sq),
 *   trigger = k_total > 0 && u_total > 0 &&
 *             sum_acc * k_total >= (tau * sum_sel) * u_total,
 * i.e. the pooled mean accumulated norm reaches tau times the pooled mean
 * selected norm (reading of "comparable": tau = 1).  The result goes to
 * *totals (DEVICE).  The caller ends the interval (zf_plan_unpack with scale
 * 1/step_in_interval) when trigger is set; the next step then starts a new
 * interval (step_in_interval = 1).
 * Channel-major plans sum the squares inside the update pass.  Row-major
 * plans do too on steps with the states in place when their buffers take
 * the 16-byte update (see Layouts); on refresh steps, and for other
 * buffers, they run the update and then a separate statistics pass that
 * reads the selected gradient columns and the packed buffer again.  Both
 * row-major forms write the same fp64 partials (per column and
 * column-score row block, in row order) to the plan's column-score
 * workspace, so they give identical statistics; the two layouts agree up to
 * the order of the fp64 sums.
 * Requirements: every descriptor of the plan provides sel_sq [k] and
 * acc_sq [m - k] (device fp32, disjoint from each other and from the
 * update's buffers), tau >= 0 (+inf allowed, never triggers when
 * sum_sel > 0), totals 8-byte aligned; else ZF_EINVAL with nothing
 * enqueued.  The plan's workspaces are shared: do not run zf_plan_update_zen
 * concurrently with another zf_plan_update_zen or zf_plan_colnorm call of
 * the same plan. */
zf_status zf_plan_update_zen(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                             int32_t mode, int64_t step_in_interval, int64_t accum_interval,
                             double tau, zf_zen_totals* totals, zf_stream stream);

/* zf_plan_update_zen for the refresh step of the offloaded optimizer while
 * the host is still applying the deferred update of the interval that
 * ended at the previous step: mode ZF_STATES_REMAP and step_in_interval 1,
 * with the entering columns' owed deferred step taken over exactly as in
 * zf_plan_update_pending (same requirements); the statistics and totals
 * are those of zf_plan_update_zen. */
zf_status zf_plan_update_zen_pending(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                     int64_t accum_interval, int64_t pend_step, float pend_scale,
                                     double tau, zf_zen_totals* totals, zf_stream stream);

/* Zen-auto's interval driven on the device, so that a step needs no host
 * round trip (paper §3.2, "Hyperparameter Auto-tuning": the deferred update
 * is triggered once the accumulated part becomes comparable; keeping that
 * decision on the GPU is this library's choice).  The interval state lives in
 * DEVICE memory (8 bytes, 4-byte aligned), initialised by the caller to
 * {0, 1} (nothing accumulated; the first step starts an interval) and then
 * owned by the calls below, in stream order. */
typedef struct zf_zen_state {
  int32_t length; /* steps of the current interval so far                     */
  int32_t ended;  /* nonzero: the last step ended its interval; 1: its hand-
                   * over is zf_plan_handover_zen's, 2: the update wrote it  */
} zf_zen_state;

/* zf_plan_update_zen whose position in the interval is read from *state
 * instead of passed: 1 on a refresh (mode ZF_STATES_REMAP or
 * ZF_STATES_INIT) or after an ended interval, else state->length + 1 (so
 * the accumulation overwrites or adds, and with the bf16 stage writes or
 * reads the stage, as zf_plan_update_zen with that step_in_interval).
 * After the statistics and totals, the same launch sequence updates the
 * state: length = that position; ended = trigger || position >=
 * accum_interval (S_max) || force_end.  force_end: the caller's own end of
 * the interval (the next step refreshes the selection, or a warm-up step):
 * 1 -- the hand-over is left to zf_plan_handover_zen; 2 -- where the plan
 * can (channel-major; row-major steps in place on the 16-byte update; every
 * descriptor with `unpacked`) the update writes it itself, scale = fp32(1 /
 * position), bit for bit what zf_plan_handover_zen would write, and sets
 * ended = 2 so that zf_plan_handover_zen writes nothing (the packed buffer
 * is then left as it was, as in zf_plan_update_handover); elsewhere as 1.
 * Call zf_plan_handover_zen after every step either way.  Other values:
 * ZF_EINVAL.
 * Both layouts, plans without a full-state store; a row-major plan without
 * the bf16 stage; the requirements of zf_plan_update_zen otherwise.  Follow
 * it with zf_plan_handover_zen. */
zf_status zf_plan_update_zen_device(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                    int32_t mode, int64_t accum_interval, int32_t force_end,
                                    double tau, zf_zen_totals* totals, zf_zen_state* state,
                                    zf_stream stream);

/* The hand-over of the step zf_plan_update_zen_device just ran: if
 * state->ended == 1, every matrix's `unpacked` buffer receives the hand-over of
 * the interval (scale = fp32(1 / state->length); from the bf16 stage after
 * a one-step interval on a plan with one; +0.0 in the selected channels'
 * rows), bit for bit as zf_plan_unpack / zf_plan_unpack_first with that
 * scale; else nothing is written.  A fixed grid that loops over the work:
 * a step that does not end its interval costs one short launch.  Both
 * layouts; channel-major plans whose descriptors all have the stage or none
 * has it, row-major plans without it. */
zf_status zf_plan_handover_zen(zf_plan* plan, const zf_zen_state* state, zf_stream stream);

/* Zen-auto on the device with deferred packing (channel-major): the
 * interval's sums are never written step by step.  The unselected part of
 * each step's gradient stays where it was written, and the caller keeps the
 * gradients of the last accum_interval (S_max) steps resident and unchanged.
 * Zen-auto's statistic of an unselected channel is the squared norm of the
 * interval's running sum (paper §3.2, "Hyperparameter Auto-tuning"), so
 * each step sums the interval's kept gradients again, in step order in fp32
 * (the accumulation's own sequence, hence the same bits), for the
 * statistics; the selected channels take the Adam step as in
 * zf_plan_update_zen_device.  At a position p the unselected channels cost
 * 2p bytes per element read, against 8-10 read and written per step when
 * packing every step: fewer bytes while the intervals are short (S_max up to
 * about 6).
 * zf_plan_update_zen_device's semantics otherwise: position from *state, the
 * statistics, totals and trigger, the new state; force_end 2 writes the
 * hand-over, scale = fp32(1 / position) times the running sum (+0.0 at the
 * selected channels), and sets ended = 2; 1 leaves it to
 * zf_plan_handover_zen_deferred; 0 no forced end.
 * earlier: HOST array of n_earlier (0..15) plans over the same matrices in
 * the same order (same n, m, k and channel-major geometry), the plans of the
 * steps before this one, oldest first, whose descriptors' grad is that
 * step's gradient: at least the last min(S_max, steps since the first) - 1
 * of them.  The update reads the last position - 1 of them, the position
 * read from *state on the device; only their gradients are read, and they
 * must not overlap what the step writes.  Channel-major plans with
 * `unpacked`, the Zen-auto statistics buffers, without a full-state store;
 * the packed buffer (acc) and the bf16 stage are not used.  ZF_EINVAL
 * (nothing enqueued) otherwise.  The earlier plans' device memory and
 * gradients must stay valid until the work on `stream` is done.  Follow it
 * with zf_plan_handover_zen_deferred with the same earlier plans. */
zf_status zf_plan_update_zen_deferred(zf_plan* plan, const zf_adam_hparams* hp, int64_t step,
                                      int32_t mode, int64_t accum_interval,
                                      const zf_plan* const* earlier, int32_t n_earlier,
                                      int32_t force_end, double tau, zf_zen_totals* totals,
                                      zf_zen_state* state, zf_stream stream);

/* The hand-over of the step zf_plan_update_zen_deferred just ran: if
 * state->ended == 1, every matrix's `unpacked` buffer receives scale =
 * fp32(1 / state->length) times the interval's sums, summed from the last
 * length - 1 earlier plans' gradients and this plan's, in step order in
 * fp32, +0.0 at the selected channels: bit for bit what packing every step
 * and zf_plan_handover_zen give.  Else nothing is written; a fixed grid, so
 * that a step that does not end its interval costs one short launch.
 * earlier as in zf_plan_update_zen_deferred; channel-major plans that
 * zf_plan_update_zen_deferred accepts (gradient, selection, states,
 * `unpacked`); ZF_EINVAL otherwise. */
zf_status zf_plan_handover_zen_deferred(zf_plan* plan, const zf_plan* const* earlier,
                                        int32_t n_earlier, const zf_zen_state* state,
                                        zf_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* ZF_H */
