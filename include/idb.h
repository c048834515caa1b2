/*
 * idb.h -- C ABI of the ID Balancing router step for AMD MI355X (gfx950).
 *
 * The calls follow the paper's statement of the problem ("ID Balancing: Stable
 * Training of Extremely Sparse MoE via PID-Based Load Control"):
 *
 *   router    z = W_r x, s = sigmoid(z), T(x) = TopK(s + b), gate weights from
 *             the unbiased s, per-expert load counts n           (Sec. 2.2,
 *             Eq. pid-routing, Eq. pid-error)
 *   controller  e = (nbar - n)/nbar, de = e - e_prev, g = 1[e_prev de > 0],
 *             b += K_i e + K_d g de, b -= mean(b)                 (Alg. 1,
 *             Eq. rapid-integral, rapid-delta, rapid-gate, rapid-update)
 *   statistics  MaxVio, MinVio                                    (Sec. 4.1, Eq. vio)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Memory: every pointer argument that is not a host struct is a DEVICE
 *   pointer on the device that owns `stream`.  The caller allocates and owns
 *   all buffers; the library allocates nothing and keeps no state between
 *   calls.  Calls are reentrant and thread-safe.
 * - Asynchrony: every call only enqueues work on `stream` (0 = the null
 *   stream) and returns without synchronising.  Outputs are valid once the
 *   stream reaches that point.
 * - Errors: arguments are checked before anything is enqueued.  On an invalid
 *   argument the call returns IDB_ERR_INVALID_ARG (or IDB_ERR_UNSUPPORTED for
 *   a valid but unsupported shape), enqueues nothing and leaves every output
 *   untouched; these checks make no HIP call.  A failed launch returns
 *   IDB_ERR_HIP.  idb_last_error() gives a message for the last failing call on
 *   the calling thread.  Errors that depend on data (an empty batch) cannot be
 *   returned synchronously; the controller writes them to its device status.
 * - Layouts are row-major and densely packed.  x, W_g and workspace must be
 *   16-byte aligned; every other buffer 4-byte aligned (8 for int64/double).
 * - NaN or infinite inputs are a caller error and are not checked.
 * - Determinism: for the same inputs and variant, every output is bit-identical
 *   run to run; integer counts are exact.
 */
#ifndef IDB_H
#define IDB_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum idb_status {
    IDB_OK = 0,
    IDB_ERR_INVALID_ARG = 1, /* bad pointer, size, alignment or workspace       */
    IDB_ERR_UNSUPPORTED = 2, /* valid request outside what the kernels handle   */
    IDB_ERR_EMPTY_BATCH = 3, /* device status only: all counts zero, no update  */
    IDB_ERR_HIP = 4          /* a HIP launch failed                             */
} idb_status;

typedef enum idb_dtype {
    IDB_DTYPE_BF16 = 0, /* x and W_g hold bfloat16 values                     */
    IDB_DTYPE_F32 = 1   /* x and W_g hold fp32 values                         */
} idb_dtype;

typedef enum idb_weight_layout {
    IDB_WEIGHT_ROW_MAJOR = 0, /* W_g is [E][d] row-major                                  */
    IDB_WEIGHT_PACKED = 1     /* W_g was written by idb_router_pack_weight (same byte size) */
} idb_weight_layout;

typedef enum idb_integral_mode {
    IDB_INTEGRAL_ERROR = 0, /* ID Balancing: integral step K_i * e (Eq. rapid-integral)   */
    IDB_INTEGRAL_SIGN = 1   /* DeepSeek loss-free: K_i * sign(e), sign(0) = 0 (Eq. pid-deepseek) */
} idb_integral_mode;

/* Controller configuration (host struct). */
typedef struct idb_controller_cfg {
    int32_t E;             /* number of routed experts, 1 <= E <= 1024             */
    float Ki;              /* integral gain K_i >= 0, shared by all experts          */
    float Kd;              /* derivative gain K_d >= 0                               */
    int32_t integral_mode; /* idb_integral_mode                                       */
    int32_t center;        /* 1: subtract the mean after the update (Eq. rapid-update) */
} idb_controller_cfg;

/* Controller state (host struct of device pointers, caller-owned).  The full
 * state of Alg. 1 is (bias, e_prev); step counts successful updates.  Start
 * from bias = e_prev = 0, step = 0.  Saving and restoring these buffers
 * checkpoints the controller exactly. */
typedef struct idb_controller_state {
    float* bias;     /* [E] expert bias b; also the routing input of the next step */
    float* e_prev;   /* [E] normalised load error of the previous update            */
    int64_t* step;   /* [1] number of successful updates                           */
    int32_t* status; /* [1] idb_status of the last update (OK, EMPTY_BATCH, INVALID_ARG) */
} idb_controller_state;

/* ---------------------------------------------------------------------------
 * Router step (Sec. 2.2; Eq. pid-routing; Eq. pid-error counts).
 *
 *   x           [T][d] hidden states, dtype as given, 16-byte aligned.
 *   W_g         [E][d] router matrix W_r, same dtype, row-major or in the
 *               packed layout of idb_router_pack_weight (weight_layout).
 *   bias        [E] fp32 expert bias b, read only (frozen within the step).
 *   T, d, E, K  tokens, hidden size, experts, experts per token.
 *               1 <= T <= 2^26; 1 <= K <= E; E <= 1024, E % 32 == 0 and
 *               K <= 32 (else IDB_ERR_UNSUPPORTED); d % 64 == 0 (bf16) or
 *               d % 32 == 0 (fp32), d <= 65536.
 *   expert_idx  [T][K] int32 out: the K experts with the largest s + b
 *               (fp32 add), in rank order: larger s + b first, lower expert
 *               index first among equal values (-0 == +0).
 *   gate_w      [T][K] fp32 out: gate_w[t][r] = s[t][idx_r] / den, den the
 *               fp32 sum of the selected unbiased scores in rank order
 *               (den == 0 gives 1/K).
 *   counts      [E] int32: counts[i] += number of tokens routed to expert i.
 *               Zeroed first unless accumulate_counts != 0 (microbatch
 *               summing, Alg. 1).
 *   scores_dump nullable [T][E] fp32 out, 16-byte aligned: the scores s the
 *               selection used (debug / parity; the arithmetic is unchanged).
 *   workspace   device scratch of at least idb_router_workspace_bytes().
 *   variant     0 = automatic tiling; other values force a tiling (see
 *               idb_router_variant_info).  Variants 1-5 (32x32 MFMA tiles)
 *               give identical outputs; variant 6 (16x16 tiles) accumulates
 *               the contraction in another order, so its scores can differ
 *               in the last fp32 bits.  Given its scores, every variant's
 *               selection, gate weights and counts are exact.
 * The T x E score matrix is never written to memory unless scores_dump is set.
 * ------------------------------------------------------------------------- */
size_t idb_router_workspace_bytes(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype, int32_t variant);

idb_status idb_router_forward(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                              const float* bias, int64_t T,
                              int32_t d, int32_t E, int32_t K, int32_t* expert_idx, float* gate_w,
                              int32_t* counts, int32_t accumulate_counts, float* scores_dump, void* workspace,
                              size_t workspace_bytes, int32_t variant, hipStream_t stream);

/* The two launches idb_router_forward makes, exposed so a caller can time or
 * overlap them separately.  Same arguments; calling score_select then merge
 * on one stream is exactly idb_router_forward.
 *   score_select: gate contraction, sigmoid, biased Top-K per expert slice
 *                 (and, when the tiling covers all experts in one slice, the
 *                 final outputs); zeroes counts unless accumulating.
 *   merge:        merges the slices' candidates into the final Top-K, gate
 *                 weights and counts; enqueues nothing for single-slice
 *                 tilings. */
idb_status idb_router_score_select(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                   const float* bias, int64_t T,
                                   int32_t d, int32_t E, int32_t K, int32_t* expert_idx, float* gate_w,
                                   int32_t* counts, int32_t accumulate_counts, float* scores_dump,
                                   void* workspace, size_t workspace_bytes, int32_t variant, hipStream_t stream);
idb_status idb_router_merge(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype, int32_t* expert_idx,
                            float* gate_w, int32_t* counts, void* workspace, size_t workspace_bytes,
                            int32_t variant, hipStream_t stream);

/* idb_router_score_select for measurement: the same arguments, checks and
 * outputs, with the fused router kernel started by an extended launch that
 * writes that kernel's own start and end timestamps into start_event and
 * stop_event (HIP events the caller created, e.g. with hipEventCreate; either
 * may be null, and with both null this is idb_router_score_select).  The
 * elapsed time between the two events is the kernel's execution time alone,
 * without the dispatch of the launch or the cost of separately recorded
 * events; a counts-zeroing launch that precedes the kernel (single-slice
 * tilings) is outside the interval.  The events must belong to the device
 * of `stream` and must not be recorded elsewhere until the kernel is done. */
idb_status idb_router_score_select_timed(const void* x, const void* W_g, idb_dtype dtype,
                                         idb_weight_layout weight_layout, const float* bias, int64_t T, int32_t d,
                                         int32_t E, int32_t K, int32_t* expert_idx, float* gate_w, int32_t* counts,
                                         int32_t accumulate_counts, float* scores_dump, void* workspace,
                                         size_t workspace_bytes, int32_t variant, hipStream_t stream,
                                         hipEvent_t start_event, hipEvent_t stop_event);

/* The router matrix in the layout the MFMA A operands are read in: for every
 * 16-expert block b, 128-byte chunk c of the rows and 64-byte half s < 2 of
 * the chunk, one contiguous 1 KB piece, at byte ((b*NCH + c)*2 + s)*1024 with
 * NCH = row bytes / 128, holds for lane slot l < 64 the bytes
 * [c*128 + 64 s + 16 (l/16), +16) of row 16 b + l%16.  A pure byte
 * permutation of W_g; packing once per weight update lets every router call
 * read W with fully coalesced loads.  W_packed must not overlap W_g; both
 * 16-byte aligned.  E % 32 == 0, d as for idb_router_forward. */
size_t idb_router_packed_weight_bytes(int32_t E, int32_t d, idb_dtype dtype);
idb_status idb_router_pack_weight(const void* W_g, idb_dtype dtype, int32_t E, int32_t d, void* W_packed,
                                  hipStream_t stream);

/* Tiling of a variant for a shape: out[0] = tokens per workgroup, out[1] =
 * expert slices, out[2] = waves per workgroup, out[3] = experts per wave,
 * out[4] = resolved variant id.  Returns IDB_ERR_UNSUPPORTED when the
 * variant cannot run the shape.  Host only, no HIP call. */
idb_status idb_router_variant_info(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype, int32_t variant,
                                   int32_t out[5]);

/* ---------------------------------------------------------------------------
 * Selection from given scores (Eq. pid-routing and the gate-weight rule of
 * Sec. 2.2, then the counts of Eq. pid-error): the router step without the
 * gate contraction.  scores [T][E] fp32, bias [E] fp32; outputs as for
 * idb_router_forward.  1 <= T <= 2^26, 1 <= K <= E; E <= 1024 and K <= 32
 * (else IDB_ERR_UNSUPPORTED).  Any E in that range.
 * ------------------------------------------------------------------------- */
idb_status idb_select_from_scores(const float* scores, const float* bias, int64_t T, int32_t E, int32_t K,
                                  int32_t* expert_idx, float* gate_w, int32_t* counts, int32_t accumulate_counts,
                                  hipStream_t stream);

/* ---------------------------------------------------------------------------
 * One ID controller update (Alg. 1, one iteration of one MoE layer; in SIGN
 * mode Eq. pid-deepseek).  counts [E] int32 are the loads summed over
 * microbatches (and data-parallel ranks).  With S = sum(counts):
 *   e_i  = (S - E n_i) / S, one correctly rounded fp64 division, then fp32
 *   de_i = e_i - e_prev_i
 *   g_i  = (e_prev_i > 0 and de_i > 0) or (e_prev_i < 0 and de_i < 0)
 *   b~_i = (b_i + K_i e_i) [+ K_d de_i if g_i], fp32, left to right, no FMA
 *   if center: b_i = b~_i - m, m = (fixed pairwise tree sum of b~ padded with
 *              +0 to a power of two) / E; else b_i = b~_i
 *   e_prev = e; step += 1; status = IDB_OK
 * S == 0: status = IDB_ERR_EMPTY_BATCH; a negative count: status =
 * IDB_ERR_INVALID_ARG; in both cases bias, e_prev and step are unchanged.
 * One single-workgroup launch.
 * ------------------------------------------------------------------------- */
idb_status idb_controller_update(const int32_t* counts, const idb_controller_cfg* cfg,
                                 const idb_controller_state* state, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Load statistics (Sec. 4.1, Eq. vio) from counts [E] int32, 1 <= E <= 1<<20:
 *   out[0] = MaxVio = (E max n - S) / S,  out[1] = MinVio = (S - E min n) / S,
 * each one fp64 division of an exact integer numerator; NaN for S == 0.
 * out is a device double[2].
 * ------------------------------------------------------------------------- */
idb_status idb_load_stats(const int32_t* counts, int32_t E, double* out_maxvio_minvio, hipStream_t stream);

/* One launch for both calls of an iteration's controller phase: writes
 * MaxVio/MinVio of counts into out_maxvio_minvio (exactly as idb_load_stats)
 * and applies the ID update (exactly as idb_controller_update), on stream.
 * Same argument rules as the two calls; out_maxvio_minvio must not be null. */
idb_status idb_controller_step(const int32_t* counts, const idb_controller_cfg* cfg,
                               const idb_controller_state* state, double* out_maxvio_minvio, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * One whole iteration of Alg. 1 for one batch and one MoE layer: the router
 * step with bias = state->bias (frozen while routing), then, once every token
 * is counted, MaxVio/MinVio of counts (when out_maxvio_minvio is not null)
 * and the ID update of state from counts.  The results are exactly those of
 * idb_router_forward (scores_dump = NULL) followed by idb_controller_step (or
 * idb_controller_update) on the same stream; E is cfg->E, the other arguments
 * as for those calls, with the same workspace size.  With accumulate_counts
 * the update uses the accumulated counts (the last microbatch of an
 * iteration).  Two launches for multi-slice tilings: the fused router kernel,
 * then the slice merge, whose last workgroup to finish applies the update.
 * The workspace must not be shared with a call still running on another
 * stream.
 * ------------------------------------------------------------------------- */
idb_status idb_router_step(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                           int64_t T, int32_t d, int32_t K, const idb_controller_cfg* cfg,
                           const idb_controller_state* state, int32_t* expert_idx, float* gate_w, int32_t* counts,
                           int32_t accumulate_counts, double* out_maxvio_minvio, void* workspace,
                           size_t workspace_bytes, int32_t variant, hipStream_t stream);

/* The second launch of idb_router_step on its own: after
 * idb_router_score_select on the same stream, with the same shape, variant,
 * workspace and outputs, it merges the expert slices (gate weights, counts)
 * and, once every token is counted, writes MaxVio/MinVio (when
 * out_maxvio_minvio is not null) and applies the ID update of state; for
 * one-slice tilings, whose router kernel already finished the outputs, it is
 * the controller step's launch.  idb_router_score_select (bias =
 * state->bias) followed by idb_router_merge_step enqueues exactly the kernels
 * of idb_router_step, with the same results, so a caller can time or overlap
 * the two launches separately.  The controller reads counts as the merge
 * leaves them (accumulated when score_select accumulated). */
idb_status idb_router_merge_step(int64_t T, int32_t d, int32_t K, idb_dtype dtype, const idb_controller_cfg* cfg,
                                 const idb_controller_state* state, int32_t* expert_idx, float* gate_w,
                                 int32_t* counts, double* out_maxvio_minvio, void* workspace, size_t workspace_bytes,
                                 int32_t variant, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * idb_router_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The call allocates nothing (no
 * hipMalloc, hipFree or allocating library routine): the workspace is a fixed
 * device array of IDB_NOALLOC_SCRATCH_BYTES inside the library, one copy per
 * device, held until the process ends.  Arguments and results are exactly
 * those of idb_router_step with workspace = that array.
 * - Size limit: the tiling's workspace (idb_router_workspace_bytes) must fit
 *   in IDB_NOALLOC_SCRATCH_BYTES, e.g. T <= 65536 at E = 768, K <= 10 on the
 *   default tiling; larger shapes return IDB_ERR_UNSUPPORTED and enqueue
 *   nothing.  One-slice tilings need no scratch.
 * - The stream must belong to the calling thread's current device (else
 *   IDB_ERR_INVALID_ARG).  The first call on a device looks up the array's
 *   address there (hipGetSymbolAddress) and keeps it.
 * - Every call on a device shares that device's array, which keeps the last
 *   call's contents; the router kernel clears what must start at zero (the
 *   merge's ticket) itself.  Calls that overlap on one device (other streams,
 *   other threads) race on the array and must be serialised by the caller.
 * ------------------------------------------------------------------------- */
#define IDB_NOALLOC_SCRATCH_BYTES ((size_t)16 * 1024 * 1024 + 256)
idb_status idb_router_step_noalloc(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                   int64_t T, int32_t d, int32_t K, const idb_controller_cfg* cfg,
                                   const idb_controller_state* state, int32_t* expert_idx, float* gate_w,
                                   int32_t* counts, int32_t accumulate_counts, double* out_maxvio_minvio,
                                   int32_t variant, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * All MoE layers' controller updates of one iteration in one launch (Alg. 1
 * runs per layer; one workgroup per layer), with the load statistics and the
 * update's diagnostics.
 *   counts    [L][E] int32, the layers' summed loads.
 *   state     bias and e_prev [L][E] fp32, step [L] int64, status [L] int32.
 *   out_stats nullable [L][2]: MaxVio, MinVio per layer (as idb_load_stats).
 *   out_diag  nullable [L][4] fp64 per layer:
 *     [0] active-gate fraction #{g_i = 1} / E of this update (Eq. rapid-gate;
 *         Sec. 3 reports its trajectory);
 *     [1] share of the assignments on the busiest 10% of experts, the
 *         m = ceil(E / 10) largest counts over S (balanced: m / E);
 *     [2] inactive-expert ratio #{n_i = 0} / E (Sec. 4.3);
 *     [3] mean |b_new - b_old| of this update (the bias drift of Sec. 3 is
 *         the same mean between checkpoints; fp64 over the fixed pairwise
 *         tree);
 *     each ratio one fp64 division; NaN x 4 for a layer whose update did not
 *     run (empty or invalid batch).
 * Each layer's bias, e_prev, step and status are exactly those of
 * idb_controller_update on that layer.  1 <= L <= 65535, cfg as for
 * idb_controller_update.
 * ------------------------------------------------------------------------- */
idb_status idb_controller_update_layers(const int32_t* counts, int32_t L, const idb_controller_cfg* cfg,
                                        const idb_controller_state* state, double* out_stats, double* out_diag,
                                        hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Routing entropies (Sec. 4.3), in nats, averaged over the T tokens:
 *   out[0] = mean H_topK, H_topK = -sum_r w_r log w_r over gate_w [T][K]
 *            (0 log 0 = 0);
 *   out[1] = mean H_full, H_full = -sum_e p_e log p_e, p_e = c_e / sum c,
 *            c_e = max(fl32(s_e + b_e), 0) over scores [T][E] and bias [E]
 *            (0 when every c_e is 0); NaN when scores is NULL.
 * Natural logarithms in fp64; deterministic (fixed partial sums in the
 * workspace, idb_routing_entropy_workspace_bytes() bytes, then added in
 * order).  out is a device double[2].  1 <= T <= 2^26, 1 <= K <= 32,
 * E <= 1024.
 * ------------------------------------------------------------------------- */
size_t idb_routing_entropy_workspace_bytes(void);
idb_status idb_routing_entropy(const float* gate_w, int64_t T, int32_t K, const float* scores, const float* bias,
                               int32_t E, void* workspace, size_t workspace_bytes, double* out, hipStream_t stream);

/* The same entropies for the auxiliary-loss router, whose full-pool selection
 * scores are the softmax probabilities over its logits (Sec. 4.3):
 *   out[0] = mean H_topK over gate_w [T][K] (as idb_routing_entropy);
 *   out[1] = mean H_full, H_full = -sum_e p_e log p_e, p = softmax(z) over the
 *            fp32 logits [T][E] (idb_aux_router_forward's logits_dump), taken
 *            as log Z - (sum_e t_e (z_e - M)) / Z with M the token's largest
 *            logit, t_e = exp(z_e - M) from the hardware fp32 exponential and
 *            Z = sum_e t_e, both sums in fp64.
 * Workspace and determinism as idb_routing_entropy; 1 <= T <= 2^26,
 * 1 <= K <= 32, 1 <= E <= 1024; finite logits. */
idb_status idb_routing_entropy_softmax(const float* gate_w, int64_t T, int32_t K, const float* logits, int32_t E,
                                       void* workspace, size_t workspace_bytes, double* out, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Quantile Balancing (Eq. pid-quantile, Eq. pid-quantile-def): the paper's
 * strongest baseline controller, on the same fused router.
 *
 * idb_qb_router_forward: idb_router_forward's outputs (identical values),
 * plus, for Quantile Balancing's update,
 *   alpha     [T] fp32 out: per token the (K+1)-th largest biased score
 *             fl32(s + b) in the order of Eq. pid-routing (-0 written +0);
 *   scores_t  [E][T] fp32 out: the scores s, expert-major.
 * Needs K + 1 <= E and K + 1 <= 32, and a workspace of at least
 * idb_qb_router_workspace_bytes() (K + 1 candidates per token and slice).
 *
 * idb_qb_update: for each expert j, with margins d_ij = fl32(s_ij - alpha_i)
 * (-0 read as +0) and k = ceil(T (E - K) / E) in exact integers, q_j = the
 * k-th smallest d_.j (the 1 - K/E quantile as the inverted empirical CDF),
 * Q_j = -q_j, and bias[j] = Q_j for rho == 0, else the EMA variant
 * fl32(fl32(rho bias[j]) + fl32(fl32(1 - rho) Q_j)).  scores_t [E][T] and
 * alpha [T] as written by idb_qb_router_forward; bias [E] is updated in
 * place.  1 <= T <= 2^26, 1 <= K < E <= 1024, 0 <= rho < 1.  One workgroup
 * per expert (exact radix select of the k-th margin).
 *   counts            nullable [E] int32 in: the step's assignments per
 *                     expert (as written by idb_qb_router_forward);
 *   out_maxvio_minvio nullable fp64 [2] out: MaxVio, MinVio of those counts
 *                     (Eq. vio; the same bits as idb_load_stats), written by
 *                     the first workgroup in the same launch.
 * counts and out_maxvio_minvio are both given or both null (else
 * IDB_ERR_INVALID_ARG, nothing launched); out_maxvio_minvio 8-byte aligned.
 * ------------------------------------------------------------------------- */
size_t idb_qb_router_workspace_bytes(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype,
                                     int32_t variant);
idb_status idb_qb_router_forward(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                 const float* bias, int64_t T, int32_t d, int32_t E, int32_t K, int32_t* expert_idx,
                                 float* gate_w, int32_t* counts, int32_t accumulate_counts, float* scores_t,
                                 float* alpha, void* workspace, size_t workspace_bytes, int32_t variant,
                                 hipStream_t stream);
idb_status idb_qb_update(const float* scores_t, const float* alpha, int64_t T, int32_t E, int32_t K, float rho,
                         float* bias, const int32_t* counts, double* out_maxvio_minvio, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Auxiliary-loss balancing's forward statistics (Eq. pid-auxloss), on the
 * fused router.  The router keeps no bias: with logits z = W_g x (as
 * idb_router_forward) and p = softmax(z) over all E experts,
 *   expert_idx [T][K] int32 out: the K largest z per token in rank order
 *              (softmax preserves the order; equal logits: lowest index
 *              first), decided on the fp32 logits;
 *   gate_w     [T][K] fp32 out: the selected p renormalised,
 *              exp(z_r - z_top) / (fp32 sum of those in rank order);
 *   counts     [E] int32 out: assignments per expert;
 *   f          [E] fp64 out: f_i = n_i / T;
 *   P          [E] fp64 out: P_i = (1/T) sum over the tokens of p_i, from
 *              per-tile fp32 column sums (M = the token's largest logit,
 *              p = exp(z - M) / sum exp(z - M)) added in fp64 in a fixed
 *              order, so repeated calls give identical bits;
 *   loss       fp64 out (device scalar): alpha * sum_i f_i P_i.
 *   out_maxvio_minvio nullable fp64 [2] out: MaxVio, MinVio of the counts
 *              (as idb_load_stats).
 *   logits_dump nullable [T][E] fp32 out: the logits the selection ranked.
 * counts, f, P and the loss are written by the second launch from per-tile
 * rows (no atomics: identical bits on every call).
 * Only tilings whose workgroups cover all E experts run this (the statistics
 * need each token's whole softmax in one workgroup): E <= 768 for bf16, E <=
 * 128 for fp32; other shapes or variants return IDB_ERR_UNSUPPORTED.  Other
 * limits as for idb_router_forward; alpha finite.  The workspace (at least
 * idb_aux_router_workspace_bytes(), 16-byte aligned) holds the per-tile rows
 * and a ticket; it must not be shared with a call still running on another
 * stream.  Two launches: the fused router kernel, then the statistics kernel.
 * ------------------------------------------------------------------------- */
size_t idb_aux_router_workspace_bytes(int64_t T, int32_t d, int32_t E, int32_t K, idb_dtype dtype,
                                      int32_t variant);
idb_status idb_aux_router_forward(const void* x, const void* W_g, idb_dtype dtype, idb_weight_layout weight_layout,
                                  int64_t T, int32_t d, int32_t E, int32_t K, double alpha, int32_t* expert_idx,
                                  float* gate_w, int32_t* counts, double* f, double* P, double* loss,
                                  double* out_maxvio_minvio, float* logits_dump, void* workspace,
                                  size_t workspace_bytes, int32_t variant, hipStream_t stream);

/* Static description of a status code; message of the last failing call on
 * this thread (empty string if none). */
const char* idb_status_string(idb_status s);
const char* idb_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* IDB_H */
