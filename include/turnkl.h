/*
 * turnkl.h -- fused turn-aware reverse-KL distillation loss for MI355X (gfx950).
 *
 * This is the data-parallel hot path of one TurnOPD training step (arXiv
 * 2607.05804).  For a packed batch of multi-turn agent trajectories it
 * computes, in one stream-ordered call:
 *
 *   1. the (trajectory, turn) segments of the batch and their supervised-token
 *      counts (Sec. 3: a trace is x, o_1, r_1, ..., o_T, r_T and only response
 *      tokens carry the loss mask; Sec. 4.4: n_t supervised tokens at turn t,
 *      N = sum_t n_t);
 *   2. the progressive turn-normalised token weights (Sec. 5.2:
 *      q_traj_t = n_t / sum_j n_j, q_turn_t = 1 / T,
 *      q_blend_t = (1 - alpha) q_traj_t + alpha q_turn_t; App. D, Algorithm 1:
 *      w_blend = (1 - alpha) w_traj + alpha w_turn), averaged over
 *      trajectories as the seq-mean-token-mean base aggregation does;
 *   3. the per-token reverse KL D_KL(p_student || p_teacher) over the full
 *      vocabulary (Sec. 3, Eq. opd-rkl; temperature 1, App. D);
 *   4. its gradient with respect to the student logits (the teacher is
 *      frozen, Sec. 3): G[i, v] = grad_scale * w_i * p_s(v) * (log p_s(v) -
 *      log p_t(v) - KL_i);
 *   5. the loss L = sum_i w_i KL_i (App. D, Algorithm 1), together with its
 *      alpha = 0 and alpha = 1 forms;
 *   6. per-turn-index statistics of the per-token KL (Sec. 4.3, Eq.
 *      observed-turn-kl: K_t; Sec. 5.1 and App. D: survivors n_t and K_t feed
 *      the rollout-depth controller; Sec. 4.4: s_t, the turn's loss share).
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers owned by the caller unless marked "host".
 *     The library allocates no memory and keeps no per-call state; all
 *     scratch lives in the caller's workspace, except for
 *     turnkl_fwd_bwd_noalloc, whose scratch is a fixed array in the library.
 *   - Measurement and test hooks are declared in turnkl_testing.h.
 *   - Work is enqueued on `stream` and is asynchronous; the success path never
 *     synchronises with the host.  Calls on distinct workspaces may run
 *     concurrently; calls sharing a workspace must be stream-ordered.
 *   - Argument errors detectable on the host are returned synchronously before
 *     anything is enqueued and leave every output untouched.
 *   - Data-dependent errors (bad ids or mask) are detected on the device and
 *     recorded in the workspace; turnkl_get_status returns them.
 */
#ifndef TURNKL_H_
#define TURNKL_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of the logits and of the gradient. */
typedef enum {
  TURNKL_BF16 = 0, /* bfloat16; the gradient is rounded to nearest even */
  TURNKL_F32 = 1,
} turnkl_dtype;

/* Return codes. */
typedef enum {
  TURNKL_OK = 0,
  TURNKL_ERR_INVALID_ARG = -1,   /* NULL, size, stride, dtype or alpha out of range */
  TURNKL_ERR_ALIAS = -2,         /* grad_out overlaps an input other than exact in-place */
  TURNKL_ERR_WORKSPACE = -3,     /* workspace smaller than turnkl_workspace_bytes() */
  TURNKL_ERR_UNSORTED = -4,      /* device: trajectory or turn ids out of order */
  TURNKL_ERR_TURN_RANGE = -5,    /* device: turn id outside [0, max_turns) */
  TURNKL_ERR_PAD_MASK = -6,      /* device: padding token (traj_id < 0) with mask 1 */
  TURNKL_ERR_HIP = -7,           /* a HIP runtime call failed */
  TURNKL_ERR_SYNC_TIMEOUT = -8,  /* device: cross-workgroup exchange did not complete */
  TURNKL_ERR_TOPK_ID = -9,       /* device: a top-K support id outside [0, vocab) */
  TURNKL_ERR_OUTCOME = -10,      /* device: outcome flag not constant over a trajectory */
  TURNKL_ERR_SCRATCH = -11,      /* turnkl_fwd_bwd_noalloc: problem larger than its scratch */
} turnkl_status;

/* Statistics of one turn index t over the supervised tokens at that turn. */
typedef struct {
  int64_t n_tokens;  /* supervised tokens at turn t, summed over trajectories */
  int64_t n_traj;    /* trajectories with >= 1 supervised token at turn t (survivors n_t) */
  double kl_mean;    /* pooled mean per-token KL at turn t (K_t); 0 if n_tokens == 0 */
  double kl_m2;      /* sum over those tokens of (KL - kl_mean)^2 */
  double kl_var;     /* kl_m2 / n_tokens (population variance); 0 if n_tokens == 0 */
  double loss_mass;  /* sum over those tokens of w_i * KL_i (turn t's share of L) */
} turnkl_turn_stat;

/*
 * Optional variants of the weights and statistics, shared by turnkl_fwd_bwd
 * and turnkl_fwd_bwd_topk.  A NULL options pointer, or a zeroed struct, means
 * none of them.
 *
 * Turn-support floor (App. D, full-configuration table: the internal blend's
 * min_floor = 8 and min_frac = 0.15 give n_min = max(min_floor,
 * ceil(min_frac * n_traj)); Sec. 7.2 calls the turns that enough trajectories
 * reach "valid turns").  The paper does not say how n_min enters the turn
 * term; this library reads it as follows.  n_traj is B, the trajectories of
 * the call with a supervised token, and frac * B is rounded once in double
 * before the ceiling.  Turn t is valid when its survivor count n_t (the
 * trajectories of the call with a supervised token at t) is >= n_min.  The
 * turn term of trajectory b gives each of its T_vb valid supervised turns
 * 1 / T_vb and its other turns 0; a trajectory with no valid supervised turn
 * uses its trajectory term n_bt / N_b instead.  So
 *   w_i = m_i / B * ((1 - alpha) / N_b + alpha * u_bt),
 *   u_bt = [t valid] / (T_vb * n_bt) if T_vb > 0, else 1 / N_b,
 * the weights still sum to 1, L_turn uses alpha = 1 of the same form and
 * L_traj is unchanged.  support_floor = 0 with support_frac = 0 (or any
 * n_min <= 1) gives the plain weights.
 *
 * Outcome split (Sec. 4.2: K_t^fail and K_t^succ, the per-turn KL means over
 * failed and successful rollouts; G_t = K_t^fail - K_t^succ).  success holds
 * one flag per token (nonzero = the trajectory succeeded; flags of padding
 * tokens are ignored) and must be constant over each trajectory's tokens, or
 * the device reports TURNKL_ERR_OUTCOME at the first token where it changes
 * (after the other checks at that token).  outcome_stats_out receives the
 * per-turn statistics of the failed trajectories' tokens in entries
 * [0, max_turns) and of the successful ones' in [max_turns, 2 * max_turns),
 * with the fields and the accumulate_stats rule of turn_stats_out; the two
 * halves partition turn_stats_out's counts and loss mass.
 *
 * Per-token outputs (device, caller-owned, or NULL).  Neither may overlap the
 * logits, the gradient outputs, token_kl_out or each other
 * (TURNKL_ERR_ALIAS); they are unspecified after a device-detected error.
 *   token_weight_out  [n_tokens] float: w_i, the weight of token i in
 *                     L = sum_i w_i KL_i (Sec. 5.2; App. D, Algorithm 1), as
 *                     described at turnkl_fwd_bwd and above, rounded to float
 *                     from double; 0 for unsupervised and padding tokens.
 *   token_lse_out     [n_tokens x 2] float, row-major: for a supervised token
 *                     the log-partition functions log sum_v exp(zs_i[v]) and
 *                     log sum_v exp(zt_i[v]) of its student and teacher rows
 *                     (natural log; Sec. 3, Eq. opd-rkl: log p(v) = z[v] minus
 *                     this value at temperature 1), so the caller can form
 *                     log-probabilities without another pass over the rows.
 *                     On the top-K path the sums run over the token's support
 *                     S_i (of the student logits and the teacher values).
 *                     Unsupervised tokens' rows are never read: both entries
 *                     are NaN.
 */
typedef struct {
  int32_t support_floor;   /* >= 0; 0 with support_frac 0: no floor */
  double support_frac;     /* in [0, 1] */
  const uint8_t* success;  /* device [n_tokens] outcome flags, or NULL */
  turnkl_turn_stat* outcome_stats_out;  /* device [2 * max_turns], or NULL */
  float* token_weight_out; /* device [n_tokens], or NULL */
  float* token_lse_out;    /* device [n_tokens * 2], or NULL */
} turnkl_options;

/*
 * Bytes of device workspace turnkl_fwd_bwd needs for this problem (host
 * function, no device access; a pure function of its arguments).
 *
 * aligned_rows != 0 promises that every row of the student logits, the
 * teacher logits and the gradient starts on a 16-byte boundary (base pointers
 * and row strides in bytes are multiples of 16).  The size then covers the
 * 16-byte vector path, which every call with such rows takes when vocab
 * fills whole 16-byte vectors (vocab a multiple of 8 in bf16, of 4 in fp32).
 * aligned_rows = 0 covers whichever path a call takes.  The two differ in the
 * row kernel's exchange slots: at vocab = 151,936 in bf16, 96 bytes per token
 * on the vector path (3 chunks per row) and 608 on the element-wise path (19
 * chunks).  A call whose path needs more than the workspace it is given
 * returns TURNKL_ERR_WORKSPACE and enqueues nothing.
 *
 * Returns 0 when the arguments are invalid (n_tokens < 0, vocab < 1, unknown
 * dtype, max_turns < 1).  The workspace needs no initialisation; it must be
 * 256-byte aligned.
 */
size_t turnkl_workspace_bytes(int64_t n_tokens, int64_t vocab, int dtype, int32_t max_turns,
                              int aligned_rows);

/*
 * Fused forward + backward of the turn-blended reverse-KL loss.
 *
 * student_logits, teacher_logits   [n_tokens x vocab] row-major, row strides
 *                                  ld_student / ld_teacher (elements, >= vocab),
 *                                  element type `dtype`.  Rows of unsupervised
 *                                  tokens are never read.  Logits must be finite.
 * turn_id, traj_id, loss_mask      [n_tokens] each.  A segment is a maximal run
 *                                  of consecutive tokens with equal (traj_id,
 *                                  turn_id); traj_id < 0 marks padding, which
 *                                  belongs to no segment and must have mask 0.
 *                                  Trajectory ids must increase from segment to
 *                                  segment and turn ids must increase within a
 *                                  trajectory (so a turn is one contiguous run);
 *                                  0 <= turn_id < max_turns.  loss_mask[i] != 0
 *                                  marks a supervised response token.
 * alpha                            blend coefficient in [0, 1] (Sec. 5.2);
 *                                  turnkl_alpha_schedule computes the paper's
 *                                  schedule.
 * grad_scale                       multiplies the gradient (the upstream
 *                                  dLoss_total / dL); finite.
 * loss_out                         [3] float: L_blend = sum_i w_i KL_i, L_traj
 *                                  (alpha = 0) and L_turn (alpha = 1).  NaN x 3
 *                                  when the device detects a data error.
 * grad_out, ld_grad                [n_tokens x vocab] gradient in `dtype`, row
 *                                  stride ld_grad >= vocab.  May equal
 *                                  student_logits with ld_grad == ld_student
 *                                  (in place); any other overlap with either
 *                                  input is TURNKL_ERR_ALIAS.  Unsupervised rows
 *                                  are written as zeros.  NULL: forward only.
 * turn_stats_out, max_turns        [max_turns] statistics indexed by turn id, or
 *                                  NULL.  accumulate_stats != 0 merges this
 *                                  batch into the existing contents (counts and
 *                                  loss mass add; means and m2 merge exactly as
 *                                  if the tokens had been pooled; turns without
 *                                  supervised tokens in this batch are left as
 *                                  they are); 0 overwrites.
 * token_kl_out                     [n_tokens] float per-token KL (0 for
 *                                  unsupervised tokens), or NULL.
 * options                          host pointer to turnkl_options, or NULL.
 *                                  success and outcome_stats_out go together
 *                                  (success may be NULL when n_tokens == 0);
 *                                  outcome_stats_out must not overlap
 *                                  turn_stats_out (TURNKL_ERR_ALIAS).
 * workspace, workspace_bytes       scratch of at least turnkl_workspace_bytes().
 *
 * Weights: w_i = m_i / B * ((1 - alpha) / N_b + alpha / (T_b * n_bt)) for token
 * i of trajectory b at turn t, where n_bt is the supervised count of the
 * segment, N_b = sum_t n_bt, T_b = #{t : n_bt > 0} and B = #{b : N_b > 0}; the
 * weights sum to 1.  A turn-support floor in `options` replaces the turn term
 * as described at turnkl_options.  An empty batch or one without supervised
 * tokens yields a zero loss, a zero gradient and zero (or unchanged, when
 * accumulating) stats.
 *
 * Returns TURNKL_OK once everything is enqueued, or a negative host-detected
 * error with nothing enqueued.  Device-detected data errors are reported by
 * turnkl_get_status; after one, loss_out holds NaN and grad_out, turn_stats_out
 * and token_kl_out are unspecified.
 */
int turnkl_fwd_bwd(const void* student_logits, int64_t ld_student, const void* teacher_logits,
                   int64_t ld_teacher, int dtype, int64_t n_tokens, int64_t vocab,
                   const int32_t* turn_id, const int32_t* traj_id, const uint8_t* loss_mask,
                   double alpha, float grad_scale, float* loss_out, void* grad_out,
                   int64_t ld_grad, turnkl_turn_stat* turn_stats_out, int32_t max_turns,
                   int accumulate_stats, float* token_kl_out, const turnkl_options* options,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Waits for `stream`, then returns the device-side status of the last
 * turnkl_fwd_bwd call that used `workspace`: TURNKL_OK or a data error
 * (TURNKL_ERR_UNSORTED / _TURN_RANGE / _PAD_MASK / _OUTCOME, or _TOPK_ID for
 * the top-K call; the earliest offending token in token order decides; at one
 * token a padding-mask error, then a range error, then an ordering error,
 * then an outcome-flag error), or TURNKL_ERR_SYNC_TIMEOUT; TURNKL_ERR_HIP if
 * the read-back fails.
 *
 * TURNKL_ERR_SYNC_TIMEOUT.  The full-vocabulary row kernel splits a long row
 * over several workgroups that exchange partial sums through the workspace;
 * a workgroup waits for its row mates for a bounded number of polls (2^22,
 * with a short sleep between polls: seconds of wall time).  The wait can only
 * expire when the row mates cannot be scheduled, i.e. when other work holds
 * the GPU's compute slots for that long.  Then every other workgroup that
 * waits for a row mate gives up within 256 further polls (rows whose chunks
 * all arrive are still computed, and discarded), the kernels after the row
 * kernel skip their work, loss_out holds NaN, the gradient, the statistics
 * and the per-token outputs are unspecified, and the workspace is ready for
 * the next call.  The caller may simply repeat the call.  No other kernel of
 * the call waits on another workgroup, and the top-K call never returns this
 * code.
 */
int turnkl_get_status(const void* workspace, hipStream_t stream);

/*
 * Copies the segment table of the last call on `workspace` (made with the same
 * n_tokens) into caller device arrays of capacity n_tokens: first token,
 * length, trajectory id, turn id and supervised count of every segment, in
 * token order.  *n_seg (host) receives the count.  Waits for `stream`.
 * Returns TURNKL_OK, TURNKL_ERR_INVALID_ARG or TURNKL_ERR_HIP.
 */
int turnkl_get_segments(const void* workspace, int64_t n_tokens, hipStream_t stream,
                        int32_t* n_seg, int32_t* seg_start, int32_t* seg_len, int32_t* seg_traj,
                        int32_t* seg_turn, int32_t* seg_nsup);

/*
 * The paper's blend schedule (Sec. 5.2; App. D, Algorithm 1):
 * alpha_k = clip((k / K - s) / (e - s), 0, 1).  When e <= s the schedule is a
 * step: 1 once k / K >= s, else 0.  K < 1 returns NaN.  Host function.
 */
double turnkl_alpha_schedule(int64_t k, int64_t K, double s, double e);

/* Static description of a return code.  Host function. */
const char* turnkl_status_string(int status);

/*
 * turnkl_fwd_bwd without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Arguments, results and errors are those
 * of turnkl_fwd_bwd, except:
 *   - The scratch is an array inside the library of
 *     TURNKL_NOALLOC_SCRATCH_BYTES (32 MiB), one in the memory of every GPU
 *     that runs the library, held until the process ends.  A problem whose
 *     workspace would be larger (turnkl_workspace_bytes with aligned_rows = 1
 *     when the rows are 16-byte aligned, else 0) returns TURNKL_ERR_SCRATCH
 *     and enqueues nothing.  With aligned rows at vocab = 151,936 in bf16
 *     that is above about 158,000 tokens (212 bytes per token).
 *   - The call allocates nothing (no hipMalloc, hipFree or allocating library
 *     routine).  Its first call on a device looks up the device address of
 *     that device's array once.  `stream` must belong to the current device.
 *   - status_out (device int32, 4-byte aligned, or NULL) receives TURNKL_OK
 *     or the device-detected error when the call's last kernel runs: the role
 *     turnkl_get_status plays for a workspace.
 *   - All calls on one GPU share its array.  Calls ordered on one stream are
 *     safe; calls that can overlap in time on one GPU (different streams or
 *     host threads without ordering between them) race and give unspecified
 *     results.  Every call initialises what it reads of the array.
 */
#define TURNKL_NOALLOC_SCRATCH_BYTES (32u << 20)

int turnkl_fwd_bwd_noalloc(const void* student_logits, int64_t ld_student,
                           const void* teacher_logits, int64_t ld_teacher, int dtype,
                           int64_t n_tokens, int64_t vocab, const int32_t* turn_id,
                           const int32_t* traj_id, const uint8_t* loss_mask, double alpha,
                           float grad_scale, float* loss_out, void* grad_out, int64_t ld_grad,
                           turnkl_turn_stat* turn_stats_out, int32_t max_turns,
                           int accumulate_stats, float* token_kl_out,
                           const turnkl_options* options, int32_t* status_out,
                           hipStream_t stream);

/* ------------------------------------------------------------------------
 * Top-K variant of the loss: the reverse KL on the teacher's top-K support
 * (App. D: Algorithm 1 computes top-K reverse-KL token losses; the
 * configuration table sets the teacher's top-K support size, K = 50).  The
 * paper does not print the formula; this library renormalises both
 * distributions on the support S_i of token i:
 *   p^_s(v) = exp(a_v) / sum_{u in S_i} exp(a_u),  p^_t(v) likewise from the
 *   teacher's values b_v on S_i (logits or log-probabilities: a per-row
 *   constant cancels),
 *   KL_i = sum_{v in S_i} p^_s(v) (log p^_s(v) - log p^_t(v))   (Sec. 3, Eq.
 *   opd-rkl restricted to S_i),
 *   G[i, v] = grad_scale * w_i * p^_s(v) (log p^_s(v) - log p^_t(v) - KL_i)
 *   for v in S_i and 0 for every other id.
 * Segments, weights, losses and per-turn statistics are those of
 * turnkl_fwd_bwd, computed from these KL_i.
 * ------------------------------------------------------------------------ */

/* Workspace bytes for turnkl_fwd_bwd_topk (host); 0 for invalid arguments. */
size_t turnkl_topk_workspace_bytes(int64_t n_tokens, int32_t k, int32_t max_turns);

/*
 * Top-K fused forward + backward.  Arguments as for turnkl_fwd_bwd, except:
 *   teacher_ids    device, int32 [n_tokens][ld_topk]: row i holds the K
 *                  distinct ids of S_i in [0, vocab) (a duplicate id counts
 *                  twice and makes the dense gradient's entry unspecified);
 *   teacher_vals   device, float32 [n_tokens][ld_topk]: the teacher's values
 *                  at those ids;
 *   k              1 .. min(1024, vocab);
 *   grad_out       optional dense gradient, dtype [n_tokens][ld_grad], zero
 *                  off the support; may equal student_logits with the same
 *                  leading dimension (in place: every student logit is read
 *                  before any gradient row is written);
 *   grad_topk_out  optional, float32 [n_tokens][ld_grad_topk]: G on the
 *                  support, in the order of teacher_ids (zeros for
 *                  unsupervised tokens);
 *   workspace      at least turnkl_topk_workspace_bytes(n_tokens, k, max_turns).
 * Only the rows of supervised tokens are read from student_logits, teacher_ids
 * and teacher_vals.  Errors: as turnkl_fwd_bwd (TURNKL_ERR_ALIAS when either
 * gradient output overlaps an input or the other output), plus the device
 * error TURNKL_ERR_TOPK_ID for an id outside [0, vocab) in a supervised row.
 * The profiling hook of turnkl_profile_row_kernel (turnkl_testing.h)
 * brackets the top-K kernels (support rows, then the dense gradient).
 */
int turnkl_fwd_bwd_topk(const void* student_logits, int64_t ld_student, int dtype,
                        int64_t n_tokens, int64_t vocab, const int32_t* teacher_ids,
                        const float* teacher_vals, int64_t ld_topk, int32_t k,
                        const int32_t* turn_id, const int32_t* traj_id, const uint8_t* loss_mask,
                        double alpha, float grad_scale, float* loss_out, void* grad_out,
                        int64_t ld_grad, float* grad_topk_out, int64_t ld_grad_topk,
                        turnkl_turn_stat* turn_stats_out, int32_t max_turns, int accumulate_stats,
                        float* token_kl_out, const turnkl_options* options, void* workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Adaptive rollout-depth controller (Sec. 5.1; App. D, Algorithm 1 and the
 * full-configuration table).  HOST functions: all pointers are host memory,
 * nothing touches the GPU.  They consume the per-turn statistics that
 * turnkl_fwd_bwd wrote for a probe batch (after the caller copies the
 * turnkl_turn_stat array to the host), and return the rollout depth cap that
 * the rollout engine applies on the following steps.
 *
 * Turn indices are 0-based throughout; the cap adds 1 to turn an index into a
 * number of turns.  round() is round-half-to-even.
 *
 *   probe batch   K_t = kl_mean[t], n_t = n_traj[t] of the batch's stats;
 *   efficiency    m_t = [K_t]_+ n_t / n_0 (0 when n_0 = 0),
 *                 q_t = m_t / (sum_j m_j + eps), H_eff = round(sum_t t q_t);
 *   coverage      with L_i the turn counts of the batch's successful
 *                 trajectories (or of all trajectories, for the paper's
 *                 full-population variant), refreshed only when at least
 *                 min_cov_traj of them are given:
 *                 H_cov = min{H >= 0 : #{i : L_i - 1 <= H} / n >= p}
 *                 (0 until first refreshed, then kept);
 *   update        H_ctrl = max(H_eff, H_cov),
 *                 Hbar_k = (1 - ema_alpha) Hbar_{k-1} + ema_alpha H_ctrl on
 *                 probe steps (Hbar_0 = h_max), unchanged otherwise;
 *   plan          cap_k = clip(round(Hbar_{k-1}) + 1, h_min, h_max); step k
 *                 (k = 1, 2, ...) is a probe when k <= warmup_steps or
 *                 k % probe_interval == 0; a probe rolls out to h_max, any
 *                 other step to cap_k.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t h_min, h_max;        /* clamp of the applied cap (2, 50) */
  int32_t warmup_steps;        /* steps 1..warmup_steps are probes (3) */
  int32_t probe_interval;      /* and every probe_interval-th step (8) */
  int32_t min_cov_traj;        /* successful trajectories needed to refresh H_cov (8) */
  double coverage_quantile;    /* p in (0, 1] (0.80) */
  double ema_alpha;            /* in [0, 1] (0.30); not the loss-blend alpha */
  double eps;                  /* >= 0, guard of the q_t normaliser (1e-12) */
} turnkl_depth_config;

typedef struct {
  double h_bar;      /* EMA of H_ctrl; h_max after init */
  double h_eff_bar;  /* last centroid before rounding; -1 before the first probe */
  int32_t h_eff;     /* last efficiency centroid; -1 before the first probe */
  int32_t h_cov;     /* coverage floor; 0 until first refreshed */
  int32_t h_ctrl;    /* last max(H_eff, H_cov); -1 before the first probe */
  int32_t n_probes;  /* probe updates so far */
} turnkl_depth_state;

/* Fill `cfg` (host) with the values of App. D's configuration table. */
void turnkl_depth_default_config(turnkl_depth_config* cfg);

/* Initialise `st` (host) for `cfg`.  TURNKL_ERR_INVALID_ARG for a null pointer
 * or a configuration outside the ranges above (h_min >= 1, h_max >= h_min,
 * warmup_steps >= 0, probe_interval >= 1, min_cov_traj >= 0). */
int turnkl_depth_init(const turnkl_depth_config* cfg, turnkl_depth_state* st);

/* Step `step` (>= 1): the cap, whether the step is a probe (0/1) and the
 * rollout depth to use (host outputs).  Does not modify the state. */
int turnkl_depth_plan(const turnkl_depth_config* cfg, const turnkl_depth_state* st, int64_t step,
                      int32_t* cap, int32_t* probe, int32_t* rollout_depth);

/* One probe update.  `stats` (host) holds n_turns >= 1 entries of the probe
 * batch's per-turn statistics; `success_lengths` (host, may be NULL when
 * n_success == 0) the turn counts (>= 1) of its successful trajectories.
 * TURNKL_ERR_INVALID_ARG for null pointers, bad sizes or a length < 1; the
 * state is then left unchanged. */
int turnkl_depth_update(const turnkl_depth_config* cfg, turnkl_depth_state* st,
                        const turnkl_turn_stat* stats, int32_t n_turns,
                        const int32_t* success_lengths, int64_t n_success);

/* ------------------------------------------------------------------------
 * Turn-level loss-allocation diagnostics (HOST functions over the per-turn
 * statistics of one batch, as turnkl_fwd_bwd writes them, copied to the host).
 *
 *   s_t            Sec. 4.4: loss_mass[t] / sum_u loss_mass[u], the share of
 *                  the batch's loss mass that turn t carries (s_t^traj when
 *                  the statistics were taken at alpha = 0; the budget the
 *                  blended objective spends otherwise, Sec. 7.2).  0 for every
 *                  turn when the batch has no loss mass.
 *   reliable prefix  the P leading turns t = 0, 1, ... whose survivor count
 *                  n_t is at least max(n_min, 1), n_min = max(support_floor,
 *                  ceil(support_frac * n_traj)) (App. D's floor formula; with
 *                  (8, 0.10) and n_traj = n_0 it is the per-step part of the
 *                  plotting rule of Sec. 4.1).
 *   thirds         the first and the last ceil(P / 3) turns of the prefix.
 *   Table 1 / 3    shallow and deep budget (sums of s_t over each third),
 *                  deep support (mean over the deep third of n_t / n_0) and
 *                  the deep/shallow raw-KL ratio (mean of K_t over the deep
 *                  third / mean over the shallow third; NaN when P = 0 or the
 *                  shallow mean is 0).
 *   G_t            Sec. 4.2: K_t^fail - K_t^succ from the outcome statistics
 *                  of turnkl_options; NaN where either outcome has no
 *                  supervised token at turn t.
 * All return TURNKL_OK, or TURNKL_ERR_INVALID_ARG for null pointers, n_turns
 * < 1, n_traj < 0, support_floor < 0 or support_frac outside [0, 1].
 * ------------------------------------------------------------------------ */
typedef struct {
  int64_t n_min;            /* support floor applied to the prefix */
  int32_t prefix;           /* P */
  int32_t third;            /* ceil(P / 3); 0 when P = 0 */
  double shallow_budget;    /* sum of s_t over the shallow third */
  double deep_budget;       /* sum of s_t over the deep third */
  double deep_support;      /* mean of n_t / n_0 over the deep third */
  double deep_shallow_kl;   /* mean K_t, deep third / shallow third */
} turnkl_budget;

/* share (host) [n_turns] receives s_t for stats (host) [n_turns]. */
int turnkl_loss_share(const turnkl_turn_stat* stats, int32_t n_turns, double* share);

/* The Table 1 / Table 3 figures of one batch into *out (host). */
int turnkl_budget_report(const turnkl_turn_stat* stats, int32_t n_turns, int64_t n_traj,
                         int32_t support_floor, double support_frac, turnkl_budget* out);

/* gap (host) [n_turns] receives G_t from outcome_stats (host) [2 * n_turns]:
 * failed trajectories first, then successful ones. */
int turnkl_outcome_gap(const turnkl_turn_stat* outcome_stats, int32_t n_turns, double* gap);

#ifdef __cplusplus
}
#endif

#endif /* TURNKL_H_ */
