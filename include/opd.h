/*
 * opd.h - C ABI of the learner-time on-policy-distillation (OPD) loss for
 * AMD Instinct MI355X (gfx950).
 *
 * One call takes the student logits of N generated tokens over a vocabulary
 * of V entries, plus the finite teacher-score cache those tokens carry, and
 * returns the per-token loss and its gradient with respect to every logit
 * (Sec. 4.1, "Stage 3: Student update": the learner recomputes log p_theta
 * on the cached actions).  All work runs in HIP kernels on the caller's
 * stream; nothing is computed on the host.
 *
 * Conventions shared by every entry point
 *  - Array pointers are DEVICE pointers owned by the caller.  The library
 *    keeps no reference to them after the call returns and allocates no
 *    device memory.
 *  - Logit rows have stride `ld` elements (ld >= V).  logits, dlogits and
 *    teacher_logits must be 16-byte aligned and ld * element_size must be a
 *    multiple of 16 bytes (ld % 8 == 0 when any of them is bf16, else
 *    ld % 4 == 0).  Columns [V, ld) of dlogits are never written.
 *  - Calls are stream-ordered and asynchronous.  Argument errors are
 *    reported synchronously, before anything is launched; a HIP launch
 *    failure returns OPD_ERR_HIP.  Faults in the DATA (a cached id outside
 *    [0, V), NaN or infinite logits) never fault the device: an out-of-range
 *    id makes that row's loss NaN and fills its dlogits row with NaN, and
 *    NaN/Inf logits propagate into that row's outputs.
 *  - N may be as large as INT32_MAX: calls whose grid would exceed HIP's
 *    limit of 2^32 work-items launch over consecutive row chunks.
 *  - Results are deterministic: repeated calls with the same inputs produce
 *    bitwise-identical outputs (fixed-order reductions, no float atomics).
 *  - Entry points hold no mutable global state and are safe to call from
 *    several host threads (each call on its own stream and buffers).
 */
#ifndef OPD_H
#define OPD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OPD_VERSION 5
/* Largest cached support size k, and largest sample count M. */
#define OPD_K_MAX 256

typedef enum opd_status {
  OPD_OK = 0,
  OPD_ERR_NULL = -1,      /* a pointer the estimator needs is NULL */
  OPD_ERR_SHAPE = -2,     /* N < 0, V < 2, V >= 2^31, or ld < V */
  OPD_ERR_SUPPORT = -3,   /* k or M outside [1, min(V, OPD_K_MAX)], or RKL_MC1 with M != 1 */
  OPD_ERR_DTYPE = -4,     /* unknown logits or dlogits dtype */
  OPD_ERR_ALIGN = -5,     /* a logit/gradient pointer or row stride is not 16-byte aligned */
  OPD_ERR_WORKSPACE = -6, /* split-vocabulary path forced with a missing or short workspace */
  OPD_ERR_ESTIMATOR = -7, /* unknown estimator */
  OPD_ERR_FLAGS = -8,     /* unknown or contradictory flag bits */
  OPD_ERR_HIP = -9,       /* a HIP runtime call or kernel launch failed */
  OPD_ERR_PARAM = -10,    /* invalid scalar option (clip_eps of a clipped estimator), or
                             coverage_out for an estimator without a cached support */
  OPD_ERR_SCRATCH = -11   /* opd_loss_fwd_bwd_noalloc: the call needs more scratch than
                             OPD_NOALLOC_SCRATCH_BYTES */
} opd_status;

/*
 * Estimators.  Notation of Sec. 3: p_theta = softmax(z) the current student,
 * q the teacher, p_old the stale behaviour policy.  For token t with logits
 * z (row of `logits`), L = log sum_j exp(z_j) and log p_theta(j) = z_j - L.
 *
 * OPD_FKL_TOPK  Forward KL on the cached support S = {idx[t, 0..k)}, teacher
 *               and student both renormalised on S (Sec. 3, "Sparse and
 *               sampled implementations"; normalisers of App. A.1):
 *                 loss = sum_S q~ (log q~ - log p~),
 *                 dloss/dz_{a_i} = p~_i - q~_i, zero off S.
 * OPD_RKL_TOPK  Sparse reverse KL D_R^S = KL(p~ || q~) (App. A.1), support
 *               held fixed:  dloss/dz_{a_i} = p~_i ((log p~_i - log q~_i) - D_R^S).
 *               Renormalisation cancels L, so both top-k estimators read only
 *               the k cached logits unless lse_out is requested.
 * OPD_RKL_MC1   One-sample MC reverse KL with old-to-current importance
 *               ratio and the advantage recomputed under the current student,
 *               unclipped (Sec. 5.1, L_theta^noclip):
 *                 loss = -rho(a) sg(A_theta(a)),  A_theta = log q - log p_theta,
 *                 rho = p_theta(a) / p_old(a).   Requires M == 1.
 * OPD_RKL_MC    M-sample average of the same surrogate (Sec. 6.2; App. E):
 *                 loss = -(1/M) sum_i rho(a_i) sg(A_theta(a_i)),
 *                 dloss/dz_j = c p_theta(j) - (1/M) sum_{i: a_i = j} rho_i A_i,
 *               c = -loss.  Samples are iid with replacement; repeated ids are
 *               separate terms, accumulated in ascending i.
 * OPD_FKL_DENSE Full-vocabulary forward KL against dense teacher logits
 *               (Sec. 3, eq. dense-forward-kl): gradient p_theta - q.
 * OPD_RKL_DENSE Full-vocabulary reverse KL (Sec. 3, eq. dense-reverse-kl and
 *               eq. reverse-kl-gradient): gradient p_j ((log p_j - log q_j) - D_R).
 *
 * The remaining members of the surrogate ablation of Sec. 5.1, on the same
 * M behaviour samples as OPD_RKL_MC.  With rho_bar = clip(rho, 1 - eps,
 * 1 + eps), eps = opts->clip_eps, and A_old = log q - log p_old (rollout-time,
 * from teacher_logp and behav_logp):
 * OPD_RKL_MC_CLIP      L_theta^clip = -(1/M) sum_i min(rho_i A_theta,i, rho_bar_i A_theta,i)
 * OPD_RKL_MC_OLD       L_old^noclip = -(1/M) sum_i rho_i A_old,i
 * OPD_RKL_MC_OLD_CLIP  L_old^clip   = -(1/M) sum_i min(rho_i A_old,i, rho_bar_i A_old,i),
 *                      the PPO-style adaptation
 * The advantage is a stop-gradient weight.  Where the min selects the
 * clipped term outside [1 - eps, 1 + eps] the sample contributes no gradient;
 * ties (rho inside the range) count as unclipped.
 * OPD_RKL_MC_NOIS      MC without importance sampling (the App. F ablation):
 *                      the samples are used as if drawn from p_theta,
 *                      L = -(1/M) sum_i sg(A_theta,i) log p_theta(a_i), gradient
 *                      -(1/M) sum_i A_theta,i (1[j = a_i] - p_j).  behav_logp
 *                      is not read (may be NULL).
 *
 * Truncated top-k: the dense KLs of Sec. 3 with the action sum cut to the
 * cached support S = {idx[t, 0..k)} and no renormalisation (p_theta and q keep
 * their full-vocabulary normalisers, so teacher_logp must be normalised over
 * the full vocabulary).  Not a KL in general (can be negative); the gradient
 * is dense, so the row is read.
 * OPD_FKL_TOPK_TRUNC   sum_S q (log q - log p_theta);
 *                      dloss/dz_j = Z_q^S p_j - q_j 1[j in S], Z_q^S = q(S)
 * OPD_RKL_TOPK_TRUNC   sum_S p_theta (log p_theta - log q);
 *                      dloss/dz_j = p_j 1[j in S](log p_j - log q_j + 1)
 *                                   - p_j sum_S p (log p - log q + 1)
 */
typedef enum opd_estimator {
  OPD_FKL_TOPK = 0,
  OPD_RKL_TOPK = 1,
  OPD_RKL_MC1 = 2,
  OPD_RKL_MC = 3,
  OPD_FKL_DENSE = 4,
  OPD_RKL_DENSE = 5,
  OPD_RKL_MC_CLIP = 6,
  OPD_RKL_MC_OLD = 7,
  OPD_RKL_MC_OLD_CLIP = 8,
  OPD_RKL_MC_NOIS = 9,
  OPD_FKL_TOPK_TRUNC = 10,
  OPD_RKL_TOPK_TRUNC = 11
} opd_estimator;

typedef enum opd_dtype { OPD_F32 = 0, OPD_BF16 = 1 } opd_dtype;

/* Flags (opd_opts.flags). */
#define OPD_FLAG_SKIP_MASKED 1u   /* leave dlogits rows of masked tokens untouched */
#define OPD_FLAG_FORCE_ROWWISE 2u /* one workgroup per token row, whatever N is */
#define OPD_FLAG_FORCE_SPLITV 4u  /* split each row over several workgroups (needs workspace) */

/*
 * The teacher-score cache of N tokens (Sec. 4.1, Stage 1 and Stage 2).
 * Row-major device arrays; which fields are read depends on the estimator.
 *   idx            [N, k] int32  top-k support S (the top-k estimators, renormalised
 *                  and truncated); ids must be distinct within a row
 *                  (opd_validate_cache checks this)
 *   sampled_ids    [N, M] int32  behaviour-policy samples a_i ~ p_old (the
 *                  MC estimators, OPD_RKL_MC1 and OPD_RKL_MC_*); repeats allowed
 *   teacher_logp   [N, k] or [N, M] fp32  log q(a|s) at idx / sampled_ids,
 *                  normalised over the full vocabulary (the top-k estimators
 *                  renormalise on S, so any per-row constant cancels there)
 *   behav_logp     [N, M] fp32  log p_old(a|s) at sampled_ids (MC only),
 *                  recorded per token by the rollout policy
 *   teacher_logits [N, ld] dense teacher logits (dense estimators only),
 *                  same dtype and stride as the student logits
 */
typedef struct opd_cache {
  const int32_t* idx;
  const int32_t* sampled_ids;
  const float* teacher_logp;
  const float* behav_logp;
  const void* teacher_logits;
} opd_cache;

/*
 * grad_scale    gamma: dlogits[t, :] = gamma * mask[t] * dloss_t/dz_t; 1.0 gives
 *               the gradient of the masked sum of per-token losses.  Reductions
 *               over tokens (token mean, sequence mean) are the caller's: they
 *               are a choice of gamma.
 * dlogits_dtype OPD_F32 (default) or OPD_BF16 (round to nearest even).
 * flags         OPD_FLAG_* bits.
 * clip_eps      clip range eps of the clipped estimators; must be positive
 *               and finite for them (the paper uses 0.2, App. B, Table 3);
 *               ignored otherwise.
 * A NULL opts pointer means {1.0f, OPD_F32, 0, 0.2f}.
 */
typedef struct opd_opts {
  float grad_scale;
  int32_t dlogits_dtype;
  uint32_t flags;
  float clip_eps;
} opd_opts;

/*
 * Fused forward + backward of the OPD loss over N token rows.
 *
 *   logits        [N, ld] student logits, dtype OPD_F32 or OPD_BF16
 *   N, V, ld      tokens, vocabulary size, row stride (elements)
 *   cache         see opd_cache; must not be NULL
 *   estimator     opd_estimator
 *   k             support size for the top-k estimators (else ignored)
 *   M             samples per token for the MC estimators (else ignored)
 *   mask          [N] uint8, nullable (NULL = every token valid).  A masked
 *                 token (mask == 0) has loss 0, lse_out 0, gathered_out 0, and
 *                 a zero dlogits row (untouched with OPD_FLAG_SKIP_MASKED);
 *                 its logits are not read.
 *   opts          nullable, see opd_opts
 *   loss          [N] fp32 per-token loss (the MC loss is the surrogate value,
 *                 an unbiased estimate of the dense reverse KL, and can be
 *                 negative)
 *   dlogits       [N, ld] gradient, dtype opts->dlogits_dtype; may not alias
 *                 logits
 *   lse_out       [N] fp32 log sum_j exp(z_j), nullable.  For the top-k
 *                 estimators, requesting it adds one read of the logits.
 *   gathered_out  [N, k or M] fp32 student logits at the cached ids (exact
 *                 widening), nullable; not produced by the dense estimators.
 *   coverage_out  [N, 2] fp32 support coverage, nullable: the restricted
 *                 normalisers of App. A.1 on the cached support S,
 *                 Z_p^S = sum_{a in S} p_theta(a|s) (the student's mass on S)
 *                 and Z_q^S = sum_i exp(teacher_logp[t, i]) (the teacher's),
 *                 each cached entry counted once; 0 and 0 for a masked token.
 *                 A stale support (Sec. 6) shows as Z_p^S falling away from
 *                 Z_q^S.  Only the estimators that read a support (the
 *                 renormalised and truncated top-k) take it (else
 *                 OPD_ERR_PARAM); for the renormalised ones it adds one read
 *                 of the logits, as lse_out does.
 *   workspace     device scratch for the split-vocabulary path, nullable;
 *   workspace_bytes  its size.  The split path is taken for small N (or when
 *                 forced) only if workspace_bytes >= opd_workspace_bytes(...);
 *                 otherwise the row-per-workgroup path runs.
 *   stream        hipStream_t to launch on (NULL = default stream)
 * Returns OPD_OK or an opd_status error.  N == 0 is a no-op returning OPD_OK.
 */
int opd_loss_fwd_bwd(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                     const opd_cache* cache, int32_t estimator, int32_t k, int32_t M,
                     const uint8_t* mask, const opd_opts* opts, float* loss, void* dlogits,
                     float* lse_out, float* gathered_out, float* coverage_out, void* workspace,
                     size_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * fused forward + backward as opd_loss_fwd_bwd, with the same arguments
 * except the workspace, the same kernels and bitwise the same results.  The
 * split-vocabulary path keeps its per-(row, chunk) statistics in a static
 * device array of OPD_NOALLOC_SCRATCH_BYTES that the library holds on each
 * GPU it runs on until the process ends (its address is looked up once per
 * device, on the first call that needs it, with that device current).  The
 * call allocates nothing: no hipMalloc, hipFree or allocating library call.
 *   - A call whose split path needs more than OPD_NOALLOC_SCRATCH_BYTES
 *     (opd_workspace_bytes(...) of the same arguments) returns
 *     OPD_ERR_SCRATCH when the split path is forced (OPD_FLAG_FORCE_SPLITV);
 *     unforced, such a call runs the row-per-workgroup path, which needs no
 *     scratch.  (Unforced split calls, below 64 rows, need at most 126 KiB.)
 *   - Every record the split path reads is written earlier in the same call,
 *     so nothing carries over from the previous call's contents.
 *   - All calls on one GPU share that GPU's array: calls that overlap in time
 *     on one GPU (on different streams, or from several host threads) race
 *     and may return wrong results.  Serialise them.
 * Other errors as for opd_loss_fwd_bwd.
 */
#define OPD_NOALLOC_SCRATCH_BYTES (1u << 20)
int opd_loss_fwd_bwd_noalloc(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                             const opd_cache* cache, int32_t estimator, int32_t k, int32_t M,
                             const uint8_t* mask, const opd_opts* opts, float* loss,
                             void* dlogits, float* lse_out, float* gathered_out,
                             float* coverage_out, void* stream);

/* OPD_NOALLOC_SCRATCH_BYTES of the built library. */
size_t opd_noalloc_scratch_bytes(void);

/*
 * Bytes of workspace opd_loss_fwd_bwd uses for these arguments (0 when the
 * call takes the row-per-workgroup path): the split-vocabulary path's
 * per-(row, chunk) statistics records, N * P * 32 bytes.  Pure host function:
 * the answer depends only on its arguments.  Invalid arguments return 0.
 */
size_t opd_workspace_bytes(int64_t N, int64_t V, int32_t dtype, int32_t estimator, int32_t k,
                           int32_t M, uint32_t flags);

/*
 * Checks a cache against the preconditions of the estimator and ADDS the
 * number of violations to *violations (a device int32 the caller zeroes):
 *   - ids outside [0, V);
 *   - repeated ids within a top-k row: a support S is a set of actions, and
 *     the restricted normalisers and renormalised distributions on S
 *     (App. A.1) count each action once.  Repeats within an MC row are legal,
 *     since the m samples are drawn iid with replacement (Sec. 6.2; App. E),
 *     and are not counted;
 *   - non-finite teacher_logp (and behav_logp for the estimators with an
 *     importance ratio or A_old): a log-probability the cache records for an
 *     action it holds is finite.
 * Each bad entry counts once, each repeated top-k pair once.  Stream-ordered;
 * read the counter after synchronising.  Dense estimators have no cache to
 * check (returns OPD_OK).  Errors: OPD_ERR_ESTIMATOR, OPD_ERR_SHAPE,
 * OPD_ERR_SUPPORT, OPD_ERR_NULL, OPD_ERR_HIP.
 */
int opd_validate_cache(const opd_cache* cache, int32_t estimator, int64_t N, int64_t V,
                       int32_t k, int32_t M, int32_t* violations, void* stream);

/*
 * Building the cache (Sec. 4.1, Stage 1 "Student rollout" and Stage 2
 * "Teacher scoring").  Each call reads N rows of logits (the rollout policy
 * p_old for Stage 1, the teacher for Stage 2) with the same dtype, ld and
 * alignment rules as opd_loss_fwd_bwd, and writes per-row results.  A masked
 * row (mask[t] == 0) is not read and gets 0 in every output.  lse_out, when
 * not NULL, receives log sum_j exp(z_j) per row.  No workspace; one
 * workgroup per row.
 *
 * opd_sample_actions: M iid draws per row from softmax(z), as the rollout
 *   makes them (temperature 1, no top-p or top-k truncation; App. B), by
 *   inversion: draw i is the first index whose cumulative probability (index
 *   order) exceeds uniforms[t, i].  The uniforms are supplied by the caller
 *   ([N, M] fp32 in [0, 1)), so the draws are a deterministic function of
 *   them.  The CDF is evaluated in double precision (terms exp(z_j - max) to
 *   about 1.5e-15 relative, double sums), so a draw is the one exact arithmetic
 *   gives unless uniforms[t, i] lies within about 1e-14 of a cumulative value;
 *   terms follow double's gradual underflow, -inf logits have exactly zero
 *   mass, and a drawn id always has nonzero probability.
 *     sampled_ids [N, M] int32 out; logp [N, M] fp32 out (nullable) =
 *     log softmax(z) at the draw, the rollout-time log-probability the MC
 *     estimators read as behav_logp.  A uniform outside [0, 1) (or NaN), or a
 *     row with a NaN or +inf logit or no finite logit, gives id -1, logp NaN.
 *     1 <= M <= OPD_K_MAX.
 *
 * opd_topk_support: the k largest logits of each row, S = TopK(softmax(z), k)
 *   (Sec. 5: S_old at rollout time, or a teacher-selected support at scoring
 *   time), in descending order; equal values are ordered by lower index.
 *   The order is the IEEE-754 total order of the values with -0 equal to +0
 *   (a +NaN ranks above +inf, a -NaN below -inf).
 *     idx [N, k] int32 out; logp [N, k] fp32 out (nullable) = log softmax(z)
 *     at idx.  1 <= k <= min(V, OPD_K_MAX).
 *
 * opd_score_actions: log softmax(z) at given ids (teacher scoring of cached
 *   actions, or rollout log-probs of a given support).
 *     ids [N, K] int32 in (repeats allowed); logp [N, K] fp32 out, NaN for an
 *     id outside [0, V).  1 <= K <= OPD_K_MAX.
 *
 * Errors as for opd_loss_fwd_bwd: OPD_ERR_DTYPE, OPD_ERR_SHAPE,
 * OPD_ERR_SUPPORT (M, k or K out of range), OPD_ERR_ALIGN, OPD_ERR_NULL (a
 * required pointer), OPD_ERR_HIP.  N == 0 is a no-op returning OPD_OK.
 */
int opd_sample_actions(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                       int32_t M, const float* uniforms, const uint8_t* mask, int32_t* sampled_ids,
                       float* logp, float* lse_out, void* stream);
int opd_topk_support(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld, int32_t k,
                     const uint8_t* mask, int32_t* idx, float* logp, float* lse_out, void* stream);
int opd_score_actions(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                      const int32_t* ids, int32_t K, const uint8_t* mask, float* logp,
                      float* lse_out, void* stream);

/*
 * Diagnostics of the Monte-Carlo estimator: the importance-ratio tail that
 * Sec. 5.2 tracks (the p99 of rho_theta, Fig. 5) and the variance of the
 * m-sample estimator at a fixed prefix and over a sequence (App. E, Table 6).
 * Inputs are per token t what an MC loss call returns or reads: lse [N]
 * (lse_out, log sum_j exp z_j), gathered [N, M] (gathered_out, the student
 * logits at the M draws), teacher_logp and behav_logp [N, M] (the cache).
 * With log p = gathered - lse, A = teacher_logp - log p, rho = exp(log p -
 * behav_logp), the one-sample terms are X = -rho A (the loss is their mean).
 * Outputs (device fp32, each nullable):
 *   row_mean [N]     (1/M) sum_i X_i
 *   row_var [N]      unbiased variance of X_i over i (NaN when M = 1)
 *   row_rho_max [N]  max_i rho_i (NaN ratios ignored)
 *   rho_quantile [1] nearest-rank quantile of rho over all valid entries:
 *                    the r-th smallest, r = max(1, ceil(quantile * n)) (in
 *                    double, from the fp32 quantile); NaN ratios rank above
 *                    +inf
 *   clip_frac [1]    fraction of valid entries with |rho - 1| > clip_eps
 *   ratio_local [n_groups], ratio_seq [n_groups]
 *                    variance ratios for group sizes m = group_sizes[k]
 *                    (host array; M a multiple of m, M / m >= 2): the draws
 *                    of a token split into M / m groups of m consecutive
 *                    draws with means Y_g;
 *                      ratio_local = sum_t var_g(Y_g) / sum_t row_var_t,
 *                    and, with tokens [s seq_len, (s + 1) seq_len) forming
 *                    sequence s and S_g its valid-token average of Y_g,
 *                      ratio_seq = sum_s var_g(S_g) / sum_s var_i(S1_i)
 *                    (S1: the same with single draws).  var is unbiased.
 *                    ratio_seq needs seq_len > 0.
 * Masked tokens (mask[t] == 0) are excluded and get 0 in the per-token
 * outputs.  The workspace (size from opd_mc_diag_workspace_bytes, 16-byte
 * aligned) holds intermediates; the quantile is exact (radix selection with
 * integer histograms); sums run in a fixed order.
 * Errors: OPD_ERR_SHAPE (N < 0 or N >= 2^32 / 64: the batch reductions run
 * in one grid), OPD_ERR_SUPPORT (M outside [1, OPD_K_MAX]),
 * OPD_ERR_PARAM (quantile outside (0, 1], clip_eps negative or not finite,
 * more than 8 or invalid group sizes, seq_len < 0, ratio_seq without
 * seq_len), OPD_ERR_NULL, OPD_ERR_WORKSPACE, OPD_ERR_HIP.
 */
typedef struct opd_mc_diag {
  float* row_mean;
  float* row_var;
  float* row_rho_max;
  float* rho_quantile;
  float* clip_frac;
  float* ratio_local;
  float* ratio_seq;
} opd_mc_diag;

/* Workspace bytes of opd_mc_diagnostics (0 for invalid arguments). */
size_t opd_mc_diag_workspace_bytes(int64_t N, int32_t M, const int32_t* group_sizes,
                                   int32_t n_groups, int64_t seq_len);

int opd_mc_diagnostics(const float* lse, const float* gathered, const float* teacher_logp,
                       const float* behav_logp, int64_t N, int32_t M, const uint8_t* mask,
                       float quantile, float clip_eps, const int32_t* group_sizes,
                       int32_t n_groups, int64_t seq_len, const opd_mc_diag* out, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Static description of a status code ("ok", "null pointer", ...); a code
 * outside opd_status gives "unknown status".  Never NULL. */
const char* opd_status_string(int status);

/* OPD_VERSION of the built library. */
int opd_version(void);

#ifdef __cplusplus
}
#endif
#endif /* OPD_H */
