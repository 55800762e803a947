/*
 * The oracle: a plain, slow, double-precision CPU implementation of the
 * learner-time on-policy-distillation (OPD) loss and its gradient with respect
 * to the student logits.  It is test infrastructure: only the tests, the smoke
 * check and the benchmark's CPU-baseline leg use it, and it shares no code
 * with the GPU library.
 */
#ifndef OPD_ORACLE_H
#define OPD_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORACLE_FKL_TOPK = 0,  /* forward KL on a cached support, renormalised (Sec. 3; App. A.1) */
  ORACLE_RKL_TOPK = 1,  /* reverse KL on a cached support, renormalised (App. A.1) */
  ORACLE_RKL_MC1 = 2,   /* one-sample MC, A_theta, no clip (Sec. 5.1, L_theta^noclip) */
  ORACLE_RKL_MC = 3,    /* m-sample MC average (Sec. 6.2; App. E) */
  ORACLE_FKL_DENSE = 4, /* full-vocabulary forward KL (Sec. 3, eq. dense-forward-kl) */
  ORACLE_RKL_DENSE = 5, /* full-vocabulary reverse KL (Sec. 3, eq. dense-reverse-kl) */
  ORACLE_RKL_MC_CLIP = 6,     /* L_theta^clip (Sec. 5.1, two-by-two ablation) */
  ORACLE_RKL_MC_OLD = 7,      /* L_old^noclip (Sec. 5.1) */
  ORACLE_RKL_MC_OLD_CLIP = 8, /* L_old^clip, the PPO-style adaptation (Sec. 5.1) */
  ORACLE_RKL_MC_NOIS = 9,     /* MC without importance sampling (App. F ablation) */
  ORACLE_FKL_TOPK_TRUNC = 10, /* forward KL summed over S, full-vocabulary normalisers */
  ORACLE_RKL_TOPK_TRUNC = 11  /* reverse KL summed over S, full-vocabulary normalisers */
};

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

/* One token row, everything in double.
 *   z[V]      student logits;  y[V] teacher logits (dense estimators, else NULL)
 *   ids[K]    cached support (top-k) or behaviour samples (MC)
 *   tau[K]    teacher log-probs log q(a|s) at ids (full-vocabulary normalised)
 *   beta[K]   behaviour log-probs log p_old(a|s) at ids (MC only, else NULL)
 *   gamma     gradient scale; valid = 0 marks a padded token
 *   eps       clip range of the clipped surrogates (ignored otherwise)
 * Outputs: *loss, grad[V] (nullable), *lse (log-partition of z; nullable),
 * gathered[K] = z at ids (nullable).  Returns 0, or -1 on bad arguments
 * (id out of range, K < 1, missing input). */
int oracle_row(int est, const double* z, const double* y, int64_t V, const int32_t* ids,
               const double* tau, const double* beta, int K, double gamma, double eps, int valid,
               double* loss, double* grad, double* lse, double* gathered);

/* Rows of stored inputs (fp32, or bf16 bit patterns widened exactly), rows
 * processed by `nthreads` threads (0 = all).  logits/teacher_logits are
 * [n_rows, ld]; ids/tau/beta are [n_rows, K]; mask [n_rows] is nullable;
 * grad is [n_rows, V] (nullable), lse [n_rows], gathered [n_rows, K]
 * (nullable).  Returns 0 or the first row error. */
int oracle_rows(int est, int dtype, const void* logits, const void* teacher_logits, int64_t n_rows,
                int64_t V, int64_t ld, const int32_t* ids, const float* tau, const float* beta,
                int K, const uint8_t* mask, double gamma, double eps, double* loss, double* grad,
                double* lse, double* gathered, int nthreads);

/* Support coverage (App. A.1's restricted normalisers): Z_p^S = sum over the
 * cached support of p_theta, Z_q^S = sum of exp(tau_i).  The batch form
 * writes [n_rows, 2] (Z_p^S, Z_q^S), zeros for masked rows. */
int oracle_support_coverage(const double* z, int64_t V, const int32_t* ids, const double* tau,
                            int K, double* zp, double* zq);
int oracle_coverage_rows(int dtype, const void* logits, int64_t n_rows, int64_t V, int64_t ld,
                         const int32_t* ids, const float* tau, int K, const uint8_t* mask,
                         double* cov, int nthreads);

/* Building the cache (Sec. 4.1, Stages 1 and 2).  Rows in double unless
 * stored.  See opd_oracle.c for the definitions.
 *   oracle_cdf         F[j] = sum_{l<=j} softmax(z)_l, summed in index order
 *   oracle_sample_row  M draws by inversion of F at uniforms u[M] in [0, 1)
 *   oracle_topk_row    the k largest of a stored row, ties by lower index
 *   oracle_score_row   log softmax(z) at ids (NaN for an id outside [0, V)) */
int oracle_cdf(const double* z, int64_t V, double* F);
int oracle_sample_row(const double* z, int64_t V, const float* u, int M, int32_t* ids,
                      double* logp, double* lse);
int oracle_topk_row(int dtype, const void* row, int64_t V, int k, int32_t* idx, double* logp,
                    double* lse);
int oracle_score_row(const double* z, int64_t V, const int32_t* ids, int K, double* logp,
                     double* lse);
/* Batch driver: op 0 sample, 1 top-k, 2 score (see opd_oracle.c). */
int oracle_cache_rows(int op, int dtype, const void* logits, int64_t n_rows, int64_t V, int64_t ld,
                      int K, const float* uniforms, const uint8_t* mask, int32_t* ids,
                      double* logp, double* lse, int nthreads);

/* Diagnostics of the MC estimator (Sec. 5.2, Fig. 5; App. E): per-token mean,
 * unbiased variance and maximum importance ratio of the one-sample terms,
 * the q-quantile (nearest rank) of the ratio over the batch, the fraction of
 * ratios outside [1 - eps, 1 + eps], and fixed-prefix and sequence-level
 * variance ratios for group sizes m.  See opd_oracle.c. */
int oracle_mc_diagnostics(const double* lse, const double* gathered, const float* tau,
                          const float* beta, int64_t N, int M, const uint8_t* mask, double q,
                          double eps, const int* group_sizes, int n_groups, int64_t seq_len,
                          double* row_mean, double* row_var, double* row_rhomax,
                          double* rho_quantile, double* clip_frac, double* ratio_local,
                          double* ratio_seq);

/* Number of threads oracle_rows uses for nthreads = 0. */
int oracle_max_threads(void);

#ifdef __cplusplus
}
#endif
#endif
