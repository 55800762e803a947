/*
 * The oracle for the learner-time OPD loss: a plain double-precision CPU
 * implementation, written from the paper's definitions, for testing only.
 * Nothing here is blocked, fused or reordered beyond what the definitions
 * state, so each function can be checked against the paper by eye.
 *
 * Test infrastructure: only tests/, the smoke check and the benchmark's
 * CPU-baseline leg may load or call this code.  It shares no code with the
 * GPU library.
 *
 * Notation (Sec. 3): at a fixed prefix s, p_theta = softmax(z) is the current
 * student, q the teacher, p_old the stale behaviour policy.  The cache holds,
 * per token, either a support S = {a_i} with teacher log-probs
 * tau_i = log q(a_i|s), or M behaviour samples a_i ~ p_old with
 * tau_i = log q(a_i|s) and beta_i = log p_old(a_i|s).
 */
#include "opd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* log sum_j exp(x_j): the log-partition of a logit row, two sweeps. */
static double log_partition(const double* x, int64_t V) {
  double m = x[0];
  for (int64_t j = 1; j < V; ++j)
    if (x[j] > m) m = x[j];
  double s = 0.0;
  for (int64_t j = 0; j < V; ++j) s += exp(x[j] - m);
  return m + log(s);
}

/*
 * Sparse top-k KL on a cached support S, both distributions renormalised on S
 * (Sec. 3, "Sparse and sampled implementations"; App. A.1):
 *   Z_p^S = sum_{u in S} p_theta(u|s),   Z_q^S = sum_{u in S} q(u|s),
 *   p~(a) = p_theta(a|s) / Z_p^S,        q~(a) = q(a|s) / Z_q^S   (a in S).
 * Forward:  KL(q~ || p~) = sum_S q~ (log q~ - log p~);
 *           d/dz_{a_i} = p~_i - q~_i, zero off S.
 * Reverse:  D_R^S = KL(p~ || q~) = -sum_S p~ (log q~ - log p~);
 *           d/dz_{a_i} = p~_i ((log p~_i - log q~_i) - D_R^S), zero off S.
 * The support is held fixed during the update (App. A.1).
 */
static void topk_kl(int reverse, const double* z, int64_t V, double L, const int32_t* ids,
                    const double* tau, int K, double gamma, double* loss, double* grad) {
  double Zp = 0.0, Zq = 0.0;
  for (int i = 0; i < K; ++i) {
    Zp += exp(z[ids[i]] - L); /* p_theta(a_i|s) */
    Zq += exp(tau[i]);        /* q(a_i|s) */
  }
  const double logZp = log(Zp), logZq = log(Zq);
  double kl = 0.0;
  for (int i = 0; i < K; ++i) {
    const double log_pt = (z[ids[i]] - L) - logZp; /* log p~(a_i) */
    const double log_qt = tau[i] - logZq;          /* log q~(a_i) */
    if (reverse)
      kl += exp(log_pt) * (log_pt - log_qt);
    else
      kl += exp(log_qt) * (log_qt - log_pt);
  }
  *loss = kl;
  if (!grad) return;
  for (int64_t j = 0; j < V; ++j) grad[j] = 0.0;
  for (int i = 0; i < K; ++i) {
    const double log_pt = (z[ids[i]] - L) - logZp;
    const double log_qt = tau[i] - logZq;
    const double pt = exp(log_pt), qt = exp(log_qt);
    grad[ids[i]] += reverse ? gamma * pt * ((log_pt - log_qt) - kl) : gamma * (pt - qt);
  }
}

/*
 * Monte-Carlo reverse KL with old-to-current importance sampling and the
 * advantage recomputed under the current student, no clipping
 * (Sec. 5.1, L_theta^noclip; Sec. 6.2 and App. E for m samples):
 *   A_theta(a) = log q(a|s) - log p_theta(a|s)        (stop-gradient)
 *   rho(a)     = p_theta(a|s) / p_old(a|s)
 *   L_m        = -(1/m) sum_i rho(a_i) sg(A_theta(a_i)).
 * Samples are iid with replacement, so ids may repeat; each occurrence is a
 * separate term.  With A held fixed, d rho_i / d z_j = rho_i (1[j = a_i] - p_j),
 * so  dL_m/dz_j = c p_j - (1/m) sum_{i: a_i = j} rho_i A_i,
 * with c = (1/m) sum_i rho_i A_i = -L_m.
 */
static void mc_rkl(const double* z, int64_t V, double L, const int32_t* ids, const double* tau,
                   const double* beta, int M, double gamma, double* loss, double* grad) {
  double c = 0.0;
  for (int i = 0; i < M; ++i) {
    const double logp = z[ids[i]] - L; /* log p_theta(a_i|s) */
    const double A = tau[i] - logp;    /* A_theta(a_i, s) */
    const double rho = exp(logp - beta[i]);
    c += rho * A;
  }
  c /= (double)M;
  *loss = -c;
  if (!grad) return;
  for (int64_t j = 0; j < V; ++j) grad[j] = gamma * c * exp(z[j] - L);
  for (int i = 0; i < M; ++i) {
    const double logp = z[ids[i]] - L;
    const double A = tau[i] - logp;
    const double rho = exp(logp - beta[i]);
    grad[ids[i]] -= gamma * rho * A / (double)M;
  }
}

/*
 * Truncated top-k KL: the dense KL of Sec. 3 with the sum over actions cut to
 * the cached support S and no renormalisation (p_theta and q keep their
 * full-vocabulary normalisers):
 *   forward  sum_{a in S} q(a) (log q(a) - log p_theta(a)),
 *            d/dz_j = Z_q^S p_j - q_j 1[j in S];
 *   reverse  sum_{a in S} p_theta(a) (log p_theta(a) - log q(a)),
 *            d/dz_j = p_j 1[j in S] (log p_j - log q_j + 1)
 *                     - p_j sum_{a in S} p(a) (log p(a) - log q(a) + 1).
 * Unlike the renormalised forms, the gradient is dense (every p_j moves).
 */
static void topk_truncated(int reverse, const double* z, int64_t V, double L, const int32_t* ids,
                           const double* tau, int K, double gamma, double* loss, double* grad) {
  double kl = 0.0, mass = 0.0;
  for (int i = 0; i < K; ++i) {
    const double logp = z[ids[i]] - L;
    if (reverse) {
      kl += exp(logp) * (logp - tau[i]);
      mass += exp(logp) * (logp - tau[i] + 1.0);
    } else {
      kl += exp(tau[i]) * (tau[i] - logp);
      mass += exp(tau[i]);
    }
  }
  *loss = kl;
  if (!grad) return;
  for (int64_t j = 0; j < V; ++j) grad[j] = gamma * (reverse ? -mass : mass) * exp(z[j] - L);
  for (int i = 0; i < K; ++i) {
    const double logp = z[ids[i]] - L;
    grad[ids[i]] += reverse ? gamma * exp(logp) * (logp - tau[i] + 1.0) : -gamma * exp(tau[i]);
  }
}

/*
 * The rest of the two-by-two surrogate family of Sec. 5.1 (the equation
 * block of the ablation), over behaviour samples a_i ~ p_old:
 *   rho_i     = p_theta(a_i) / p_old(a_i),  rho_bar_i = clip(rho_i, 1 - eps, 1 + eps)
 *   A_old(a)  = log q(a) - log p_old(a)     (rollout-time advantage)
 *   A_theta(a) = log q(a) - log p_theta(a)  (recomputed under the current student)
 *   noclip:  L = -(1/m) sum_i rho_i sg(A_i)
 *   clip:    L = -(1/m) sum_i min(rho_i sg(A_i), rho_bar_i sg(A_i))
 * With A held fixed, d rho_i / d z_j = rho_i (1[j = a_i] - p_j).  Where the
 * min selects the clipped term and the clip is active, that term does not
 * depend on z, so the sample contributes nothing; where it selects the
 * unclipped term (ties, i.e. rho inside the clip range, count as unclipped:
 * there both terms are the same function of z) it contributes
 * -(1/m) A_i rho_i (1[j = a_i] - p_j).
 */
static void mc_surrogate(int theta_adv, int clip, const double* z, int64_t V, double L,
                         const int32_t* ids, const double* tau, const double* beta, int M,
                         double eps, double gamma, double* loss, double* grad) {
  double total = 0.0; /* sum_i of the surrogate terms */
  double c = 0.0;     /* (1/m) sum_i A_i rho_i over samples whose unclipped term is selected */
  for (int i = 0; i < M; ++i) {
    const double logp = z[ids[i]] - L;
    const double A = theta_adv ? tau[i] - logp : tau[i] - beta[i];
    const double rho = exp(logp - beta[i]);
    const double rho_bar = fmin(fmax(rho, 1.0 - eps), 1.0 + eps);
    const double unclipped = rho * A, clipped = rho_bar * A;
    if (!clip || unclipped <= clipped) {
      total += unclipped;
      c += A * rho;
    } else {
      total += clipped;
    }
  }
  *loss = -total / (double)M;
  c /= (double)M;
  if (!grad) return;
  for (int64_t j = 0; j < V; ++j) grad[j] = gamma * c * exp(z[j] - L);
  for (int i = 0; i < M; ++i) {
    const double logp = z[ids[i]] - L;
    const double A = theta_adv ? tau[i] - logp : tau[i] - beta[i];
    const double rho = exp(logp - beta[i]);
    const double rho_bar = fmin(fmax(rho, 1.0 - eps), 1.0 + eps);
    if (!clip || rho * A <= rho_bar * A) grad[ids[i]] -= gamma * A * rho / (double)M;
  }
}

/*
 * MC without importance sampling, the ablation of App. F: the behaviour
 * samples are used as if they had been drawn from p_theta, i.e. the
 * on-policy estimator of App. A.2, -(1/m) sum_i A_theta(a_i) grad log p_theta(a_i),
 * applied to p_old samples.  Its surrogate is
 *   L = -(1/m) sum_i sg(A_theta(a_i)) log p_theta(a_i),
 * with gradient -(1/m) sum_i A_i (1[j = a_i] - p_j).
 */
static void mc_no_is(const double* z, int64_t V, double L, const int32_t* ids, const double* tau,
                     int M, double gamma, double* loss, double* grad) {
  double total = 0.0, c = 0.0;
  for (int i = 0; i < M; ++i) {
    const double logp = z[ids[i]] - L;
    const double A = tau[i] - logp;
    total += A * logp;
    c += A;
  }
  *loss = -total / (double)M;
  c /= (double)M;
  if (!grad) return;
  for (int64_t j = 0; j < V; ++j) grad[j] = gamma * c * exp(z[j] - L);
  for (int i = 0; i < M; ++i) {
    const double A = tau[i] - (z[ids[i]] - L);
    grad[ids[i]] -= gamma * A / (double)M;
  }
}

/*
 * Dense full-vocabulary KL (Sec. 3):
 *   D_F = sum_a q (log q - log p_theta),   dD_F/dz_j = p_j - q_j;
 *   D_R = sum_a p_theta (log p_theta - log q),
 *   dD_R/dz_j = p_j ((log p_j - log q_j) - D_R)   (eq. reverse-kl-gradient
 *   pushed through the softmax Jacobian).
 * A term whose weight is zero (q_j for D_F, p_j for D_R) is zero, by the
 * convention 0 log(0/x) = 0 of the KL divergence: an action that both
 * distributions give logit -inf drops out, as if absent from the vocabulary.
 */
static void dense_kl(int reverse, const double* z, const double* y, int64_t V, double L,
                     double gamma, double* loss, double* grad) {
  const double Ly = log_partition(y, V);
  double kl = 0.0;
  for (int64_t j = 0; j < V; ++j) {
    const double logp = z[j] - L, logq = y[j] - Ly;
    const double w = reverse ? exp(logp) : exp(logq);
    if (w != 0.0) kl += reverse ? w * (logp - logq) : w * (logq - logp);
  }
  *loss = kl;
  if (!grad) return;
  for (int64_t j = 0; j < V; ++j) {
    const double logp = z[j] - L, logq = y[j] - Ly;
    const double p = exp(logp), q = exp(logq);
    if (reverse)
      grad[j] = p != 0.0 ? gamma * p * ((logp - logq) - kl) : 0.0;
    else
      grad[j] = gamma * (p - q);
  }
}

int oracle_row(int est, const double* z, const double* y, int64_t V, const int32_t* ids,
               const double* tau, const double* beta, int K, double gamma, double eps, int valid,
               double* loss, double* grad, double* lse, double* gathered) {
  const int dense = est == ORACLE_FKL_DENSE || est == ORACLE_RKL_DENSE;
  const int mc = est == ORACLE_RKL_MC || est == ORACLE_RKL_MC1 ||
                 (est >= ORACLE_RKL_MC_CLIP && est <= ORACLE_RKL_MC_NOIS);
  const int clip = est == ORACLE_RKL_MC_CLIP || est == ORACLE_RKL_MC_OLD_CLIP;
  if (!z || !loss || V < 1 || est < ORACLE_FKL_TOPK || est > ORACLE_RKL_TOPK_TRUNC) return -1;
  if (dense && !y) return -1;
  if (!dense && (K < 1 || !ids || !tau)) return -1;
  if (mc && est != ORACLE_RKL_MC_NOIS && !beta) return -1;
  if (clip && !(eps > 0.0 && isfinite(eps))) return -1;
  if (est == ORACLE_RKL_MC1 && K != 1) return -1;
  if (!dense)
    for (int i = 0; i < K; ++i)
      if (ids[i] < 0 || ids[i] >= V) return -1;

  if (!valid) { /* padded token: contributes nothing */
    *loss = 0.0;
    if (grad) memset(grad, 0, sizeof(double) * (size_t)V);
    if (lse) *lse = 0.0;
    if (gathered && !dense) memset(gathered, 0, sizeof(double) * (size_t)K);
    return 0;
  }
  const double L = log_partition(z, V);
  if (lse) *lse = L;
  if (gathered && !dense)
    for (int i = 0; i < K; ++i) gathered[i] = z[ids[i]];
  switch (est) {
    case ORACLE_FKL_TOPK: topk_kl(0, z, V, L, ids, tau, K, gamma, loss, grad); break;
    case ORACLE_RKL_TOPK: topk_kl(1, z, V, L, ids, tau, K, gamma, loss, grad); break;
    case ORACLE_RKL_MC1:
    case ORACLE_RKL_MC: mc_rkl(z, V, L, ids, tau, beta, K, gamma, loss, grad); break;
    case ORACLE_FKL_DENSE: dense_kl(0, z, y, V, L, gamma, loss, grad); break;
    case ORACLE_RKL_DENSE: dense_kl(1, z, y, V, L, gamma, loss, grad); break;
    case ORACLE_RKL_MC_CLIP:
      mc_surrogate(1, 1, z, V, L, ids, tau, beta, K, eps, gamma, loss, grad);
      break;
    case ORACLE_RKL_MC_OLD:
      mc_surrogate(0, 0, z, V, L, ids, tau, beta, K, eps, gamma, loss, grad);
      break;
    case ORACLE_RKL_MC_OLD_CLIP:
      mc_surrogate(0, 1, z, V, L, ids, tau, beta, K, eps, gamma, loss, grad);
      break;
    case ORACLE_RKL_MC_NOIS: mc_no_is(z, V, L, ids, tau, K, gamma, loss, grad); break;
    case ORACLE_FKL_TOPK_TRUNC: topk_truncated(0, z, V, L, ids, tau, K, gamma, loss, grad); break;
    case ORACLE_RKL_TOPK_TRUNC: topk_truncated(1, z, V, L, ids, tau, K, gamma, loss, grad); break;
  }
  return 0;
}

/*
 * Support coverage: the restricted normalisers of App. A.1 on the cached
 * support S = {a_i},
 *   Z_p^S = sum_{u in S} p_theta(u|s),     Z_q^S = sum_{u in S} q(u|s),
 * the share of the student's and of the teacher's mass that S holds.  A
 * stale support (Sec. 6, sparse top-k under rollout reuse) shows up as a
 * student coverage that falls away from the teacher's.  q at a cached action
 * is the cached full-vocabulary teacher probability exp(tau_i).  Each cached
 * entry counts once (the support's ids are distinct by precondition).
 */
int oracle_support_coverage(const double* z, int64_t V, const int32_t* ids, const double* tau,
                            int K, double* zp, double* zq) {
  if (!z || !ids || !tau || !zp || !zq || V < 1 || K < 1) return -1;
  for (int i = 0; i < K; ++i)
    if (ids[i] < 0 || ids[i] >= V) return -1;
  const double L = log_partition(z, V);
  double sp = 0.0, sq = 0.0;
  for (int i = 0; i < K; ++i) {
    sp += exp(z[ids[i]] - L);
    sq += exp(tau[i]);
  }
  *zp = sp;
  *zq = sq;
  return 0;
}

/* Exact widening of one stored logit to double. */
static double widen(int dtype, const void* base, int64_t off) {
  if (dtype == ORACLE_BF16) {
    const uint32_t bits = (uint32_t)((const uint16_t*)base)[off] << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
  }
  return (double)((const float*)base)[off];
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

int oracle_rows(int est, int dtype, const void* logits, const void* teacher_logits, int64_t n_rows,
                int64_t V, int64_t ld, const int32_t* ids, const float* tau, const float* beta,
                int K, const uint8_t* mask, double gamma, double eps, double* loss, double* grad,
                double* lse, double* gathered, int nthreads) {
  const int dense = est == ORACLE_FKL_DENSE || est == ORACLE_RKL_DENSE;
  if (!logits || !loss || n_rows < 0 || V < 1 || ld < V) return -1;
  if (dtype != ORACLE_F32 && dtype != ORACLE_BF16) return -1;
  if (dense && !teacher_logits) return -1;
  int err = 0;
  if (nthreads <= 0) nthreads = oracle_max_threads();
#ifdef _OPENMP
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)V);
    double* y = dense ? (double*)malloc(sizeof(double) * (size_t)V) : NULL;
    double* t = (double*)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
    double* b = (double*)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
    if (!z || (dense && !y) || !t || !b) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      err = -2;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t r = 0; r < n_rows; ++r) {
        for (int64_t j = 0; j < V; ++j) z[j] = widen(dtype, logits, r * ld + j);
        if (dense)
          for (int64_t j = 0; j < V; ++j) y[j] = widen(dtype, teacher_logits, r * ld + j);
        for (int i = 0; i < K && !dense; ++i) {
          t[i] = (double)tau[r * K + i];
          b[i] = beta ? (double)beta[r * K + i] : 0.0;
        }
        const int rc = oracle_row(est, z, y, V, dense ? NULL : ids + r * K, t, beta ? b : NULL,
                                  K, gamma, eps, mask ? mask[r] != 0 : 1, loss + r,
                                  grad ? grad + r * V : NULL, lse ? lse + r : NULL,
                                  gathered && !dense ? gathered + r * K : NULL);
        if (rc) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
          err = rc;
        }
      }
    }
    free(z);
    free(y);
    free(t);
    free(b);
  }
  return err;
}

/* Support coverage of stored rows: cov[2 r] = Z_p^S, cov[2 r + 1] = Z_q^S
 * (0 and 0 for a masked row). */
int oracle_coverage_rows(int dtype, const void* logits, int64_t n_rows, int64_t V, int64_t ld,
                         const int32_t* ids, const float* tau, int K, const uint8_t* mask,
                         double* cov, int nthreads) {
  if (!logits || !ids || !tau || !cov || n_rows < 0 || V < 1 || ld < V || K < 1) return -1;
  if (dtype != ORACLE_F32 && dtype != ORACLE_BF16) return -1;
  int err = 0;
  if (nthreads <= 0) nthreads = oracle_max_threads();
#ifdef _OPENMP
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)V);
    double* t = (double*)malloc(sizeof(double) * (size_t)K);
    if (!z || !t) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      err = -2;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t r = 0; r < n_rows; ++r) {
        cov[2 * r] = cov[2 * r + 1] = 0.0;
        if (mask && mask[r] == 0) continue;
        for (int64_t j = 0; j < V; ++j) z[j] = widen(dtype, logits, r * ld + j);
        for (int i = 0; i < K; ++i) t[i] = (double)tau[r * K + i];
        if (oracle_support_coverage(z, V, ids + r * K, t, K, cov + 2 * r, cov + 2 * r + 1)) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
          err = -1;
        }
      }
    }
    free(z);
    free(t);
  }
  return err;
}

/* ------------------------------------------------------------------------
 * Building the cache (Sec. 4.1, Stage 1 "Student rollout" and Stage 2
 * "Teacher scoring").  Rollout draws actions from the stale student p_old at
 * temperature 1 with no top-p or top-k truncation (App. B, Table 3) and
 * stores their rollout-time log-probs; a top-k support is the k most probable
 * actions (S_old = TopK(p_old, k), Sec. 5, "Sparse top-k"); teacher scoring
 * evaluates log q on the cached actions.
 * ------------------------------------------------------------------------ */

/* Cumulative distribution of softmax(z) in index order:
 * F[j] = sum_{l <= j} exp(z_l - L), summed left to right. */
int oracle_cdf(const double* z, int64_t V, double* F) {
  if (!z || !F || V < 1) return -1;
  const double L = log_partition(z, V);
  /* The running sum is kept in long double (64-bit significand): summed in
   * double, its rounding error grows to about V 2^-53 of the total, which at
   * V = 151,936 exceeds the error of a device CDF evaluated in double. */
  long double acc = 0.0L;
  for (int64_t j = 0; j < V; ++j) {
    acc += (long double)exp(z[j] - L);
    F[j] = (double)acc;
  }
  return 0;
}

/*
 * M iid draws from softmax(z) by inversion, one per uniform u_i in [0, 1):
 * a_i is the first index whose cumulative probability exceeds u_i.  Should
 * rounding leave u_i at or above the last cumulative value, a_i is the last
 * index of nonzero probability.  logp_i = log softmax(z)[a_i], the rollout-time
 * log-probability the cache stores.  A uniform outside [0, 1) (or NaN), or a
 * row whose softmax is undefined (a NaN or +inf logit, or every logit -inf),
 * gives a_i = -1 and logp_i = NaN.
 */
int oracle_sample_row(const double* z, int64_t V, const float* u, int M, int32_t* ids,
                      double* logp, double* lse) {
  if (!z || !u || !ids || V < 1 || M < 1) return -1;
  const double L = log_partition(z, V);
  if (lse) *lse = L;
  const int defined = isfinite(L);
  double* F = defined ? (double*)malloc(sizeof(double) * (size_t)V) : NULL;
  if (defined && !F) return -2;
  int64_t last = -1; /* last index of nonzero probability */
  if (defined) {
    oracle_cdf(z, V, F);
    for (int64_t j = V - 1; j >= 0 && last < 0; --j)
      if (exp(z[j] - L) > 0.0) last = j;
  }
  for (int i = 0; i < M; ++i) {
    const double ui = (double)u[i];
    int64_t a = -1;
    if (defined && ui >= 0.0 && ui < 1.0) {
      for (int64_t j = 0; j < V; ++j)
        if (F[j] > ui) {
          a = j;
          break;
        }
      if (a < 0) a = last;
    }
    ids[i] = (int32_t)a;
    if (logp) logp[i] = a >= 0 ? z[a] - L : NAN;
  }
  free(F);
  return 0;
}

/* Sort key of one stored logit: the IEEE-754 total order of its bits, with
 * -0 taken as +0 (so equal values tie); bf16 is widened first.  Larger key =
 * larger value; +NaN sorts above +inf and -NaN below -inf. */
static uint32_t order_key(int dtype, const void* base, int64_t off) {
  uint32_t bits;
  if (dtype == ORACLE_BF16)
    bits = (uint32_t)((const uint16_t*)base)[off] << 16;
  else
    memcpy(&bits, (const float*)base + off, 4);
  if (bits == 0x80000000u) bits = 0u;
  return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}

typedef struct {
  uint32_t key;
  int32_t j;
} ranked;

/* Descending value, then ascending index. */
static int rank_cmp(const void* pa, const void* pb) {
  const ranked* a = (const ranked*)pa;
  const ranked* b = (const ranked*)pb;
  if (a->key != b->key) return a->key > b->key ? -1 : 1;
  return a->j < b->j ? -1 : (a->j > b->j ? 1 : 0);
}

/*
 * The k largest logits of one stored row (raw fp32 or bf16 bits), in
 * descending order, equal values by ascending index: TopK(softmax(z), k),
 * since softmax is monotone.  logp_i = log softmax(z)[idx_i].
 */
int oracle_topk_row(int dtype, const void* row, int64_t V, int k, int32_t* idx, double* logp,
                    double* lse) {
  if (!row || !idx || V < 1 || k < 1 || k > V) return -1;
  ranked* r = (ranked*)malloc(sizeof(ranked) * (size_t)V);
  double* z = (double*)malloc(sizeof(double) * (size_t)V);
  if (!r || !z) {
    free(r);
    free(z);
    return -2;
  }
  for (int64_t j = 0; j < V; ++j) {
    r[j].key = order_key(dtype, row, j);
    r[j].j = (int32_t)j;
    z[j] = widen(dtype, row, j);
  }
  qsort(r, (size_t)V, sizeof(ranked), rank_cmp);
  const double L = log_partition(z, V);
  if (lse) *lse = L;
  for (int i = 0; i < k; ++i) {
    idx[i] = r[i].j;
    if (logp) logp[i] = z[r[i].j] - L;
  }
  free(r);
  free(z);
  return 0;
}

/* Full-vocabulary log-probabilities log softmax(z)[a_i] at given actions
 * (teacher scoring of a cache, or rollout log-probs of a support); an id
 * outside [0, V) gives NaN. */
int oracle_score_row(const double* z, int64_t V, const int32_t* ids, int K, double* logp,
                     double* lse) {
  if (!z || !ids || !logp || V < 1 || K < 1) return -1;
  const double L = log_partition(z, V);
  if (lse) *lse = L;
  for (int i = 0; i < K; ++i) logp[i] = (ids[i] >= 0 && ids[i] < V) ? z[ids[i]] - L : NAN;
  return 0;
}

/*
 * Batch drivers over stored rows ([n_rows, ld], fp32 or bf16 bits), `nthreads`
 * threads (0 = all).  A masked row (mask[r] == 0) gets ids/idx 0, logp 0 and
 * lse 0 and is not read.
 *   op 0  sampling:  aux_in = uniforms [n_rows, K] float; ids [n_rows, K] out
 *   op 1  top-k:     ids [n_rows, K] out (K = k)
 *   op 2  scoring:   ids [n_rows, K] in
 * logp [n_rows, K] and lse [n_rows] are nullable outputs.
 */
int oracle_cache_rows(int op, int dtype, const void* logits, int64_t n_rows, int64_t V, int64_t ld,
                      int K, const float* uniforms, const uint8_t* mask, int32_t* ids,
                      double* logp, double* lse, int nthreads) {
  if (!logits || !ids || n_rows < 0 || V < 1 || ld < V || K < 1) return -1;
  if (dtype != ORACLE_F32 && dtype != ORACLE_BF16) return -1;
  if (op < 0 || op > 2 || (op == 0 && !uniforms) || (op == 1 && K > V)) return -1;
  int err = 0;
  if (nthreads <= 0) nthreads = oracle_max_threads();
#ifdef _OPENMP
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc(sizeof(double) * (size_t)V);
    double* lp = (double*)malloc(sizeof(double) * (size_t)K);
    if (!z || !lp) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      err = -2;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t r = 0; r < n_rows; ++r) {
        int32_t* rid = ids + r * K;
        double L = 0.0;
        int rc = 0;
        if (mask && mask[r] == 0) {
          for (int i = 0; i < K; ++i) {
            if (op != 2) rid[i] = 0;
            lp[i] = 0.0;
          }
        } else {
          if (op != 1)
            for (int64_t j = 0; j < V; ++j) z[j] = widen(dtype, logits, r * ld + j);
          if (op == 0)
            rc = oracle_sample_row(z, V, uniforms + r * K, K, rid, lp, &L);
          else if (op == 1)
            rc = oracle_topk_row(dtype, (const char*)logits +
                                            (size_t)(r * ld) * (dtype == ORACLE_BF16 ? 2 : 4),
                                 V, K, rid, lp, &L);
          else
            rc = oracle_score_row(z, V, rid, K, lp, &L);
        }
        if (logp)
          for (int i = 0; i < K; ++i) logp[r * K + i] = lp[i];
        if (lse) lse[r] = L;
        if (rc) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
          err = rc;
        }
      }
    }
    free(z);
    free(lp);
  }
  return err;
}

/* ------------------------------------------------------------------------
 * Diagnostics of the Monte-Carlo estimator (Sec. 5.2, Fig. 5: the p99 tail
 * of the importance ratio rho_theta; App. E: variance of the m-sample
 * estimator at a fixed prefix and after averaging over the tokens of a
 * sequence).  Inputs are what the loss call returns or reads per token t:
 * L_t = log sum_j exp(z_j), the student logits z_{t,i} at the M cached
 * samples, and the cached tau_{t,i} = log q, beta_{t,i} = log p_old.
 *   log p_theta = z - L,  A = tau - log p_theta,  rho = exp(log p_theta - beta),
 *   X_{t,i} = -rho_{t,i} A_{t,i}   (one-sample estimate; the loss is their mean)
 * Per valid token: mean_t = (1/M) sum_i X, var_t = unbiased sample variance of
 * X over i (M >= 2, else NaN), rhomax_t = max_i rho.
 * Over all valid entries: the q-quantile of rho by nearest rank (the r-th
 * smallest, r = ceil(q n), at least 1), and the fraction with |rho - 1| > eps.
 * Variance ratios for group sizes m (M a multiple of m, G = M / m >= 2):
 * group g holds samples [g m, g m + m); Y_{t,g} its mean.
 *   local:  R_m = sum_t var_g(Y_{t,g}) / sum_t var_t
 *   seq:    tokens [s T, s T + T) form sequence s; S_{s,g} = mean over its
 *           valid tokens of Y_{t,g}; R_m = sum_s var_g(S_{s,g}) / sum_s
 *           var_i(S1_{s,i}), S1 the same with single samples (m = 1).
 * var_g is the unbiased variance over the G groups.  Replicate groups of the
 * iid draws stand in for repeated sampling at the fixed prefix (or path).
 * ------------------------------------------------------------------------ */

static double unbiased_var(const double* x, int n) {
  double mean = 0.0;
  for (int i = 0; i < n; ++i) mean += x[i];
  mean /= n;
  double ss = 0.0;
  for (int i = 0; i < n; ++i) ss += (x[i] - mean) * (x[i] - mean);
  return ss / (n - 1);
}

static int cmp_double(const void* pa, const void* pb) {
  const double a = *(const double*)pa, b = *(const double*)pb;
  /* NaN after every number */
  if (isnan(a) || isnan(b)) return isnan(a) - isnan(b);
  return a < b ? -1 : (a > b ? 1 : 0);
}

int oracle_mc_diagnostics(const double* lse, const double* gathered, const float* tau,
                          const float* beta, int64_t N, int M, const uint8_t* mask, double q,
                          double eps, const int* group_sizes, int n_groups, int64_t seq_len,
                          double* row_mean, double* row_var, double* row_rhomax,
                          double* rho_quantile, double* clip_frac, double* ratio_local,
                          double* ratio_seq) {
  if (!lse || !gathered || !tau || !beta || N < 0 || M < 1 || !(q > 0.0 && q <= 1.0)) return -1;
  if (n_groups < 0 || (n_groups > 0 && !group_sizes) || seq_len < 0) return -1;
  for (int k = 0; k < n_groups; ++k)
    if (group_sizes[k] < 1 || M % group_sizes[k] != 0 || M / group_sizes[k] < 2) return -1;
  double* X = (double*)malloc(sizeof(double) * (size_t)(N * M + 1));
  double* rho = (double*)malloc(sizeof(double) * (size_t)(N * M + 1));
  double* Y = (double*)malloc(sizeof(double) * (size_t)(M + 1));
  if (!X || !rho || !Y) {
    free(X);
    free(rho);
    free(Y);
    return -2;
  }
  int64_t n = 0, clipped = 0;
  double sum_var = 0.0;
  for (int64_t t = 0; t < N; ++t) {
    const int valid = mask ? mask[t] != 0 : 1;
    double mean = 0.0, mx = NAN; /* the largest ratio, NaN ratios ignored */
    for (int i = 0; i < M && valid; ++i) {
      const double lp = gathered[t * M + i] - lse[t];
      const double r = exp(lp - (double)beta[t * M + i]);
      const double A = (double)tau[t * M + i] - lp;
      X[t * M + i] = -r * A;
      rho[n++] = r;
      if (fabs(r - 1.0) > eps) ++clipped;
      mean += X[t * M + i];
      if (!isnan(r) && (isnan(mx) || r > mx)) mx = r;
    }
    const double var = (valid && M >= 2) ? unbiased_var(X + t * M, M) : NAN;
    if (valid && M >= 2) sum_var += var;
    if (row_mean) row_mean[t] = valid ? mean / M : 0.0;
    if (row_var) row_var[t] = valid ? var : 0.0;
    if (row_rhomax) row_rhomax[t] = valid ? mx : 0.0;
  }
  if (rho_quantile) {
    if (n == 0) {
      *rho_quantile = NAN;
    } else {
      qsort(rho, (size_t)n, sizeof(double), cmp_double);
      int64_t r = (int64_t)ceil(q * (double)n);
      if (r < 1) r = 1;
      *rho_quantile = rho[r - 1];
    }
  }
  if (clip_frac) *clip_frac = n ? (double)clipped / (double)n : NAN;
  for (int k = 0; k < n_groups; ++k) {
    const int m = group_sizes[k], G = M / m;
    if (ratio_local) {
      double sum_g = 0.0;
      for (int64_t t = 0; t < N; ++t) {
        if (mask && mask[t] == 0) continue;
        for (int g = 0; g < G; ++g) {
          double y = 0.0;
          for (int i = g * m; i < g * m + m; ++i) y += X[t * M + i];
          Y[g] = y / m;
        }
        sum_g += unbiased_var(Y, G);
      }
      ratio_local[k] = sum_g / sum_var;
    }
    if (ratio_seq && seq_len > 0) {
      double num = 0.0, den = 0.0;
      double* S = (double*)calloc((size_t)M, sizeof(double));
      double* S1 = (double*)calloc((size_t)M, sizeof(double));
      for (int64_t s0 = 0; s0 < N; s0 += seq_len) {
        const int64_t s1 = s0 + seq_len < N ? s0 + seq_len : N;
        int64_t nv = 0;
        for (int i = 0; i < M; ++i) S[i] = S1[i] = 0.0;
        for (int64_t t = s0; t < s1; ++t) {
          if (mask && mask[t] == 0) continue;
          ++nv;
          for (int i = 0; i < M; ++i) S1[i] += X[t * M + i];
          for (int g = 0; g < G; ++g) {
            double y = 0.0;
            for (int i = g * m; i < g * m + m; ++i) y += X[t * M + i];
            S[g] += y / m;
          }
        }
        if (nv == 0) continue;
        for (int i = 0; i < M; ++i) S1[i] /= (double)nv;
        for (int g = 0; g < G; ++g) S[g] /= (double)nv;
        num += unbiased_var(S, G);
        den += unbiased_var(S1, M);
      }
      ratio_seq[k] = num / den;
      free(S);
      free(S1);
    }
  }
  free(X);
  free(rho);
  free(Y);
  return 0;
}
