/*
 * Seeded, counter-based synthetic inputs for the learner-time OPD loss.
 *
 * The learner consumes what two earlier pipeline stages leave behind
 * (Sec. 4.1, "Stage 1: Student rollout" and "Stage 2: Teacher scoring"):
 * a row of student logits per generated token, plus a finite teacher-score
 * cache for that token.  This module plays those two stages on synthetic
 * data.  It draws
 *   - student logits  z = round(sigma_s * N(0,1) [+ boost with prob p]),
 *   - teacher logits  y = round(z + sigma_t * N(0,1)),
 *   - behaviour (stale-student) logits b = z + sigma_b * N(0,1), never stored,
 * and from them builds either the teacher top-k cache (ids of the k largest
 * y, with the teacher log-probs there) or the Monte-Carlo cache (M ids drawn
 * iid with replacement from softmax(b), with teacher and behaviour
 * log-probs there; App. E).  "round" is the storage dtype: fp32, or fp32
 * then bf16 with round-to-nearest-even at each step.
 *
 * It holds none of the learner's loss arithmetic and shares no code with the
 * oracle or with the GPU library; both sides read its outputs only.
 *
 * Random numbers.  SplitMix64 (Steele, Lea & Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014) is used as a counter-based
 * generator: the n-th output of a SplitMix64 sequence seeded with s is
 * mix64(s + (n + 1) * 0x9E3779B97F4A7C15), so any (stream, row, column)
 * draw is computed directly, and any row can be regenerated on its own.
 * Normals use the Box-Muller transform in double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#include "opd_synth.h"

#define GOLDEN_GAMMA 0x9E3779B97F4A7C15ULL

enum {
  STREAM_STUDENT = 1,
  STREAM_BOOST = 2,
  STREAM_TEACHER = 3,
  STREAM_BEHAVIOUR = 4,
  STREAM_SAMPLE = 5,
  STREAM_LENGTH = 6
};

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return mix64(seed ^ mix64(stream * GOLDEN_GAMMA + 0x2545F4914F6CDD1DULL));
}

/* n-th SplitMix64 output of the sequence seeded with key. */
static inline uint64_t draw(uint64_t key, uint64_t n) {
  return mix64(key + (n + 1) * GOLDEN_GAMMA);
}

/* counter for (row, col): rows get disjoint 2^32-wide blocks of the sequence */
static inline uint64_t ctr(int64_t row, int64_t col) {
  return ((uint64_t)row << 32) + (uint64_t)col;
}

/* uniform on [0, 1) with 53 random bits */
static inline double unif_co(uint64_t x) { return (double)(x >> 11) * 0x1.0p-53; }
/* uniform on (0, 1] with 53 random bits */
static inline double unif_oc(uint64_t x) { return (double)((x >> 11) + 1) * 0x1.0p-53; }

/* Standard normals of one row, columns [0, V): Box-Muller on the uniform
 * pair drawn at columns (2i, 2i+1); column 2i takes the cosine branch and
 * column 2i+1 the sine branch. */
static void normal_row(uint64_t key, int64_t row, int64_t V, double* out) {
  for (int64_t c0 = 0; c0 < V; c0 += 2) {
    const double u1 = unif_oc(draw(key, ctr(row, c0)));
    const double u2 = unif_co(draw(key, ctr(row, c0 + 1)));
    const double r = sqrt(-2.0 * log(u1));
    const double t = 6.283185307179586 * u2;
    out[c0] = r * cos(t);
    if (c0 + 1 < V) out[c0 + 1] = r * sin(t);
  }
}

static inline float f32_from_bits(uint32_t u) {
  float f;
  memcpy(&f, &u, 4);
  return f;
}
static inline uint32_t bits_from_f32(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

/* fp32 -> bf16, round to nearest, ties to even (finite inputs only). */
static inline uint16_t bf16_rne(float f) {
  const uint32_t u = bits_from_f32(f);
  const uint32_t lsb = (u >> 16) & 1u;
  return (uint16_t)((u + 0x7FFFu + lsb) >> 16);
}

/* Round a double to the storage dtype and return the stored value. */
static inline double round_to_dtype(double v, int dtype, uint16_t* bf_out, float* f_out) {
  const float f = (float)v;
  if (dtype == SYNTH_BF16) {
    const uint16_t h = bf16_rne(f);
    if (bf_out) *bf_out = h;
    return (double)f32_from_bits((uint32_t)h << 16);
  }
  if (f_out) *f_out = f;
  return (double)f;
}

static int check_cfg(const synth_cfg* c) {
  if (!c) return -1;
  if (c->V < 2 || c->V > ((int64_t)1 << 31) - 1) return -2;
  if (c->dtype != SYNTH_F32 && c->dtype != SYNTH_BF16) return -3;
  return 0;
}

/* Fill z[0..V) with the stored student logits of row `row`. */
static void student_row(const synth_cfg* c, int64_t row, double* z, void* out) {
  const uint64_t ks = stream_key(c->seed, STREAM_STUDENT);
  const uint64_t kb = stream_key(c->seed, STREAM_BOOST);
  const int64_t V = c->V;
  uint16_t* ob = (c->dtype == SYNTH_BF16) ? (uint16_t*)out : NULL;
  float* of = (c->dtype == SYNTH_F32) ? (float*)out : NULL;
  normal_row(ks, row, V, z);
  for (int64_t j = 0; j < V; ++j) {
    double v = c->sigma_student * z[j];
    if (c->boost_prob > 0.0 && unif_co(draw(kb, ctr(row, j))) < c->boost_prob) v += c->boost_value;
    z[j] = round_to_dtype(v, c->dtype, ob ? ob + j : NULL, of ? of + j : NULL);
  }
}

static void teacher_row(const synth_cfg* c, int64_t row, const double* z, double* y, void* out) {
  const uint64_t kt = stream_key(c->seed, STREAM_TEACHER);
  const int64_t V = c->V;
  uint16_t* ob = (c->dtype == SYNTH_BF16) ? (uint16_t*)out : NULL;
  float* of = (c->dtype == SYNTH_F32) ? (float*)out : NULL;
  normal_row(kt, row, V, y);
  for (int64_t j = 0; j < V; ++j) {
    const double v = z[j] + c->sigma_teacher * y[j];
    y[j] = round_to_dtype(v, c->dtype, ob ? ob + j : NULL, of ? of + j : NULL);
  }
}

static void behaviour_row(const synth_cfg* c, int64_t row, const double* z, double* b) {
  const uint64_t kb = stream_key(c->seed, STREAM_BEHAVIOUR);
  normal_row(kb, row, c->V, b);
  for (int64_t j = 0; j < c->V; ++j) b[j] = z[j] + c->sigma_behaviour * b[j];
}

/* log sum_j exp(x_j), two sweeps in double.  Used only to turn the synthetic
 * teacher and behaviour logits into the log-probabilities those stages would
 * have recorded. */
static double log_normaliser(const double* x, int64_t V) {
  double m = x[0];
  for (int64_t j = 1; j < V; ++j) m = x[j] > m ? x[j] : m;
  double s = 0.0;
  for (int64_t j = 0; j < V; ++j) s += exp(x[j] - m);
  return m + log(s);
}

/* "a ranks above b": larger value, ties broken by the lower index */
static inline int ranks_above(double va, int32_t ia, double vb, int32_t ib) {
  return va > vb || (va == vb && ia < ib);
}

/* Indices of the k largest y (lower index wins ties), in descending order. */
static void top_k(const double* y, int64_t V, int k, int32_t* idx) {
  /* min-heap on rank of the current k best: heap[0] is the weakest kept */
  int n = 0;
  for (int64_t j = 0; j < V; ++j) {
    const int32_t jj = (int32_t)j;
    if (n < k) {
      int p = n++;
      idx[p] = jj;
      while (p > 0) { /* sift up: weaker entries go to the root */
        const int q = (p - 1) / 2;
        if (ranks_above(y[idx[q]], idx[q], y[idx[p]], idx[p])) {
          const int32_t t = idx[q]; idx[q] = idx[p]; idx[p] = t; p = q;
        } else break;
      }
    } else if (ranks_above(y[j], jj, y[idx[0]], idx[0])) {
      idx[0] = jj;
      int p = 0;
      for (;;) { /* sift down */
        const int l = 2 * p + 1, r = l + 1;
        int w = p;
        if (l < n && ranks_above(y[idx[w]], idx[w], y[idx[l]], idx[l])) w = l;
        if (r < n && ranks_above(y[idx[w]], idx[w], y[idx[r]], idx[r])) w = r;
        if (w == p) break;
        const int32_t t = idx[w]; idx[w] = idx[p]; idx[p] = t; p = w;
      }
    }
  }
  /* heap -> descending order by repeated extraction of the weakest */
  for (int end = n - 1; end > 0; --end) {
    const int32_t t = idx[0]; idx[0] = idx[end]; idx[end] = t;
    int p = 0;
    for (;;) {
      const int l = 2 * p + 1, r = l + 1;
      int w = p;
      if (l < end && ranks_above(y[idx[w]], idx[w], y[idx[l]], idx[l])) w = l;
      if (r < end && ranks_above(y[idx[w]], idx[w], y[idx[r]], idx[r])) w = r;
      if (w == p) break;
      const int32_t s = idx[w]; idx[w] = idx[p]; idx[p] = s; p = w;
    }
  }
}

int synth_rows(const synth_cfg* c, int64_t r0, int64_t r1, void* logits, int64_t ld,
               void* teacher_logits, int k, int32_t* topk_idx, float* topk_tau, int M,
               int32_t* mc_ids, float* mc_tau, float* mc_beta, int nthreads) {
  const int rc = check_cfg(c);
  if (rc) return rc;
  if (r1 < r0 || r0 < 0) return -4;
  if ((logits || teacher_logits) && ld < c->V) return -5;
  const int want_topk = topk_idx != NULL || topk_tau != NULL;
  const int want_mc = mc_ids != NULL || mc_tau != NULL || mc_beta != NULL;
  if (want_topk && (k < 1 || k > c->V)) return -6;
  if (want_mc && M < 1) return -7;
  const int need_teacher = teacher_logits != NULL || want_topk || want_mc;
  const int64_t V = c->V;
  const size_t esz = c->dtype == SYNTH_BF16 ? 2 : 4;
  int failed = 0;
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads)
#endif
  {
    double* z = (double*)malloc(sizeof(double) * V);
    double* y = (double*)malloc(sizeof(double) * V);
    double* w = (double*)malloc(sizeof(double) * V);
    int32_t* sel = (int32_t*)malloc(sizeof(int32_t) * (k > 0 ? k : 1));
    double* cum = want_mc ? (double*)malloc(sizeof(double) * V) : NULL;
    if (!z || !y || !w || !sel || (want_mc && !cum)) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
      failed = 1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 4)
#endif
      for (int64_t r = r0; r < r1; ++r) {
        const int64_t lr = r - r0;
        void* lout = logits ? (char*)logits + (size_t)lr * ld * esz : NULL;
        student_row(c, r, z, lout);
        if (!need_teacher) continue;
        void* tout = teacher_logits ? (char*)teacher_logits + (size_t)lr * ld * esz : NULL;
        teacher_row(c, r, z, y, tout);
        const double lse_y = log_normaliser(y, V);
        if (want_topk) {
          top_k(y, V, k, sel);
          for (int i = 0; i < k; ++i) {
            if (topk_idx) topk_idx[lr * k + i] = sel[i];
            if (topk_tau) topk_tau[lr * k + i] = (float)(y[sel[i]] - lse_y);
          }
        }
        if (want_mc) {
          behaviour_row(c, r, z, w);
          const double lse_b = log_normaliser(w, V);
          /* w <- behaviour log-probs */
          for (int64_t j = 0; j < V; ++j) w[j] -= lse_b;
          const uint64_t ku = stream_key(c->seed, STREAM_SAMPLE);
          /* inverse CDF on the behaviour policy, iid with replacement */
          double acc = 0.0;
          for (int64_t j = 0; j < V; ++j) {
            acc += exp(w[j]);
            cum[j] = acc;
          }
          for (int i = 0; i < M; ++i) {
            const double target = unif_co(draw(ku, ctr(r, i))) * acc;
            int64_t lo = 0, hi = V - 1; /* first j with cum[j] > target */
            while (lo < hi) {
              const int64_t mid = lo + (hi - lo) / 2;
              if (cum[mid] > target) hi = mid; else lo = mid + 1;
            }
            if (mc_ids) mc_ids[lr * M + i] = (int32_t)lo;
            if (mc_tau) mc_tau[lr * M + i] = (float)(y[lo] - lse_y);
            if (mc_beta) mc_beta[lr * M + i] = (float)w[lo];
          }
        }
      }
    }
    free(z); free(y); free(w); free(sel); free(cum);
  }
  return failed ? -8 : 0;
}

int synth_behaviour_row(const synth_cfg* c, int64_t row, double* b_out) {
  const int rc = check_cfg(c);
  if (rc) return rc;
  double* z = (double*)malloc(sizeof(double) * c->V);
  if (!z) return -8;
  student_row(c, row, z, NULL);
  behaviour_row(c, row, z, b_out);
  free(z);
  return 0;
}

int synth_teacher_row(const synth_cfg* c, int64_t row, double* y_out) {
  const int rc = check_cfg(c);
  if (rc) return rc;
  double* z = (double*)malloc(sizeof(double) * c->V);
  if (!z) return -8;
  student_row(c, row, z, NULL);
  teacher_row(c, row, z, y_out, NULL);
  free(z);
  return 0;
}

int synth_ragged_mask(uint64_t seed, int64_t n_rollouts, int64_t rollout_len, int64_t len_lo,
                      int64_t len_hi, uint8_t* mask, int32_t* lengths) {
  if (n_rollouts < 0 || rollout_len < 1 || len_lo < 0 || len_hi < len_lo || len_hi > rollout_len)
    return -4;
  const uint64_t kl = stream_key(seed, STREAM_LENGTH);
  for (int64_t r = 0; r < n_rollouts; ++r) {
    const double u = unif_co(draw(kl, (uint64_t)r));
    const int64_t len = len_lo + (int64_t)(u * (double)(len_hi - len_lo + 1));
    if (lengths) lengths[r] = (int32_t)len;
    for (int64_t t = 0; t < rollout_len; ++t) mask[r * rollout_len + t] = (uint8_t)(t < len);
  }
  return 0;
}

int synth_uniforms(uint64_t seed, uint64_t stream, int64_t row, int64_t n, double* out) {
  const uint64_t key = stream_key(seed, stream);
  for (int64_t i = 0; i < n; ++i) out[i] = unif_co(draw(key, ctr(row, i)));
  return 0;
}
