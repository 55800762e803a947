/* Seeded synthetic inputs for the learner-time OPD loss (rollout and teacher
 * scoring stand-ins).  Host-only; see opd_synth.c for the recipe. */
#ifndef OPD_SYNTH_H
#define OPD_SYNTH_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

enum { SYNTH_F32 = 0, SYNTH_BF16 = 1 };

typedef struct synth_cfg {
  uint64_t seed;
  int64_t V;
  int32_t dtype;          /* storage dtype of student and teacher logits */
  int32_t pad_;
  double sigma_student;   /* z = sigma_student * N(0,1) */
  double boost_prob;      /* per-entry probability of adding boost_value */
  double boost_value;
  double sigma_teacher;   /* y = z + sigma_teacher * N(0,1) */
  double sigma_behaviour; /* b = z + sigma_behaviour * N(0,1) */
} synth_cfg;

/* Rows [r0, r1): student logits (row stride ld, dtype), dense teacher logits,
 * teacher top-k cache [rows, k], Monte-Carlo cache [rows, M].  Every output is
 * nullable; returns 0 or a negative code. */
int synth_rows(const synth_cfg* c, int64_t r0, int64_t r1, void* logits, int64_t ld,
               void* teacher_logits, int k, int32_t* topk_idx, float* topk_tau, int M,
               int32_t* mc_ids, float* mc_tau, float* mc_beta, int nthreads);

/* Behaviour logits b (double, unrounded) and teacher logits y of one row. */
int synth_behaviour_row(const synth_cfg* c, int64_t row, double* b_out);
int synth_teacher_row(const synth_cfg* c, int64_t row, double* y_out);

/* Right-padded ragged mask: rollout r keeps its first len_r tokens,
 * len_r uniform on {len_lo, ..., len_hi}. */
int synth_ragged_mask(uint64_t seed, int64_t n_rollouts, int64_t rollout_len, int64_t len_lo,
                      int64_t len_hi, uint8_t* mask, int32_t* lengths);

/* n uniforms on [0,1) from (seed, stream, row); for tests that need their own draws. */
int synth_uniforms(uint64_t seed, uint64_t stream, int64_t row, int64_t n, double* out);

#ifdef __cplusplus
}
#endif
#endif
