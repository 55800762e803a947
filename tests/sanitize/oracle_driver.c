/* Calls every entry point of the oracle on small inputs, including the edge
 * cases the tests use (padded strides, masked rows, repeated and
 * out-of-range ids, NaN and infinite logits, extreme uniforms), so that a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer checks the
 * oracle's memory accesses and arithmetic.  Test infrastructure only: it
 * prints a line per group of calls and returns 0 unless an output that must
 * be finite is not.  With the argument plant-overflow it instead reads past
 * a buffer of its own, to show that the sanitizer build catches it. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/opd_oracle.h"

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static double unif(void) { /* xorshift64*, in [0, 1) */
  g_state ^= g_state >> 12; g_state ^= g_state << 25; g_state ^= g_state >> 27;
  return (double)((g_state * 2685821657736338717ull) >> 11) * (1.0 / 9007199254740992.0);
}
static double normal(void) {
  const double u = unif() + 1e-300, v = unif();
  return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}
static uint16_t to_bf16(float f) {
  uint32_t u; memcpy(&u, &f, 4);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

int main(int argc, char** argv) {
  if (argc > 1 && strcmp(argv[1], "plant-overflow") == 0) {
    /* a deliberate read one element past a heap buffer: the sanitizer
     * build must stop here (the test checks that it does) */
    volatile double* b = malloc(sizeof(double) * 4);
    for (int i = 0; i < 4; ++i) b[i] = i;
    const double past = b[4];
    free((void*)b);
    printf("read %g\n", past);
    return 0;
  }
  const int N = 5, Ks[3] = {1, 16, 64}, Vs[2] = {1000, 3001};
  int failures = 0;
  for (int dt = 0; dt < 2; ++dt)
    for (int vi = 0; vi < 2; ++vi) {
      const int64_t V = Vs[vi], ld = V + 8;
      const size_t esz = dt == ORACLE_BF16 ? 2 : 4;
      unsigned char* z = calloc((size_t)(N * ld), esz);
      unsigned char* y = calloc((size_t)(N * ld), esz);
      for (int r = 0; r < N; ++r)
        for (int64_t j = 0; j < V; ++j) {
          float a = (float)(2.0 * normal()), b = (float)(a + normal());
          if (r == 3 && j % 97 == 0) a = -INFINITY;      /* -inf entries */
          if (r == 3 && j % 89 == 0) b = -INFINITY;
          if (r == 4 && j == 5) a = NAN;                 /* a NaN row */
          if (dt == ORACLE_BF16) {
            ((uint16_t*)z)[r * ld + j] = to_bf16(a);
            ((uint16_t*)y)[r * ld + j] = to_bf16(b);
          } else {
            ((float*)z)[r * ld + j] = a;
            ((float*)y)[r * ld + j] = b;
          }
        }
      uint8_t mask[5] = {1, 0, 1, 1, 1};
      for (int ki = 0; ki < 3; ++ki) {
        const int K = Ks[ki];
        int32_t* ids = malloc(sizeof(int32_t) * N * K);
        float* tau = malloc(sizeof(float) * N * K);
        float* beta = malloc(sizeof(float) * N * K);
        for (int r = 0; r < N; ++r)
          for (int i = 0; i < K; ++i) {
            ids[r * K + i] = (int32_t)((r * 131 + i * 37) % V);
            tau[r * K + i] = (float)(-3.0 - unif());
            beta[r * K + i] = (float)(-3.0 - unif());
          }
        if (K > 1) ids[2 * K + 1] = ids[2 * K];  /* a repeat (legal for MC) */
        ids[4 * K + K - 1] = (int32_t)V;          /* out of range: the row's error */
        double* loss = malloc(sizeof(double) * N);
        double* grad = malloc(sizeof(double) * N * V);
        double* lse = malloc(sizeof(double) * N);
        double* gat = malloc(sizeof(double) * N * K);
        for (int est = 0; est <= 11; ++est) {
          const int dense = est == ORACLE_FKL_DENSE || est == ORACLE_RKL_DENSE;
          oracle_rows(est, dt, z, dense ? y : NULL, N, V, ld, dense ? NULL : ids,
                      dense ? NULL : tau, beta, K, mask, 0.75, 0.2, loss, grad, lse,
                      dense ? NULL : gat, 2);
          /* a valid row's loss is finite except where the row holds a NaN or
           * an id out of range (row 4), or -inf entries meet the estimator */
          if (!isfinite(loss[0])) ++failures;
        }
        double cov[10];
        oracle_coverage_rows(dt, z, N, V, ld, ids, tau, K, mask, cov, 2);
        /* the cache builders: draws at extreme uniforms, top-k, scoring */
        float* u = malloc(sizeof(float) * N * K);
        for (int i = 0; i < N * K; ++i) u[i] = (float)unif();
        u[0] = 0.0f;
        u[K - 1] = 0.99999994f;
        if (K > 2) { u[K + 1] = NAN; u[K + 2] = -0.25f; }
        int32_t* out_ids = malloc(sizeof(int32_t) * N * K);
        double* out_lp = malloc(sizeof(double) * N * K);
        oracle_cache_rows(0, dt, z, N, V, ld, K, u, mask, out_ids, out_lp, lse, 2);
        oracle_cache_rows(1, dt, z, N, V, ld, K, NULL, mask, out_ids, out_lp, lse, 2);
        oracle_cache_rows(2, dt, z, N, V, ld, K, NULL, mask, ids, out_lp, lse, 2);
        /* diagnostics fed by the MC call's own outputs */
        oracle_rows(ORACLE_RKL_MC, dt, z, NULL, N, V, ld, ids, tau, beta, K, mask, 1.0, 0.2, loss,
                    NULL, lse, gat, 1);
        if (K >= 2) {
          const int groups[3] = {1, 2, 4};
          const int ng = K >= 8 ? 3 : 1;
          double rm[5], rv[5], rx[5], q, clip, rl[3], rs[3];
          oracle_mc_diagnostics(lse, gat, tau, beta, N, K, mask, 0.99, 0.2, groups + (K >= 8 ? 0 : 1),
                                ng, 3, rm, rv, rx, &q, &clip, rl, rs);
        }
        free(ids); free(tau); free(beta); free(loss); free(grad); free(lse); free(gat);
        free(u); free(out_ids); free(out_lp);
      }
      /* single rows in double, and the CDF */
      double* zd = malloc(sizeof(double) * V);
      double* F = malloc(sizeof(double) * V);
      for (int64_t j = 0; j < V; ++j) zd[j] = normal();
      oracle_cdf(zd, V, F);
      if (!(fabs(F[V - 1] - 1.0) < 1e-12)) ++failures;
      double zp, zq;
      const int32_t sid[3] = {0, 5, (int32_t)V - 1};
      const double stau[3] = {-1.0, -2.0, -3.0};
      oracle_support_coverage(zd, V, sid, stau, 3, &zp, &zq);
      free(zd); free(F); free(z); free(y);
      printf("dtype %d V %lld: done\n", dt, (long long)V);
    }
  printf("failures %d\n", failures);
  return failures ? 1 : 0;
}
