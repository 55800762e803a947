// Internal interface between the C-ABI layer (opd_api.cpp) and the HIP
// kernels (opd_kernels.hip).  Not installed; the public interface is opd.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/opd.h"

namespace opd {

enum Est : int { FKL_TOPK = 0, RKL_TOPK = 1, RKL_MC1 = 2, RKL_MC = 3, FKL_DENSE = 4, RKL_DENSE = 5 };
// Estimators that run the RKL_MC kernels (a dense coefficient of p_theta plus
// spikes at the cached ids): the Monte-Carlo family and the truncated top-k KLs.
enum McVariant : int {
  MC_THETA = 0,
  MC_THETA_CLIP = 1,
  MC_OLD = 2,
  MC_OLD_CLIP = 3,
  MC_NO_IS = 4,
  TRUNC_FKL = 5,
  TRUNC_RKL = 6
};
enum Dt : int { F32 = 0, BF16 = 1 };

constexpr int kKMax = 256;
// Row-per-workgroup kernels: one 1024-lane workgroup per token row.
constexpr int kRowThreads = 1024;
// Every lane works on vectors of 4 consecutive elements.
constexpr int kElemsPerVec = 4;
// Resident variants keep the whole logit row in registers between the two
// sweeps: up to 76 VGPRs of packed row data per lane, i.e. 38 bf16 vectors
// (8 bytes each) or 19 fp32 vectors (16 bytes each); the small variants hold
// less than half of that for narrow rows.
constexpr int slots_large(int dt) { return dt == BF16 ? 38 : 19; }
constexpr int slots_small(int dt) { return dt == BF16 ? 16 : 8; }
// Split-vocabulary kernels: 256 lanes per (row, chunk) workgroup.
constexpr int kSplitThreads = 256;
// Pass-1 partial record per (row, chunk): m, s, m_y, s_y, t_f, t_r, pad, pad.
constexpr int kPartialFloats = 8;

// Everything a kernel needs for one call.  Plain pointers and sizes.
struct Args {
  const void* logits;
  const void* teacher;  // dense estimators only
  int64_t N, V, ld;
  int64_t nvec;         // 4-element vectors per row covering [0, V)
  int tail;             // valid elements in the last vector (== elements per vector if full)
  const int32_t* ids;   // [N, K]
  const float* tau;     // [N, K]
  const float* beta;    // [N, K] (MC only; NULL for MC_NO_IS)
  int K;
  int mc_variant;       // McVariant of the MC estimators
  float clip_eps;
  const uint8_t* mask;  // nullable
  float gamma;
  int skip_masked;
  float* loss;
  void* dlogits;
  float* lse_out;       // nullable
  float* gathered_out;  // nullable
  float* coverage_out;  // [N, 2] nullable: Z_p^S, Z_q^S (estimators with a support)
  float* ws;            // split path partials [N, P, kPartialFloats]
  int P;                // split path chunks per row
  int64_t chunk_vec;    // split path vectors per chunk
};

enum class Path { RowResidentSmall, RowResidentLarge, RowStream, Split };

// Building the cache (opd_sample_actions, opd_topk_support, opd_score_actions).
enum class CacheOp { Sample, Topk, Score };
// Top-k candidates kept in LDS before the exact counting fallback.
constexpr int kTopkCand = 4096;

struct CacheArgs {
  const void* logits;
  int64_t N, V, ld;
  int64_t nvec;         // 4-element vectors per row covering [0, V)
  int tail;             // valid elements in the last vector
  int K;                // draws M, support size k, or scored ids K
  const float* u;       // [N, K] uniforms (sampling)
  const int32_t* ids;   // [N, K] ids to score (scoring)
  const uint8_t* mask;  // nullable
  int32_t* ids_out;     // [N, K] draws or support (sampling, top-k)
  float* logp;          // [N, K] log-probs at the ids; nullable except for scoring
  float* lse_out;       // [N] nullable
  int redo;             // top-k: only the rows the streamed kernel marked
};

hipError_t launch_cache(const CacheArgs& a, CacheOp op, int in_dt, bool resident,
                        hipStream_t stream);

// Monte-Carlo diagnostics (opd_mc_diagnostics).
constexpr int kDiagMaxGroups = 8;
// workgroups of the first stage of the batch sums
constexpr int kDiagParts = 64;

struct DiagArgs {
  const float* lse;       // [N]
  const float* gathered;  // [N, M]
  const float* tau;       // [N, M]
  const float* beta;      // [N, M]
  int64_t N;
  int M;
  const uint8_t* mask;    // nullable
  float q, clip_eps;
  int n_groups;
  int group[kDiagMaxGroups];
  int64_t seq_len, nseq;
  int ncol;               // replicate columns per token
  // outputs (nullable)
  float *row_mean, *row_var, *row_rho_max, *rho_quantile, *clip_frac, *ratio_local, *ratio_seq;
  // workspace
  float* ws_rho;          // [N, M]
  float* ws_var;          // [N]
  uint32_t* ws_clip;      // [N]
  float* ws_vloc;         // [N, n_groups]
  float* ws_ycol;         // [N, ncol] (sequence ratios only, else NULL)
  float* ws_savg;         // [nseq, ncol] (sequence ratios only, else NULL)
  double* ws_parts;       // [kDiagParts, 3 + kDiagMaxGroups] first-stage sums
  uint32_t* ws_hist;      // [4 * 256 + 4] radix-select histograms and state
};

hipError_t launch_diag(const DiagArgs& a, hipStream_t stream);

// Launchers; each returns hipSuccess or the launch error.
hipError_t launch_rowwise(const Args& a, int est, int in_dt, int out_dt, Path path, bool read_row,
                          hipStream_t stream);
hipError_t launch_split(const Args& a, int est, int in_dt, int out_dt, bool read_row,
                        hipStream_t stream);
hipError_t launch_topk_sparse(const Args& a, int est, int in_dt, int out_dt, hipStream_t stream);
// The body of the loss entry points.  `scratch`, when not NULL, supplies the
// split path's workspace (at most scratch_bytes) from the library's static
// array instead of `workspace`; it is called only after every argument check.
typedef void* (*ScratchFn)();
int loss_call(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
              const ::opd_cache* cache, int32_t estimator, int32_t k, int32_t M,
              const uint8_t* mask, const ::opd_opts* opts, float* loss, void* dlogits,
              float* lse_out, float* gathered_out, float* coverage_out, void* workspace,
              size_t workspace_bytes,
              ScratchFn scratch, size_t scratch_bytes, void* stream);

hipError_t launch_validate(const int32_t* ids, const float* tau, const float* beta, int64_t N,
                           int64_t V, int K, int check_dups, int32_t* violations,
                           hipStream_t stream);

}  // namespace opd
