// C-ABI entry points of libopd: argument validation, path selection, launch.
// Every argument check runs on the host before any HIP call, so argument
// errors are reported without touching the device.
#include <limits.h>
#include <stdint.h>

#include "../../include/opd.h"
#include "opd_internal.h"

namespace {

using opd::Args;
using opd::Path;

// Below this many rows the split-vocabulary path runs (when it has a
// workspace): so few rows leave most of the 256 CUs idle, and splitting the
// rows over more workgroups outweighs the split path's second read of each
// row.  Measured on MI355X (16-sample MC, V = 151,936 bf16, inputs rotated
// so no step finds the last one's rows in the Infinity Cache), mean time per
// call, split against row path: N = 16: 24.8 against 30.5 us; 24: 23.5
// against 29.7; 32: 24.6 against 31.0; 48: 28.3 against 29.6; 64: 32.5
// against 31.0; 128: 54.8 against 37.2.
constexpr int64_t kSplitMaxRows = 64;
// Workgroups the split path aims for, and its largest chunk count.
constexpr int64_t kSplitTargetGroups = 8192;
constexpr int kSplitMaxChunks = 64;

constexpr uint32_t kKnownFlags =
    OPD_FLAG_SKIP_MASKED | OPD_FLAG_FORCE_ROWWISE | OPD_FLAG_FORCE_SPLITV;

bool valid_est(int32_t e) { return e >= OPD_FKL_TOPK && e <= OPD_RKL_TOPK_TRUNC; }
// renormalised top-k: only the k cached logits are needed
bool est_topk(int32_t e) { return e == OPD_FKL_TOPK || e == OPD_RKL_TOPK; }
bool est_trunc(int32_t e) { return e == OPD_FKL_TOPK_TRUNC || e == OPD_RKL_TOPK_TRUNC; }
// every estimator that reads the top-k cache (idx, k)
bool est_support(int32_t e) { return est_topk(e) || est_trunc(e); }
bool est_mc(int32_t e) {
  return e == OPD_RKL_MC1 || e == OPD_RKL_MC || (e >= OPD_RKL_MC_CLIP && e <= OPD_RKL_MC_NOIS);
}
bool est_clip(int32_t e) { return e == OPD_RKL_MC_CLIP || e == OPD_RKL_MC_OLD_CLIP; }

int mc_variant(int32_t e) {
  switch (e) {
    case OPD_RKL_MC_CLIP: return opd::MC_THETA_CLIP;
    case OPD_RKL_MC_OLD: return opd::MC_OLD;
    case OPD_RKL_MC_OLD_CLIP: return opd::MC_OLD_CLIP;
    case OPD_RKL_MC_NOIS: return opd::MC_NO_IS;
    case OPD_FKL_TOPK_TRUNC: return opd::TRUNC_FKL;
    case OPD_RKL_TOPK_TRUNC: return opd::TRUNC_RKL;
  }
  return opd::MC_THETA;
}

// The kernel family an estimator runs: the MC family and the truncated top-k
// KLs run the RKL_MC kernels (dense coefficient plus spikes).
int kernel_est(int32_t e) { return est_mc(e) || est_trunc(e) ? (int)opd::RKL_MC : (int)e; }
bool est_dense(int32_t e) { return e == OPD_FKL_DENSE || e == OPD_RKL_DENSE; }
int elt_bytes(int32_t dt) { return dt == OPD_BF16 ? 2 : 4; }
int elems_per_vec(int32_t) { return opd::kElemsPerVec; }

int check_shape(int64_t N, int64_t V, int64_t ld) {
  if (N < 0 || N > INT32_MAX) return OPD_ERR_SHAPE;
  if (V < 2 || V > INT32_MAX) return OPD_ERR_SHAPE;
  if (ld < V) return OPD_ERR_SHAPE;
  return OPD_OK;
}

int check_support(int32_t est, int64_t V, int32_t k, int32_t M) {
  if (est_support(est)) {
    const int64_t kmax = V < OPD_K_MAX ? V : OPD_K_MAX;
    if (k < 1 || k > kmax) return OPD_ERR_SUPPORT;
  } else if (est_mc(est)) {
    if (M < 1 || M > OPD_K_MAX) return OPD_ERR_SUPPORT;
    if (est == OPD_RKL_MC1 && M != 1) return OPD_ERR_SUPPORT;
  }
  return OPD_OK;
}

int check_flags(uint32_t flags) {
  if (flags & ~kKnownFlags) return OPD_ERR_FLAGS;
  if ((flags & OPD_FLAG_FORCE_ROWWISE) && (flags & OPD_FLAG_FORCE_SPLITV)) return OPD_ERR_FLAGS;
  return OPD_OK;
}

struct Plan {
  bool split;
  int P;
  int64_t chunk_vec;
  size_t ws_bytes;
};

// The split-path layout for N rows of nvec vectors: enough chunks for about
// kSplitTargetGroups workgroups, each chunk at least one vector per lane.
Plan split_plan(int64_t N, int64_t nvec) {
  Plan p{true, 1, nvec, 0};
  int64_t P = (kSplitTargetGroups + N - 1) / N;
  const int64_t by_width = nvec / opd::kSplitThreads;
  if (P > by_width) P = by_width;
  if (P > kSplitMaxChunks) P = kSplitMaxChunks;
  if (P < 1) P = 1;
  p.P = (int)P;
  p.chunk_vec = (nvec + P - 1) / P;
  p.ws_bytes = (size_t)N * (size_t)P * opd::kPartialFloats * sizeof(float);
  return p;
}

bool split_wanted(int64_t N, uint32_t flags) {
  if (flags & OPD_FLAG_FORCE_SPLITV) return true;
  if (flags & OPD_FLAG_FORCE_ROWWISE) return false;
  return N < kSplitMaxRows;
}

int64_t nvec_of(int64_t V, int32_t dt) {
  const int64_t epv = elems_per_vec(dt);
  return (V + epv - 1) / epv;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// A HIP grid holds fewer than 2^32 work-items: calls with more rows than one
// grid takes run as consecutive launches over row chunks.
constexpr int64_t kMaxGridLanes = 0xFFFFFFFFll;

// The arguments of rows [r0, r0 + n) of a loss call: every row-indexed
// pointer moves to row r0.
Args loss_rows(const Args& a, int64_t r0, int64_t n, int in_bytes, int out_bytes) {
  Args b = a;
  b.N = n;
  b.logits = (const char*)a.logits + r0 * a.ld * in_bytes;
  if (a.teacher) b.teacher = (const char*)a.teacher + r0 * a.ld * in_bytes;
  b.dlogits = (char*)a.dlogits + r0 * a.ld * out_bytes;
  if (a.ids) b.ids = a.ids + r0 * a.K;
  if (a.tau) b.tau = a.tau + r0 * a.K;
  if (a.beta) b.beta = a.beta + r0 * a.K;
  if (a.mask) b.mask = a.mask + r0;
  b.loss = a.loss + r0;
  if (a.lse_out) b.lse_out = a.lse_out + r0;
  if (a.gathered_out) b.gathered_out = a.gathered_out + r0 * a.K;
  if (a.coverage_out) b.coverage_out = a.coverage_out + 2 * r0;
  if (a.ws) b.ws = a.ws + r0 * a.P * opd::kPartialFloats;
  return b;
}

// The same for a cache-building call.
opd::CacheArgs cache_rows(const opd::CacheArgs& a, int64_t r0, int64_t n, int in_bytes) {
  opd::CacheArgs b = a;
  b.N = n;
  b.logits = (const char*)a.logits + r0 * a.ld * in_bytes;
  if (a.u) b.u = a.u + r0 * a.K;
  if (a.ids) b.ids = a.ids + r0 * a.K;
  if (a.mask) b.mask = a.mask + r0;
  if (a.ids_out) b.ids_out = a.ids_out + r0 * a.K;
  if (a.logp) b.logp = a.logp + r0 * a.K;
  if (a.lse_out) b.lse_out = a.lse_out + r0;
  return b;
}

// Launches a cache-building op over row chunks that each fit one grid
// (at most 1024 lanes per row).
hipError_t launch_cache_chunks(const opd::CacheArgs& a, opd::CacheOp op, int32_t dtype,
                               bool resident, hipStream_t s) {
  const int64_t max_rows = kMaxGridLanes / opd::kRowThreads;
  for (int64_t r0 = 0; r0 < a.N; r0 += max_rows) {
    const int64_t n = a.N - r0 < max_rows ? a.N - r0 : max_rows;
    const hipError_t e = opd::launch_cache(cache_rows(a, r0, n, elt_bytes(dtype)), op, dtype,
                                           resident, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Arguments shared by the cache-building entry points.
int check_row_call(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld, int32_t K,
                   int64_t kmax) {
  if (dtype != OPD_F32 && dtype != OPD_BF16) return OPD_ERR_DTYPE;
  if (int rc = check_shape(N, V, ld)) return rc;
  if (K < 1 || K > kmax) return OPD_ERR_SUPPORT;
  if (N > 0 && (!aligned16(logits) || (ld * elt_bytes(dtype)) % 16 != 0)) return OPD_ERR_ALIGN;
  return OPD_OK;
}

opd::CacheArgs row_args(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                        int32_t K, const uint8_t* mask, float* logp, float* lse_out) {
  opd::CacheArgs a{};
  a.logits = logits;
  a.N = N;
  a.V = V;
  a.ld = ld;
  a.nvec = nvec_of(V, dtype);
  a.tail = (int)(V - (a.nvec - 1) * elems_per_vec(dtype));
  a.K = K;
  a.mask = mask;
  a.logp = logp;
  a.lse_out = lse_out;
  return a;
}

// A row that fits the registers of one workgroup is read once.
bool row_fits(int64_t nvec, int32_t dtype) {
  return nvec <= (int64_t)opd::slots_large(dtype) * opd::kRowThreads;
}

// Workspace of opd_mc_diagnostics: regions in order, each 256-byte aligned.
struct DiagLayout {
  size_t rho, var, clip, vloc, ycol, savg, parts, hist, total;
  int ncol;
  int64_t nseq;
};

DiagLayout diag_layout(int64_t N, int32_t M, const int32_t* groups, int32_t n_groups,
                       int64_t seq_len) {
  DiagLayout l{};
  auto take = [&](size_t bytes) {
    const size_t at = l.total;
    l.total += (bytes + 255) & ~(size_t)255;
    return at;
  };
  l.ncol = M;
  for (int k = 0; k < n_groups; ++k) l.ncol += M / groups[k];
  const bool seq = seq_len > 0 && n_groups > 0;
  l.nseq = seq ? (N + seq_len - 1) / seq_len : 0;
  l.rho = take((size_t)N * M * 4);
  l.var = take((size_t)N * 4);
  l.clip = take((size_t)N * 4);
  l.vloc = take((size_t)N * (n_groups > 0 ? n_groups : 1) * 4);
  l.ycol = seq ? take((size_t)N * l.ncol * 4) : 0;
  l.savg = seq ? take((size_t)l.nseq * l.ncol * 4) : 0;
  l.parts = take((size_t)opd::kDiagParts * (3 + opd::kDiagMaxGroups) * 8);
  l.hist = take((4 * 256 + 4) * 4);
  return l;
}

// The diagnostics reduce over the whole batch in one grid of 64 lanes per
// token, so one call takes fewer than 2^32 / 64 tokens.
constexpr int64_t kDiagMaxRows = 0xFFFFFFFFll / 64;

int check_diag(int64_t N, int32_t M, float q, float clip_eps, const int32_t* groups,
               int32_t n_groups, int64_t seq_len) {
  if (N < 0 || N > kDiagMaxRows) return OPD_ERR_SHAPE;
  if (M < 1 || M > OPD_K_MAX) return OPD_ERR_SUPPORT;
  if (!(q > 0.0f && q <= 1.0f) || !(clip_eps >= 0.0f && clip_eps <= 3.0e38f)) return OPD_ERR_PARAM;
  if (n_groups < 0 || n_groups > opd::kDiagMaxGroups || seq_len < 0) return OPD_ERR_PARAM;
  if (n_groups > 0 && !groups) return OPD_ERR_NULL;
  for (int k = 0; k < n_groups; ++k)
    if (groups[k] < 1 || M % groups[k] != 0 || M / groups[k] < 2) return OPD_ERR_PARAM;
  return OPD_OK;
}

}  // namespace

extern "C" {

int opd_version(void) { return OPD_VERSION; }

const char* opd_status_string(int status) {
  switch (status) {
    case OPD_OK: return "ok";
    case OPD_ERR_NULL: return "a required pointer is NULL";
    case OPD_ERR_SHAPE: return "invalid shape (N, V or ld)";
    case OPD_ERR_SUPPORT: return "support size k or sample count M out of range";
    case OPD_ERR_DTYPE: return "unknown dtype";
    case OPD_ERR_ALIGN: return "pointer or row stride not 16-byte aligned";
    case OPD_ERR_WORKSPACE: return "workspace missing or too small for the split path";
    case OPD_ERR_ESTIMATOR: return "unknown estimator";
    case OPD_ERR_FLAGS: return "unknown or contradictory flags";
    case OPD_ERR_HIP: return "HIP runtime error";
    case OPD_ERR_PARAM: return "invalid scalar option or output (clip_eps, coverage_out)";
    case OPD_ERR_SCRATCH:
      return "the call needs more scratch than the no-allocation entry point holds";
  }
  return "unknown status";
}

size_t opd_workspace_bytes(int64_t N, int64_t V, int32_t dtype, int32_t estimator, int32_t k,
                           int32_t M, uint32_t flags) {
  if (!valid_est(estimator) || (dtype != OPD_F32 && dtype != OPD_BF16)) return 0;
  if (check_shape(N, V, V) != OPD_OK || N == 0) return 0;
  if (check_support(estimator, V, k, M) != OPD_OK || check_flags(flags) != OPD_OK) return 0;
  if (!split_wanted(N, flags)) return 0;
  return split_plan(N, nvec_of(V, dtype)).ws_bytes;
}

int opd_loss_fwd_bwd(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                     const opd_cache* cache, int32_t estimator, int32_t k, int32_t M,
                     const uint8_t* mask, const opd_opts* opts, float* loss, void* dlogits,
                     float* lse_out, float* gathered_out, float* coverage_out, void* workspace,
                     size_t workspace_bytes, void* stream) {
  return opd::loss_call(logits, dtype, N, V, ld, cache, estimator, k, M, mask, opts, loss, dlogits,
                        lse_out, gathered_out, coverage_out, workspace, workspace_bytes, nullptr,
                        0, stream);
}

}  // extern "C"

namespace opd {

int loss_call(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
              const opd_cache* cache, int32_t estimator, int32_t k, int32_t M,
              const uint8_t* mask, const opd_opts* opts, float* loss, void* dlogits,
              float* lse_out, float* gathered_out, float* coverage_out, void* workspace,
              size_t workspace_bytes, ScratchFn scratch, size_t scratch_bytes, void* stream) {
  if (!valid_est(estimator)) return OPD_ERR_ESTIMATOR;
  const opd_opts o = opts ? *opts : opd_opts{1.0f, OPD_F32, 0u, 0.2f};
  if (dtype != OPD_F32 && dtype != OPD_BF16) return OPD_ERR_DTYPE;
  if (o.dlogits_dtype != OPD_F32 && o.dlogits_dtype != OPD_BF16) return OPD_ERR_DTYPE;
  if (int rc = check_flags(o.flags)) return rc;
  if (int rc = check_shape(N, V, ld)) return rc;
  if (int rc = check_support(estimator, V, k, M)) return rc;
  if (est_clip(estimator) && !(o.clip_eps > 0.0f && o.clip_eps <= 3.0e38f)) return OPD_ERR_PARAM;
  // support coverage exists only for the estimators that read a support
  if (coverage_out && !est_support(estimator)) return OPD_ERR_PARAM;
  if (N == 0) return OPD_OK;

  if (!logits || !cache || !loss || !dlogits) return OPD_ERR_NULL;
  const int32_t* ids = nullptr;
  int K = 0;
  if (est_support(estimator)) {
    if (!cache->idx || !cache->teacher_logp) return OPD_ERR_NULL;
    ids = cache->idx;
    K = k;
  } else if (est_mc(estimator)) {
    if (!cache->sampled_ids || !cache->teacher_logp) return OPD_ERR_NULL;
    if (estimator != OPD_RKL_MC_NOIS && !cache->behav_logp) return OPD_ERR_NULL;
    ids = cache->sampled_ids;
    K = M;
  } else {
    if (!cache->teacher_logits) return OPD_ERR_NULL;
  }

  if (!aligned16(logits) || !aligned16(dlogits)) return OPD_ERR_ALIGN;
  if (est_dense(estimator) && !aligned16(cache->teacher_logits)) return OPD_ERR_ALIGN;
  if ((ld * elt_bytes(dtype)) % 16 != 0) return OPD_ERR_ALIGN;
  if ((ld * elt_bytes(o.dlogits_dtype)) % 16 != 0) return OPD_ERR_ALIGN;

  const int64_t nvec = nvec_of(V, dtype);
  const int epv = elems_per_vec(dtype);
  const int tail = (int)(V - (nvec - 1) * epv);

  Plan plan{false, 1, nvec, 0};
  if (split_wanted(N, o.flags)) {
    const Plan sp = split_plan(N, nvec);
    if (scratch) {
      // the no-allocation entry point: the library's static scratch array,
      // looked up only now that every argument has been checked
      if (sp.ws_bytes <= scratch_bytes) {
        workspace = scratch();
        if (!workspace) return OPD_ERR_HIP;
        plan = sp;
      } else if (o.flags & OPD_FLAG_FORCE_SPLITV) {
        return OPD_ERR_SCRATCH;
      }
    } else if (workspace && workspace_bytes >= sp.ws_bytes && aligned16(workspace)) {
      plan = sp;
    } else if (o.flags & OPD_FLAG_FORCE_SPLITV) {
      return OPD_ERR_WORKSPACE;
    }
  }

  Args a{};
  a.logits = logits;
  a.teacher = est_dense(estimator) ? cache->teacher_logits : nullptr;
  a.N = N;
  a.V = V;
  a.ld = ld;
  a.nvec = nvec;
  a.tail = tail;
  a.ids = ids;
  a.tau = est_dense(estimator) ? nullptr : cache->teacher_logp;
  a.beta = est_mc(estimator) && estimator != OPD_RKL_MC_NOIS ? cache->behav_logp : nullptr;
  a.K = K;
  a.mc_variant = mc_variant(estimator);
  a.clip_eps = o.clip_eps;
  a.mask = mask;
  a.gamma = o.grad_scale;
  a.skip_masked = (o.flags & OPD_FLAG_SKIP_MASKED) ? 1 : 0;
  a.loss = loss;
  a.dlogits = dlogits;
  a.lse_out = lse_out;
  a.gathered_out = est_dense(estimator) ? nullptr : gathered_out;
  a.coverage_out = coverage_out;
  a.ws = (float*)workspace;
  a.P = plan.P;
  a.chunk_vec = plan.chunk_vec;

  // The renormalised top-k estimators need the row itself only for lse_out
  // and the student's support coverage (both need L).
  const bool read_row = !est_topk(estimator) || lse_out != nullptr || coverage_out != nullptr;
  Path path = Path::RowStream;
  // register-resident rows (a partial last vector takes the kernels' TAIL
  // variant)
  if (nvec <= (int64_t)opd::slots_small(dtype) * opd::kRowThreads)
    path = Path::RowResidentSmall;
  else if (nvec <= (int64_t)opd::slots_large(dtype) * opd::kRowThreads)
    path = Path::RowResidentLarge;
  // rows per launch: the split grid has P workgroups of kSplitThreads lanes
  // per row, the others at most kRowThreads lanes per row (the top-k zero
  // fill chunks its own grid)
  const int64_t lanes_per_row =
      read_row && plan.split ? (int64_t)plan.P * opd::kSplitThreads : (int64_t)opd::kRowThreads;
  const int64_t max_rows = kMaxGridLanes / lanes_per_row;
  hipStream_t s = (hipStream_t)stream;
  hipError_t err = hipSuccess;
  for (int64_t r0 = 0; r0 < N && err == hipSuccess; r0 += max_rows) {
    const int64_t n = N - r0 < max_rows ? N - r0 : max_rows;
    const Args b = loss_rows(a, r0, n, elt_bytes(dtype), elt_bytes(o.dlogits_dtype));
    if (!read_row)
      err = opd::launch_topk_sparse(b, kernel_est(estimator), dtype, o.dlogits_dtype, s);
    else if (plan.split)
      err = opd::launch_split(b, kernel_est(estimator), dtype, o.dlogits_dtype, read_row, s);
    else
      err = opd::launch_rowwise(b, kernel_est(estimator), dtype, o.dlogits_dtype, path, read_row,
                                s);
  }
  return err == hipSuccess ? OPD_OK : OPD_ERR_HIP;
}

}  // namespace opd

extern "C" {

int opd_validate_cache(const opd_cache* cache, int32_t estimator, int64_t N, int64_t V,
                       int32_t k, int32_t M, int32_t* violations, void* stream) {
  if (!valid_est(estimator)) return OPD_ERR_ESTIMATOR;
  if (int rc = check_shape(N, V, V)) return rc;
  if (int rc = check_support(estimator, V, k, M)) return rc;
  if (est_dense(estimator) || N == 0) return OPD_OK;
  if (!cache || !violations) return OPD_ERR_NULL;
  const bool topk = est_support(estimator);
  const bool uses_beta = !topk && estimator != OPD_RKL_MC_NOIS;
  const int32_t* ids = topk ? cache->idx : cache->sampled_ids;
  if (!ids || !cache->teacher_logp || (uses_beta && !cache->behav_logp)) return OPD_ERR_NULL;
  const hipError_t err =
      opd::launch_validate(ids, cache->teacher_logp, uses_beta ? cache->behav_logp : nullptr, N,
                           V, topk ? k : M, topk ? 1 : 0, violations, (hipStream_t)stream);
  return err == hipSuccess ? OPD_OK : OPD_ERR_HIP;
}

int opd_sample_actions(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                       int32_t M, const float* uniforms, const uint8_t* mask, int32_t* sampled_ids,
                       float* logp, float* lse_out, void* stream) {
  if (int rc = check_row_call(logits, dtype, N, V, ld, M, OPD_K_MAX)) return rc;
  if (N == 0) return OPD_OK;
  if (!logits || !uniforms || !sampled_ids) return OPD_ERR_NULL;
  opd::CacheArgs a = row_args(logits, dtype, N, V, ld, M, mask, logp, lse_out);
  a.u = uniforms;
  a.ids_out = sampled_ids;
  const hipError_t err = launch_cache_chunks(a, opd::CacheOp::Sample, dtype, row_fits(a.nvec, dtype),
                                           (hipStream_t)stream);
  return err == hipSuccess ? OPD_OK : OPD_ERR_HIP;
}

int opd_topk_support(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld, int32_t k,
                     const uint8_t* mask, int32_t* idx, float* logp, float* lse_out,
                     void* stream) {
  if (int rc = check_row_call(logits, dtype, N, V, ld, k, V < OPD_K_MAX ? V : OPD_K_MAX)) return rc;
  if (N == 0) return OPD_OK;
  if (!logits || !idx) return OPD_ERR_NULL;
  opd::CacheArgs a = row_args(logits, dtype, N, V, ld, k, mask, logp, lse_out);
  a.ids_out = idx;
  const hipError_t err = launch_cache_chunks(a, opd::CacheOp::Topk, dtype, row_fits(a.nvec, dtype),
                                           (hipStream_t)stream);
  return err == hipSuccess ? OPD_OK : OPD_ERR_HIP;
}

int opd_score_actions(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                      const int32_t* ids, int32_t K, const uint8_t* mask, float* logp,
                      float* lse_out, void* stream) {
  if (int rc = check_row_call(logits, dtype, N, V, ld, K, OPD_K_MAX)) return rc;
  if (N == 0) return OPD_OK;
  if (!logits || !ids || !logp) return OPD_ERR_NULL;
  opd::CacheArgs a = row_args(logits, dtype, N, V, ld, K, mask, logp, lse_out);
  a.ids = ids;
  const hipError_t err = launch_cache_chunks(a, opd::CacheOp::Score, dtype, row_fits(a.nvec, dtype),
                                           (hipStream_t)stream);
  return err == hipSuccess ? OPD_OK : OPD_ERR_HIP;
}

size_t opd_mc_diag_workspace_bytes(int64_t N, int32_t M, const int32_t* group_sizes,
                                   int32_t n_groups, int64_t seq_len) {
  if (check_diag(N, M, 0.5f, 0.2f, group_sizes, n_groups, seq_len) != OPD_OK) return 0;
  return diag_layout(N, M, group_sizes, n_groups, seq_len).total;
}

int opd_mc_diagnostics(const float* lse, const float* gathered, const float* teacher_logp,
                       const float* behav_logp, int64_t N, int32_t M, const uint8_t* mask,
                       float quantile, float clip_eps, const int32_t* group_sizes,
                       int32_t n_groups, int64_t seq_len, const opd_mc_diag* out, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if (int rc = check_diag(N, M, quantile, clip_eps, group_sizes, n_groups, seq_len)) return rc;
  if (!out) return OPD_ERR_NULL;
  if (out->ratio_seq && (seq_len == 0 || n_groups == 0)) return OPD_ERR_PARAM;
  if (N == 0) return OPD_OK;
  if (!lse || !gathered || !teacher_logp || !behav_logp) return OPD_ERR_NULL;
  const DiagLayout l = diag_layout(N, M, group_sizes, n_groups, seq_len);
  if (!workspace || workspace_bytes < l.total || !aligned16(workspace)) return OPD_ERR_WORKSPACE;
  opd::DiagArgs a{};
  a.lse = lse;
  a.gathered = gathered;
  a.tau = teacher_logp;
  a.beta = behav_logp;
  a.N = N;
  a.M = M;
  a.mask = mask;
  a.q = quantile;
  a.clip_eps = clip_eps;
  a.n_groups = n_groups;
  for (int k = 0; k < n_groups; ++k) a.group[k] = group_sizes[k];
  a.seq_len = seq_len;
  a.nseq = l.nseq;
  a.ncol = l.ncol;
  a.row_mean = out->row_mean;
  a.row_var = out->row_var;
  a.row_rho_max = out->row_rho_max;
  a.rho_quantile = out->rho_quantile;
  a.clip_frac = out->clip_frac;
  a.ratio_local = out->ratio_local;
  a.ratio_seq = out->ratio_seq;
  char* ws = (char*)workspace;
  a.ws_rho = (float*)(ws + l.rho);
  a.ws_var = (float*)(ws + l.var);
  a.ws_clip = (uint32_t*)(ws + l.clip);
  a.ws_vloc = (float*)(ws + l.vloc);
  a.ws_ycol = l.nseq ? (float*)(ws + l.ycol) : nullptr;
  a.ws_savg = l.nseq ? (float*)(ws + l.savg) : nullptr;
  a.ws_parts = (double*)(ws + l.parts);
  a.ws_hist = (uint32_t*)(ws + l.hist);
  const hipError_t err = opd::launch_diag(a, (hipStream_t)stream);
  return err == hipSuccess ? OPD_OK : OPD_ERR_HIP;
}

}  // extern "C"
