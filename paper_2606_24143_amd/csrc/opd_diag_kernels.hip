// HIP kernels of the Monte-Carlo diagnostics for gfx950 (MI355X).
//
// From what the loss call returns or reads per token t (the log-partition
// L_t, the student logits at the M cached draws, the cached teacher and
// behaviour log-probs), the one-sample terms of the estimator
//   log p = z - L,  A = tau - log p,  rho = exp(log p - beta),  X = -rho A
// give the statistics of Sec. 5.2 (the tail of rho_theta, Fig. 5) and App. E
// (variance of the m-sample estimator at a fixed prefix and averaged over a
// sequence, Table 6):
//   rows     one wavefront per token: mean, unbiased variance and largest
//            rho of its M terms; count of rho outside [1 - eps, 1 + eps];
//            means of replicate groups of m draws and their variance
//   seq      one workgroup per sequence: token averages of each replicate
//            column, and their variance per group size
//   select   the nearest-rank quantile of rho by radix selection over its
//            bits (rho >= 0, so bits order like values): four 8-bit passes,
//            each an integer histogram then a one-workgroup pick
//   final    one workgroup: fixed-order sums in double, the batch outputs
// Integer histograms make the selection exact and order-independent; every
// floating-point sum has a fixed order.
#include <math.h>

#include "opd_device.h"

namespace opd {
namespace {

constexpr int kDiagThreads = 256;
constexpr int kDiagWaves = kDiagThreads / 64;

// Sort key of one ratio: its bits, with every NaN mapped above +inf.
__device__ __forceinline__ uint32_t rho_key(float r) {
  return r != r ? 0x7FC00000u : __float_as_uint(r);
}

__device__ __forceinline__ float one_rho(const DiagArgs& a, int64_t t, int i, float L, float* X) {
  const int64_t e = t * a.M + i;
  const float lp = a.gathered[e] - L;
  const float r = fast_exp2((lp - a.beta[e]) * kLog2e);
  *X = -r * (a.tau[e] - lp);
  return r;
}

__global__ void __launch_bounds__(kDiagThreads) k_diag_rows(DiagArgs a) {
  __shared__ float s_x[kDiagWaves][kKMax];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kDiagWaves + w;
  if (t >= a.N) return;
  const int M = a.M;
  const bool valid = !a.mask || a.mask[t] != 0;
  if (!valid) {
    if (lane == 0) {
      if (a.row_mean) a.row_mean[t] = 0.f;
      if (a.row_var) a.row_var[t] = 0.f;
      if (a.row_rho_max) a.row_rho_max[t] = 0.f;
    }
    return;
  }
  const float L = a.lse[t];
  float sum = 0.f, rmax = kNegInf;
  uint32_t clip = 0;
  for (int i = lane; i < M; i += 64) {
    float X;
    const float r = one_rho(a, t, i, L, &X);
    a.ws_rho[t * M + i] = r;
    s_x[w][i] = X;
    sum += X;
    rmax = fmaxf(rmax, r);
    clip += fabsf(r - 1.f) > a.clip_eps ? 1u : 0u;
  }
  sum = wave_sum(sum);
  rmax = wave_max(rmax);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) clip += __shfl_xor(clip, o, 64);
  const float mean = sum / (float)M;
  float ss = 0.f;
  for (int i = lane; i < M; i += 64) {
    const float d = s_x[w][i] - mean;
    ss += d * d;
  }
  ss = wave_sum(ss);
  const float var = M >= 2 ? ss / (float)(M - 1) : __builtin_nanf("");
  if (lane == 0) {
    if (a.row_mean) a.row_mean[t] = mean;
    if (a.row_var) a.row_var[t] = var;
    if (a.row_rho_max) a.row_rho_max[t] = rmax == kNegInf ? __builtin_nanf("") : rmax;
    a.ws_var[t] = var;
    a.ws_clip[t] = clip;
  }
  // replicate groups of m consecutive draws (single draws first, for the
  // sequence-level baseline)
  float* ycol = a.ws_ycol ? a.ws_ycol + t * a.ncol : nullptr;
  if (ycol)
    for (int i = lane; i < M; i += 64) ycol[i] = s_x[w][i];
  int col = M;
  for (int k = 0; k < a.n_groups; ++k) {
    const int m = a.group[k], G = M / m;
    float ys = 0.f;
    float y[4] = {0.f, 0.f, 0.f, 0.f};  // G <= 256: four groups per lane at most
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const int g = lane + 64 * h;
      if (g < G) {
        float acc = 0.f;
        for (int i = g * m; i < g * m + m; ++i) acc += s_x[w][i];
        y[h] = acc / (float)m;
        ys += y[h];
        if (ycol) ycol[col + g] = y[h];
      }
    }
    const float ym = wave_sum(ys) / (float)G;
    float yss = 0.f;
#pragma unroll
    for (int h = 0; h < 4; ++h)
      if (lane + 64 * h < G) yss += (y[h] - ym) * (y[h] - ym);
    yss = wave_sum(yss);
    if (lane == 0) a.ws_vloc[t * a.n_groups + k] = yss / (float)(G - 1);
    col += G;
  }
}

// One workgroup per sequence of seq_len tokens: the token average of every
// replicate column (valid tokens only), then the unbiased variance over the
// columns of each set (single draws, then each group size).
__global__ void __launch_bounds__(kDiagThreads) k_diag_seq(DiagArgs a) {
  __shared__ float s_avg[kDiagMaxCols];
  __shared__ int s_nv;
  const int64_t s = blockIdx.x;
  const int64_t t0 = s * a.seq_len, t1 = min(t0 + a.seq_len, a.N);
  if (threadIdx.x == 0) {
    int nv = 0;
    for (int64_t t = t0; t < t1; ++t) nv += (!a.mask || a.mask[t] != 0) ? 1 : 0;
    s_nv = nv;
  }
  __syncthreads();
  const int nv = s_nv;
  float* out = a.ws_wseq + s * (a.n_groups + 1);
  if (nv == 0) {
    if (threadIdx.x <= a.n_groups) out[threadIdx.x] = __builtin_nanf("");
    return;
  }
  for (int c = threadIdx.x; c < a.ncol; c += kDiagThreads) {
    float acc = 0.f;
    for (int64_t t = t0; t < t1; ++t)
      if (!a.mask || a.mask[t] != 0) acc += a.ws_ycol[t * a.ncol + c];
    s_avg[c] = acc / (float)nv;
  }
  __syncthreads();
  // set k = 0: the M single-draw columns; set k >= 1: the groups of size
  // group[k - 1]
  if (threadIdx.x <= a.n_groups) {
    const int k = threadIdx.x;
    int c0 = 0, n = a.M;
    if (k > 0) {
      c0 = a.M;
      for (int j = 0; j < k - 1; ++j) c0 += a.M / a.group[j];
      n = a.M / a.group[k - 1];
    }
    float mean = 0.f;
    for (int c = c0; c < c0 + n; ++c) mean += s_avg[c];
    mean /= (float)n;
    float ss = 0.f;
    for (int c = c0; c < c0 + n; ++c) ss += (s_avg[c] - mean) * (s_avg[c] - mean);
    out[k] = ss / (float)(n - 1);
  }
}

// The radix-select state lives in the workspace: sel[0] = key prefix chosen
// so far, sel[1] = rank still to find within it, sel[2] = count of entries.
__global__ void __launch_bounds__(kDiagThreads) k_diag_zero(DiagArgs a) {
  for (int i = threadIdx.x; i < 4 * 256 + 4; i += kDiagThreads) a.ws_hist[i] = 0u;
}

__global__ void __launch_bounds__(kDiagThreads) k_diag_hist(DiagArgs a, int pass) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0u;
  __syncthreads();
  const uint32_t prefix = pass ? a.ws_hist[4 * 256 + 0] : 0u;
  const int shift = 24 - 8 * pass;
  const int64_t total = a.N * a.M;
  for (int64_t e = (int64_t)blockIdx.x * kDiagThreads + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * kDiagThreads) {
    const int64_t t = e / a.M;
    if (a.mask && a.mask[t] == 0) continue;
    const uint32_t key = rho_key(a.ws_rho[e]);
    if (pass == 0 || (key >> (shift + 8)) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&a.ws_hist[pass * 256 + threadIdx.x], h[threadIdx.x]);
}

// One workgroup: the bucket holding the wanted rank (a sequential scan of 256
// counts by one lane; negligible).
__global__ void __launch_bounds__(64) k_diag_pick(DiagArgs a, int pass) {
  if (threadIdx.x != 0) return;
  uint32_t* sel = a.ws_hist + 4 * 256;
  const uint32_t* hist = a.ws_hist + pass * 256;
  uint32_t rank;
  if (pass == 0) {
    uint32_t n = 0;
    for (int b = 0; b < 256; ++b) n += hist[b];
    sel[2] = n;
    // nearest rank: the ceil(q n)-th smallest, at least the first
    const double want = ceil((double)a.q * (double)n);
    rank = n == 0 ? 0u : (uint32_t)(want < 1.0 ? 1.0 : (want > n ? (double)n : want));
    sel[0] = 0u;
  } else {
    rank = sel[1];
  }
  uint32_t before = 0, b = 0;
  for (; b < 255; ++b) {
    if (before + hist[b] >= rank) break;
    before += hist[b];
  }
  sel[0] = (sel[0] << 8) | b;
  sel[1] = rank - before;
  if (pass == 3 && a.rho_quantile)
    a.rho_quantile[0] = sel[2] == 0 ? __builtin_nanf("") : __uint_as_float(sel[0]);
}

// Fixed-order sums in double by one workgroup: lane j takes rows j, j + 256,
// ..., then a sequential pass over the 256 partials.
__global__ void __launch_bounds__(kDiagThreads) k_diag_final(DiagArgs a) {
  __shared__ double s_p[kDiagThreads];
  __shared__ double s_tot[4 + 2 * (kDiagMaxGroups + 1)];
  const int tid = threadIdx.x;
  auto reduce = [&](double v) {
    s_p[tid] = v;
    __syncthreads();
    double r = 0.0;
    if (tid == 0)
      for (int j = 0; j < kDiagThreads; ++j) r += s_p[j];
    __syncthreads();
    return r;  // lane 0 only
  };
  double var = 0.0, clip = 0.0, rows = 0.0;
  for (int64_t t = tid; t < a.N; t += kDiagThreads) {
    if (a.mask && a.mask[t] == 0) continue;
    rows += 1.0;
    clip += (double)a.ws_clip[t];
    if (a.M >= 2) var += (double)a.ws_var[t];
  }
  var = reduce(var);
  clip = reduce(clip);
  rows = reduce(rows);
  if (tid == 0) {
    s_tot[0] = var;
    s_tot[1] = clip;
    s_tot[2] = rows;
  }
  for (int k = 0; k < a.n_groups; ++k) {
    double v = 0.0;
    for (int64_t t = tid; t < a.N; t += kDiagThreads)
      if (!a.mask || a.mask[t] != 0) v += (double)a.ws_vloc[t * a.n_groups + k];
    v = reduce(v);
    if (tid == 0) s_tot[4 + k] = v;
  }
  if (a.ws_wseq) {
    for (int k = 0; k <= a.n_groups; ++k) {
      double v = 0.0;
      for (int64_t s = tid; s < a.nseq; s += kDiagThreads) {
        const float x = a.ws_wseq[s * (a.n_groups + 1) + k];
        if (x == x) v += (double)x;  // sequences with no valid token are NaN
      }
      v = reduce(v);
      if (tid == 0) s_tot[4 + kDiagMaxGroups + k] = v;
    }
  }
  if (tid == 0) {
    const double n = s_tot[2] * (double)a.M;
    if (a.clip_frac) a.clip_frac[0] = n > 0 ? (float)(s_tot[1] / n) : __builtin_nanf("");
    for (int k = 0; k < a.n_groups; ++k) {
      if (a.ratio_local) a.ratio_local[k] = (float)(s_tot[4 + k] / s_tot[0]);
      if (a.ratio_seq && a.ws_wseq)
        a.ratio_seq[k] =
            (float)(s_tot[4 + kDiagMaxGroups + 1 + k] / s_tot[4 + kDiagMaxGroups]);
    }
  }
}

}  // namespace

hipError_t launch_diag(const DiagArgs& a, hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  const dim3 blk(kDiagThreads);
  hipLaunchKernelGGL(k_diag_zero, dim3(1), blk, 0, stream, a);
  hipLaunchKernelGGL(k_diag_rows, dim3((unsigned)((a.N + kDiagWaves - 1) / kDiagWaves)), blk, 0,
                     stream, a);
  if (a.ws_wseq) hipLaunchKernelGGL(k_diag_seq, dim3((unsigned)a.nseq), blk, 0, stream, a);
  if (a.rho_quantile) {
    const int64_t total = a.N * a.M;
    const int64_t blocks = (total + kDiagThreads - 1) / kDiagThreads;
    const unsigned grid = (unsigned)(blocks < 2048 ? blocks : 2048);
    for (int pass = 0; pass < 4; ++pass) {
      hipLaunchKernelGGL(k_diag_hist, dim3(grid), blk, 0, stream, a, pass);
      hipLaunchKernelGGL(k_diag_pick, dim3(1), dim3(64), 0, stream, a, pass);
    }
  }
  hipLaunchKernelGGL(k_diag_final, dim3(1), blk, 0, stream, a);
  return hipGetLastError();
}

}  // namespace opd
