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
//   seq      one wavefront per (sequence, replicate column): the column's
//            average over the sequence's valid tokens
//   select   the nearest-rank quantile of rho by radix selection over its
//            bits (rho >= 0, so bits order like values): four 8-bit passes,
//            each an integer histogram then a one-workgroup pick
//   final    fixed-order sums in double (per-range parts, then one
//            workgroup), the per-sequence set variances, the batch outputs
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

// One wavefront per (sequence, replicate column): the average of that column
// over the sequence's valid tokens (lanes stride the tokens; fixed-order
// butterfly sum).  The variances over the columns of each set are taken in
// the final pass.
__global__ void __launch_bounds__(kDiagThreads) k_diag_seq(DiagArgs a) {
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.y * kDiagWaves + (threadIdx.x >> 6);
  if (c >= a.ncol) return;
  const int64_t s = blockIdx.x;
  const int64_t t0 = s * a.seq_len, t1 = min(t0 + a.seq_len, a.N);
  float acc = 0.f;
  uint32_t nv = 0;
  for (int64_t t = t0 + lane; t < t1; t += 64) {
    if (a.mask && a.mask[t] == 0) continue;
    acc += a.ws_ycol[t * a.ncol + c];
    ++nv;
  }
  acc = wave_sum(acc);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) nv += __shfl_xor(nv, o, 64);
  if (lane == 0) a.ws_savg[s * a.ncol + c] = nv ? acc / (float)nv : __builtin_nanf("");
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

// One workgroup of 256 lanes, one bucket each: an inclusive scan of the
// counts finds the bucket holding the wanted rank.
__global__ void __launch_bounds__(256) k_diag_pick(DiagArgs a, int pass) {
  __shared__ uint32_t s_w[4];
  __shared__ uint32_t s_rank;
  uint32_t* sel = a.ws_hist + 4 * 256;
  const uint32_t* hist = a.ws_hist + pass * 256;
  const int b = threadIdx.x, lane = b & 63, w = b >> 6;
  const uint32_t h = hist[b];
  // inclusive scan of the counts (integers: any order gives the same sums)
  uint32_t incl = h;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = (uint32_t)__shfl_up((int)incl, o, 64);
    if (lane >= o) incl += t;
  }
  if (lane == 63) s_w[w] = incl;
  __syncthreads();
  for (int j = 0; j < w; ++j) incl += s_w[j];
  const uint32_t n = s_w[0] + s_w[1] + s_w[2] + s_w[3];
  if (b == 0) {
    if (pass == 0) {
      sel[2] = n;
      // nearest rank: the ceil(q n)-th smallest, at least the first
      const double want = ceil((double)a.q * (double)n);
      s_rank = n == 0 ? 1u : (uint32_t)(want < 1.0 ? 1.0 : (want > n ? (double)n : want));
    } else {
      s_rank = sel[1];
    }
  }
  __syncthreads();
  const uint32_t rank = s_rank, excl = incl - h;
  // the one bucket with excl < rank <= incl (the last one if rounding ever
  // left rank beyond the total)
  if ((excl < rank && rank <= incl) || (b == 255 && incl < rank)) {
    const uint32_t prefix = pass == 0 ? 0u : sel[0];
    sel[0] = (prefix << 8) | (uint32_t)b;
    sel[1] = rank - excl;
    if (pass == 3 && a.rho_quantile)
      a.rho_quantile[0] = sel[2] == 0 ? __builtin_nanf("") : __uint_as_float((prefix << 8) | (uint32_t)b);
  }
}

// Batch sums in two fixed-order stages: kDiagParts workgroups each sum a
// contiguous range of tokens (lane-strided, then the lanes' partials in lane
// order), in double; one workgroup then adds the parts in order and forms
// the outputs.  Quantities: [0] sum of row_var, [1] clipped entries, [2]
// valid tokens, [3 + k] sum of the group-k variances.
__device__ __forceinline__ double block_sum_ordered(double v, double* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0)
    for (int j = 0; j < kDiagThreads; ++j) r += red[j];
  __syncthreads();
  return r;  // lane 0 only
}

__global__ void __launch_bounds__(kDiagThreads) k_diag_parts(DiagArgs a) {
  __shared__ double red[kDiagThreads];
  const int nq = 3 + a.n_groups;
  const int64_t per = (a.N + kDiagParts - 1) / kDiagParts;
  const int64_t t0 = blockIdx.x * per, t1 = min(t0 + per, a.N);
  double* out = a.ws_parts + (int64_t)blockIdx.x * (3 + kDiagMaxGroups);
  for (int q = 0; q < nq; ++q) {
    double v = 0.0;
    for (int64_t t = t0 + threadIdx.x; t < t1; t += kDiagThreads) {
      if (a.mask && a.mask[t] == 0) continue;
      if (q == 0)
        v += a.M >= 2 ? (double)a.ws_var[t] : 0.0;
      else if (q == 1)
        v += (double)a.ws_clip[t];
      else if (q == 2)
        v += 1.0;
      else
        v += (double)a.ws_vloc[t * a.n_groups + (q - 3)];
    }
    v = block_sum_ordered(v, red);
    if (threadIdx.x == 0) out[q] = v;
  }
}

// Unbiased variance over the columns [c0, c0 + n) of one sequence.
__device__ double seq_set_var(const float* avg, int c0, int n) {
  double mean = 0.0;
  for (int c = c0; c < c0 + n; ++c) mean += avg[c];
  mean /= n;
  double ss = 0.0;
  for (int c = c0; c < c0 + n; ++c) ss += (avg[c] - mean) * (avg[c] - mean);
  return ss / (n - 1);
}

__global__ void __launch_bounds__(kDiagThreads) k_diag_final(DiagArgs a) {
  __shared__ double red[kDiagThreads];
  __shared__ double tot[3 + kDiagMaxGroups];
  __shared__ double seq[kDiagMaxGroups + 1];
  const int tid = threadIdx.x;
  if (tid < 3 + a.n_groups) {
    double v = 0.0;
    for (int p = 0; p < kDiagParts; ++p) v += a.ws_parts[p * (3 + kDiagMaxGroups) + tid];
    tot[tid] = v;
  }
  // sequence level: set 0 = the M single-draw columns, set k >= 1 = the
  // groups of size group[k - 1]; sequences without a valid token are skipped
  if (a.ws_savg) {
    for (int k = 0; k <= a.n_groups; ++k) {
      int c0 = 0, n = a.M;
      if (k > 0) {
        c0 = a.M;
        for (int j = 0; j < k - 1; ++j) c0 += a.M / a.group[j];
        n = a.M / a.group[k - 1];
      }
      double v = 0.0;
      for (int64_t s = tid; s < a.nseq; s += kDiagThreads) {
        const float* avg = a.ws_savg + s * a.ncol;
        if (avg[0] == avg[0]) v += seq_set_var(avg, c0, n);
      }
      v = block_sum_ordered(v, red);
      if (tid == 0) seq[k] = v;
    }
  }
  __syncthreads();
  if (tid == 0) {
    const double n = tot[2] * (double)a.M;
    if (a.clip_frac) a.clip_frac[0] = n > 0 ? (float)(tot[1] / n) : __builtin_nanf("");
    for (int k = 0; k < a.n_groups; ++k) {
      if (a.ratio_local) a.ratio_local[k] = (float)(tot[3 + k] / tot[0]);
      if (a.ratio_seq && a.ws_savg) a.ratio_seq[k] = (float)(seq[1 + k] / seq[0]);
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
  if (a.ws_savg)
    hipLaunchKernelGGL(k_diag_seq, dim3((unsigned)a.nseq, (unsigned)((a.ncol + kDiagWaves - 1) / kDiagWaves)),
                       blk, 0, stream, a);
  if (a.rho_quantile) {
    const int64_t total = a.N * a.M;
    const int64_t blocks = (total + kDiagThreads - 1) / kDiagThreads;
    const unsigned grid = (unsigned)(blocks < 2048 ? blocks : 2048);
    for (int pass = 0; pass < 4; ++pass) {
      hipLaunchKernelGGL(k_diag_hist, dim3(grid), blk, 0, stream, a, pass);
      hipLaunchKernelGGL(k_diag_pick, dim3(1), dim3(256), 0, stream, a, pass);
    }
  }
  hipLaunchKernelGGL(k_diag_parts, dim3(kDiagParts), blk, 0, stream, a);
  hipLaunchKernelGGL(k_diag_final, dim3(1), blk, 0, stream, a);
  return hipGetLastError();
}

}  // namespace opd
