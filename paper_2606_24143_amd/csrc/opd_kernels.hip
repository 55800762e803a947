// HIP kernels of the learner-time OPD loss for gfx950 (MI355X).
//
// Per token row t (Sec. 3 notation): logits z, L = log sum_j exp(z_j),
// log p_theta(j) = z_j - L.  Every estimator is a two-sweep computation over
// the vocabulary:
//   sweep 1  online max / sum-exp over V (plus, for the dense estimators, the
//            teacher's normaliser and the two cross sums that give D_F, D_R);
//   gather   the student logits at the cached ids;
//   estimate one wavefront turns (L, gathered logits, cached teacher and
//            behaviour log-probs) into the loss, a per-row coefficient C of
//            p_theta and up to K point corrections ("spikes");
//   sweep 2  dlogits_j = C * p_theta(j) + spikes at cached ids, or the dense
//            gradient.
// The work is HBM-bound (a few VALU operations per byte, no contraction), so
// the kernels are organised around bytes: wide coalesced loads and stores, one read
// of each logit where the row fits in registers, non-temporal hints so the
// stream does not evict anything useful from L2.
#include <math.h>
#include <type_traits>

#include "opd_device.h"

namespace opd {
namespace {

// Spike filter: one bit per 16-byte vector index (mod kFilterBits).  A set
// bit sends that vector through the exact K-entry check; false positives
// only cost the check.
constexpr int kFilterBits = 16384;
constexpr int kFilterWords = kFilterBits / 32;

constexpr bool is_mc(int e) { return e == RKL_MC || e == RKL_MC1; }
constexpr bool is_dense(int e) { return e == FKL_DENSE || e == RKL_DENSE; }
constexpr bool is_topk(int e) { return e == FKL_TOPK || e == RKL_TOPK; }

// Per-row constants of the dense estimators from the merged statistics.
struct DenseRow {
  float Lz, Ly;  // log-partitions of student and teacher rows
  float ez;      // E_p[z - y]
  float loss;
};
template <int EST>
__device__ __forceinline__ DenseRow dense_row(const Stats& s) {
  DenseRow d;
  d.Lz = s.mz + logf(s.sz);
  d.Ly = s.my + logf(s.sy);
  d.ez = s.tr / s.sz;
  // D_R = E_p[(z - Lz) - (y - Ly)],  D_F = E_q[(y - Ly) - (z - Lz)]
  d.loss = EST == RKL_DENSE ? d.ez + (d.Ly - d.Lz) : s.tf / s.sy + (d.Lz - d.Ly);
  return d;
}

// Gradient values of one vector for the dense estimators:
//   forward  g = gamma (p - q);   reverse  g = gamma p ((z - y) - E_p[z - y]),
// the softmax-Jacobian form of eq. reverse-kl-gradient.  |gamma| enters the
// exponents as log2|gamma| (DenseGrad) and its sign the operand order (NEG),
// so no element is multiplied by gamma.
struct DenseGrad {
  float nLz, nLy;  // log2|gamma| - L * log2(e), student and teacher
  float ez;
  bool neg;        // gamma < 0
};
// (row-uniform values: read back as scalars, so they occupy no lane registers)
__device__ __forceinline__ float uniform(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}
__device__ __forceinline__ DenseGrad dense_grad_consts(const DenseRow& d, float gamma) {
  const float lg = log2f(fabsf(gamma));  // -inf for gamma = 0: every g is 0
  return DenseGrad{uniform(fmaf(-d.Lz, kLog2e, lg)), uniform(fmaf(-d.Ly, kLog2e, lg)),
                   uniform(d.ez), gamma < 0.f};
}
template <class TI, int EST, bool NEG>
__device__ __forceinline__ void dense_grad(const typename TI::Vec& xz, const typename TI::Vec& xy,
                                           const DenseGrad& k, float (&g)[TI::EPV]) {
  float fz[TI::EPV], fy[TI::EPV];
  unpack<TI>(xz, fz);
  unpack<TI>(xy, fy);
#pragma unroll
  for (int e = 0; e < TI::EPV; ++e) {
    const float p = fast_exp2(fmaf(fz[e], kLog2e, k.nLz));  // |gamma| p
    if constexpr (EST == FKL_DENSE) {
      const float q = fast_exp2(fmaf(fy[e], kLog2e, k.nLy));
      g[e] = NEG ? q - p : p - q;
    } else {
      // p = 0 where both rows are -inf and the difference is NaN: the legacy
      // multiply keeps that entry 0 (a term of zero weight is zero)
      g[e] = NEG ? mul_zero_safe(p, (fy[e] - fz[e]) + k.ez)
                 : mul_zero_safe(p, (fz[e] - fy[e]) - k.ez);
    }
  }
}
template <class TI, int EST>
__device__ __forceinline__ void dense_grad(const typename TI::Vec& xz, const typename TI::Vec& xy,
                                           const DenseGrad& k, float (&g)[TI::EPV]) {
  if (k.neg)
    dense_grad<TI, EST, true>(xz, xy, k, g);
  else
    dense_grad<TI, EST, false>(xz, xy, k, g);
}

// ---------------------------------------------------------------- cache, estimator, spikes

struct CacheLds {
  int id[kKMax];  // -1 marks an id outside [0, V)
  float z[kKMax];
  float t[kKMax];
  float b[kKMax];
  float w[kKMax];  // spike weights, already scaled by gamma
  uint32_t filter[kFilterWords];
  uint64_t skey[kKMax];  // (vector << 32 | entry), ascending (set_filter)
  uint64_t ukey[kKMax];  // the same keys by entry index
  float C;        // coefficient of p_theta in the gradient row
  int bad;        // the row has an id outside [0, V)
};

// Wave 0: read the row's cache entries and gather the student logits there.
template <class TI>
__device__ __forceinline__ void load_cache(const Args& a, int64_t row, const void* zrow,
                                           CacheLds& c) {
  const int lane = threadIdx.x & 63;
  const int K = a.K;
  int bad = 0;
  for (int i = lane; i < K; i += 64) {
    const int32_t id = a.ids[row * K + i];
    const bool ok = id >= 0 && (int64_t)id < a.V;
    c.id[i] = ok ? id : -1;
    c.z[i] = ok ? load_elem<TI>(zrow, id) : __builtin_nanf("");
    c.t[i] = a.tau[row * K + i];
    c.b[i] = a.beta ? a.beta[row * K + i] : 0.f;
    bad |= ok ? 0 : 1;
  }
  bad = __any(bad);
  if (lane == 0) c.bad = bad;
}

// Wave 0: the estimator arithmetic of one row.  gmu = gamma for a valid row.
// Writes the spike weights and C into LDS and returns the loss (lane-uniform).
// `variant` selects the per-sample weight of the Monte-Carlo family.
template <int EST>
__device__ __forceinline__ float estimate(int K, float L, float gmu, int variant, float eps,
                                          CacheLds& c) {
  const int lane = threadIdx.x & 63;
  if constexpr (is_mc(EST)) {
    // Surrogates of Sec. 5.1 over behaviour samples a_i ~ p_old:
    //   -(1/M) sum_i rho_i sg(A_i)                       (noclip)
    //   -(1/M) sum_i min(rho_i sg(A_i), rho_bar_i sg(A_i)) (clip)
    // with A = A_theta = tau - log p_theta (recomputed here) or A_old = tau - beta,
    // rho = p_theta / p_old; and the App. F ablation without the ratio,
    //   -(1/M) sum_i sg(A_theta,i) log p_theta(a_i).
    // The per-sample gradient weight w_i multiplies (1[j = a_i] - p_j); a clipped
    // term selected outside [1 - eps, 1 + eps] has w_i = 0.
    if (variant == TRUNC_FKL || variant == TRUNC_RKL) {
      // Truncated top-k (the dense KL summed over S, full-vocabulary
      // normalisers; Sec. 3): forward: C = Z_q^S, spikes -q_i;
      // reverse: u_i = p_i (log p_i - log q_i + 1), C = -sum u_i, spikes u_i.
      const bool rev = variant == TRUNC_RKL;
      float acc_c = 0.f, acc_kl = 0.f;
      for (int i = lane; i < K; i += 64) {
        const float lp = c.z[i] - L;
        float spike, cterm, kl;
        if (rev) {
          const float p = expf(lp);
          spike = p * ((lp - c.t[i]) + 1.f);
          cterm = -spike;
          kl = p * (lp - c.t[i]);
        } else {
          const float q = expf(c.t[i]);
          spike = -q;
          cterm = q;
          kl = q * (c.t[i] - lp);
        }
        c.w[i] = gmu * spike;
        acc_c += cterm;
        acc_kl += kl;
      }
      const float cc = wave_sum(acc_c);
      const float kl = wave_sum(acc_kl);
      if (lane == 0) c.C = gmu * cc;
      return kl;
    }
    const bool old_adv = variant == MC_OLD || variant == MC_OLD_CLIP;
    const bool clip = variant == MC_THETA_CLIP || variant == MC_OLD_CLIP;
    const bool no_is = variant == MC_NO_IS;
    float acc_w = 0.f, acc_term = 0.f;
    for (int i = lane; i < K; i += 64) {
      const float lp = c.z[i] - L;
      const float A = old_adv ? c.t[i] - c.b[i] : c.t[i] - lp;
      float w, term;
      if (no_is) {
        w = A;
        term = A * lp;
      } else {
        const float rho = expf(lp - c.b[i]);
        w = rho * A;
        term = w;
        if (clip) {
          const float clipped = fminf(fmaxf(rho, 1.f - eps), 1.f + eps) * A;
          if (!(w <= clipped)) {
            term = clipped;
            w = 0.f;
          }
        }
      }
      c.w[i] = w;
      acc_w += w;
      acc_term += term;
    }
    const float inv_m = 1.0f / (float)K;
    const float cw = wave_sum(acc_w) * inv_m;
    const float total = wave_sum(acc_term) * inv_m;
    for (int i = lane; i < K; i += 64) c.w[i] = -gmu * c.w[i] * inv_m;
    if (lane == 0) c.C = gmu * cw;
    return -total;
  } else {
    // renormalised restricted KL on S (Sec. 3; App. A.1): the full-vocabulary
    // normaliser cancels, so only the K gathered logits enter
    float zm = kNegInf, tm = kNegInf;
    for (int i = lane; i < K; i += 64) {
      zm = fmaxf(zm, c.z[i]);
      tm = fmaxf(tm, c.t[i]);
    }
    zm = wave_max(zm);
    tm = wave_max(tm);
    float sz = 0.f, st = 0.f;
    for (int i = lane; i < K; i += 64) {
      sz += expf(c.z[i] - zm);
      st += expf(c.t[i] - tm);
    }
    const float lse_s = zm + logf(wave_sum(sz));
    const float lse_t = tm + logf(wave_sum(st));
    float part = 0.f;
    for (int i = lane; i < K; i += 64) {
      const float lpt = c.z[i] - lse_s, lqt = c.t[i] - lse_t;
      part += EST == FKL_TOPK ? expf(lqt) * (lqt - lpt) : expf(lpt) * (lpt - lqt);
    }
    const float kl = wave_sum(part);
    for (int i = lane; i < K; i += 64) {
      const float lpt = c.z[i] - lse_s, lqt = c.t[i] - lse_t;
      const float pt = expf(lpt), qt = expf(lqt);
      c.w[i] = EST == FKL_TOPK ? gmu * (pt - qt) : gmu * pt * ((lpt - lqt) - kl);
    }
    if (lane == 0) c.C = 0.f;
    return kl;
  }
}

// Wave 0: the filter bits, and the entries sorted by (vector, index) in
// skey (a rank sort: entry i goes to the number of keys below its own; the
// keys are distinct, and an id outside [0, V) sorts last).
template <int EPV>
__device__ __forceinline__ void set_filter(int K, CacheLds& c) {
  const int lane = threadIdx.x & 63;
  auto key = [&](int i) {
    const int id = c.id[i];
    const uint32_t v = id >= 0 ? (uint32_t)id / (uint32_t)EPV : 0xFFFFFFFFu;
    return ((uint64_t)v << 32) | (uint32_t)i;
  };
  for (int i = lane; i < K; i += 64) {
    const int id = c.id[i];
    if (id >= 0) {
      const int v = id / EPV;
      atomicOr(&c.filter[(v & (kFilterBits - 1)) >> 5], 1u << (v & 31));
    }
  }
  // the keys by entry index, then each group of 64 ranked against all K and
  // written to its place in skey
  for (int i = lane; i < K; i += 64) c.ukey[i] = key(i);
#pragma unroll 1
  for (int i0 = 0; i0 < K; i0 += 64) {  // wave-uniform
    const uint64_t ki = i0 + lane < K ? c.ukey[i0 + lane] : ~0ull;
    int r = 0;
#pragma unroll 4
    for (int j = 0; j < K; ++j) r += c.ukey[j] < ki ? 1 : 0;
    if (i0 + lane < K) c.skey[r] = ki;
  }
}

// Add the spikes that fall inside vector v, in ascending cache order: a
// binary search of skey for v's first entry, then v's run.
template <int EPV, class IdxT>
__device__ __forceinline__ void apply_spikes(IdxT v, float (&g)[EPV], int K, const CacheLds& c) {
  const uint32_t word = c.filter[(v & (kFilterBits - 1)) >> 5];
  if ((word >> (v & 31)) & 1u) {
    const uint64_t lo = (uint64_t)(uint32_t)v << 32;
    int a = 0, b = K;
    while (a < b) {
      const int mid = (a + b) >> 1;
      if (c.skey[mid] < lo) a = mid + 1;
      else b = mid;
    }
    const int64_t base = (int64_t)v * EPV;
    for (; a < K && (c.skey[a] >> 32) == (uint64_t)(uint32_t)v; ++a) {
      const int i = (int)(uint32_t)c.skey[a];
      const int64_t off = (int64_t)c.id[i] - base;
      const float w = c.w[i];
#pragma unroll
      for (int e = 0; e < EPV; ++e)
        if (off == e) g[e] += w;
    }
  }
}

// Exact spike map of a resident row: bit s of spk[s >> 5][lane] is set when
// the vector that lane holds in register slot s carries a spike, and bit i
// of ent[s] (K bits) when cache entry i falls in slot s.  Wave 0 marks the K
// cached ids after the estimator has run; sweep 2 then tests one bit per
// slot instead of looking every vector up, and a vector with a spike visits
// only its slot's entries.
constexpr int kEntWords = kKMax / 64;
template <int NT>
__device__ __forceinline__ void mark_spike_slots(int K, uint32_t nvec, const CacheLds& c,
                                                 uint32_t (*spk)[NT],
                                                 uint64_t (*ent)[kEntWords]) {
  const uint32_t full = nvec / NT;  // slots that are not moved back
  for (int i = threadIdx.x & 63; i < K; i += 64) {
    const int id = c.id[i];
    if (id < 0) continue;
    const uint32_t v = (uint32_t)id / 4u;
    const uint32_t s = v < full * NT ? v / NT : full;
    const uint32_t lane = v - slot_base<NT>((int)s, nvec);
    atomicOr(&spk[s >> 5][lane], 1u << (s & 31));
    atomicOr(&ent[s][i >> 6], 1ull << (i & 63));
  }
}

// Add the spikes that fall inside vector v (a vector known to hold at least
// one), in ascending cache order: the entries of v's slot (ent, the same for
// every lane of the wave), lowest index first.
template <int EPV>
__device__ __forceinline__ void add_spikes(uint32_t v, float (&g)[EPV], int K,
                                           const uint64_t* ent, const CacheLds& c) {
  const int base = (int)(v * EPV);
#pragma unroll 1
  for (int wd = 0; wd < ((K + 63) >> 6); ++wd) {
    uint64_t m = ent[wd];
    m = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(m >> 32)) << 32) |
        (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)m);
#pragma unroll 1
    while (m != 0ull) {
      const int i = wd * 64 + __builtin_ctzll(m);
      m &= m - 1ull;
      const uint32_t off = (uint32_t)(c.id[i] - base);
      if (off < (uint32_t)EPV) {
        const float w = c.w[i];
#pragma unroll
        for (int e = 0; e < EPV; ++e)
          if (off == (uint32_t)e) g[e] += w;
      }
    }
  }
}

// A masked token: zero its gradient vectors [v0, v1) (unless told to skip)
// and, if `writer`, its per-token outputs.
template <class TI, class TO, int NT>
__device__ void masked_row(const Args& a, int64_t row, void* grow, int64_t v0, int64_t v1,
                           bool writer) {
  constexpr int EPV = TI::EPV;
  if (!a.skip_masked) {
    float g[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) g[e] = 0.f;
    for (int64_t v = v0 + threadIdx.x; v < v1; v += NT)
      store_vec<TI, TO>(grow, v, g, v == a.nvec - 1 ? a.tail : EPV);
  }
  if (writer) {
    if (threadIdx.x == 0) {
      a.loss[row] = 0.f;
      if (a.lse_out) a.lse_out[row] = 0.f;
    }
    if (a.gathered_out)
      for (int i = threadIdx.x; i < a.K; i += NT) a.gathered_out[row * a.K + i] = 0.f;
    if (a.coverage_out && threadIdx.x < 2) a.coverage_out[2 * row + threadIdx.x] = 0.f;
  }
}

// Wave 0 after the statistics are known: estimator, spikes, per-token outputs.
template <class TI, int EST, bool FILTER = true>
__device__ __forceinline__ void finish_row(const Args& a, int64_t row, float L, bool writer,
                                           CacheLds& c) {
  const int lane = threadIdx.x & 63;
  const float loss = estimate<EST>(a.K, L, a.gamma, a.mc_variant, a.clip_eps, c);
  if constexpr (FILTER) set_filter<TI::EPV>(a.K, c);
  if (writer) {
    if (lane == 0) {
      a.loss[row] = c.bad ? __builtin_nanf("") : loss;
      if (a.lse_out) a.lse_out[row] = L;
    }
    if (a.gathered_out)
      for (int i = lane; i < a.K; i += 64) a.gathered_out[row * a.K + i] = c.z[i];
    if (a.coverage_out) {
      // support coverage (App. A.1's restricted normalisers): the student's
      // mass Z_p^S = sum_i exp(z_{a_i} - L) and the teacher's Z_q^S =
      // sum_i exp(tau_i) on the cached support
      float zp = 0.f, zq = 0.f;
      for (int i = lane; i < a.K; i += 64) {
        zp += expf(c.z[i] - L);
        zq += expf(c.t[i]);
      }
      zp = wave_sum(zp);
      zq = wave_sum(zq);
      if (lane == 0) {
        a.coverage_out[2 * row] = zp;
        a.coverage_out[2 * row + 1] = zq;
      }
    }
  }
}

// ---------------------------------------------------------------- row-per-workgroup kernels

// The row jitter of the row kernels: calls over at least kJitterMinRows rows
// (16 rounds of the 256 CUs).  Measured over 32,768 unmasked rows of
// V = 151,936 bf16 in k_row_resident: MC1 5.80 ms without, 5.23 ms with;
// twice the wait 5.37 ms, 0..15 x 1024 or 0..31 x 512 cycles 5.24-5.26 ms.
// k_row_dense_resident waits twice as long (its rows take longer): FKL and
// RKL over 16,384 rows 3.59 -> 3.51 ms (half the wait: 3.53 ms, three
// times: 3.54 ms).
constexpr int64_t kJitterMinRows = 4096;

// One 1024-lane workgroup per token row, the whole row held in registers
// between the sweeps (NSLOT 16-byte vectors per lane): HBM sees one read of
// the logits and one write of the gradient.  TAIL: V is not a multiple of
// the elements per vector, so the row's last vector is masked past V after
// its load and stored element by element.
template <class TI, class TO, int EST, int NSLOT, bool TAIL>
__global__ void __launch_bounds__(kRowThreads) k_row_resident(Args a) {
  constexpr int NT = kRowThreads, NW = NT / 64, EPV = TI::EPV;
  static_assert(!is_dense(EST), "dense estimators stream two rows");
  __shared__ float s_red[NW];
  __shared__ CacheLds c;
  __shared__ uint32_t s_spk[2][NT];
  __shared__ uint64_t s_ent[NSLOT][kEntWords];
  static_assert(NSLOT <= 64, "spike map holds 64 slots");
  const int tid = threadIdx.x;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  if (a.mask && a.mask[row] == 0) {
    masked_row<TI, TO, NT>(a, row, grow, 0, a.nvec, true);
    return;
  }
  s_spk[0][tid] = 0u;
  s_spk[1][tid] = 0u;
  for (int w = tid; w < NSLOT * kEntWords; w += NT) (&s_ent[0][0])[w] = 0ull;
  const uint32_t nvec = (uint32_t)a.nvec;  // <= NSLOT * NT
  const int K = a.K;
  // Every row takes nearly the same time, so the workgroups on all CUs
  // fall into step: they load together and store together, and HBM idles
  // between the bursts.  A wait of 0..7 x 2048 cycles, a hash of the row,
  // keeps them out of step.
  if (a.N >= kJitterMinRows) {
    const uint32_t n = ((uint32_t)row * 0x9E3779B1u) >> 29;
    for (uint32_t i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(32);
  }

  // The first 64 cache entries are requested before the row, so the
  // dependent gather below does not wait behind the whole row.
  int32_t id0 = 0;
  float t0 = 0.f, b0 = 0.f;
  if (tid < K && tid < 64) {
    id0 = a.ids[row * K + tid];
    t0 = a.tau[row * K + tid];
    if (a.beta) b0 = a.beta[row * K + tid];
  }

  typename TI::Vec x[NSLOT];
  {
    // Unconditional loads at a wave-uniform slot base plus one lane offset,
    // so the wait counts stay exact and one register addresses every slot.
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      const uint32_t b = slot_base<NT>(s, nvec);
      x[s] = ld_nt<TI>((const typename TI::Vec*)zrow + b, slot_off<NT>(s, b, tid, nvec));
    }
  }
  if (tid < 64) {
    int bad = 0;
    if (tid < K) {
      const bool ok = id0 >= 0 && (int64_t)id0 < a.V;
      c.id[tid] = ok ? id0 : -1;
      c.z[tid] = ok ? load_elem<TI>(zrow, id0) : __builtin_nanf("");
      c.t[tid] = t0;
      c.b[tid] = b0;
      bad = ok ? 0 : 1;
    }
    for (int i = tid + 64; i < K; i += 64) {
      const int32_t id = a.ids[row * K + i];
      const bool ok = id >= 0 && (int64_t)id < a.V;
      c.id[i] = ok ? id : -1;
      c.z[i] = ok ? load_elem<TI>(zrow, id) : __builtin_nanf("");
      c.t[i] = a.tau[row * K + i];
      c.b[i] = a.beta ? a.beta[row * K + i] : 0.f;
      bad |= ok ? 0 : 1;
    }
    bad = __any(bad);
    if (tid == 0) c.bad = bad;
  }

  float L;
  {
    // only a slot that reaches past the row end has lanes to mask (a
    // wave-uniform test, so full slots cost no lane work); in the slot that
    // holds the row's last vector, that vector's elements past V become -inf
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      if ((uint32_t)(s * NT + NT) > nvec && !slot_owns<NT>(s, slot_base<NT>(s, nvec), tid, nvec))
        x[s] = neg_inf_vec<TI>();
      if constexpr (TAIL)
        if ((uint32_t)s == (nvec - 1) / NT && slot_base<NT>(s, nvec) + (uint32_t)tid == nvec - 1)
          mask_tail<TI>(x[s], a.tail);
    }
    // sweep 1a: row max (EPV independent chains)
    float mx[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) mx[e] = kNegInf;
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      float f[EPV];
      unpack<TI>(x[s], f);
#pragma unroll
      for (int e = 0; e < EPV; ++e) mx[e] = fmaxf(mx[e], f[e]);
    }
    float m = mx[0];
#pragma unroll
    for (int e = 1; e < EPV; ++e) m = fmaxf(m, mx[e]);
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) keep_packed(x[s]);
    m = block_max<NW>(m, s_red);
    // sweep 1b: sum of exp(z - m) over the registers
    const float nm = -m * kLog2e;
    float sm[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) sm[e] = 0.f;
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      float f[EPV];
      unpack<TI>(x[s], f);
#pragma unroll
      for (int e = 0; e < EPV; ++e) sm[e] += fast_exp2(fmaf(f[e], kLog2e, nm));
    }
    float ssum = 0.f;
#pragma unroll
    for (int e = 0; e < EPV; ++e) ssum += sm[e];
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) keep_packed(x[s]);
    ssum = block_sum<NW>(ssum, s_red);
    L = m + logf(ssum);
  }

  if (tid < 64) {
    finish_row<TI, EST, false>(a, row, L, true, c);
    mark_spike_slots<NT>(K, nvec, c, s_spk, s_ent);
  }
  __syncthreads();
  // A row with an id outside [0, V) becomes NaN through its coefficient (MC:
  // C * p) or its fill value (top-k), with no per-element test.
  const bool bad = c.bad != 0;
  const float C = bad ? __builtin_nanf("") : c.C;
  const float g0 = bad ? __builtin_nanf("") : 0.f;
  const float nL = -L * kLog2e;

  // sweep 2: gradient row
  {
    const uint32_t nvec2 = fresh_s(nvec);
    const int tid2 = fresh_v(tid);
    const uint32_t spk_lo = s_spk[0][tid2], spk_hi = s_spk[1][tid2];
    auto grad_vec = [&](const typename TI::Vec& xs, int s, uint32_t b) {
      float g[EPV];
      if constexpr (is_mc(EST)) {
        float f[EPV];
        unpack<TI>(xs, f);
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = C * fast_exp2(fmaf(f[e], kLog2e, nL));
      } else {
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = g0;
      }
      if ((((s < 32 ? spk_lo : spk_hi) >> (s & 31)) & 1u) != 0u)
        add_spikes<EPV>(b + (uint32_t)tid2, g, K, s_ent[s], c);
      // (with TAIL the row's last vector stores its V - (nvec - 1) EPV
      // elements only)
      int valid = EPV;
      if constexpr (TAIL)
        valid = (uint32_t)(s * NT + NT) >= nvec2 && b + (uint32_t)tid2 == nvec2 - 1 ? a.tail : EPV;
      store_vec<TI, TO>((char*)grow + (size_t)b * EPV * TO::BYTES, (uint32_t)tid2, g, valid);
    };
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      if ((uint32_t)(s * NT + NT) <= nvec2) {  // a full slot: every lane owns its vector
        grad_vec(x[s], s, (uint32_t)(s * NT));
      } else {
        const uint32_t b = slot_base<NT>(s, nvec2);
        if (slot_owns<NT>(s, b, tid2, nvec2)) grad_vec(x[s], s, b);
      }
    }
  }
}

// Dense estimators, student row resident: one 1024-lane workgroup per row
// holds z in registers (as k_row_resident does) and streams the teacher row
// y twice, with cached loads.  256 rows in flight keep about 76 MB of
// teacher rows live, which fits the 256 MB Infinity Cache, so the second
// read of y can be served from there instead of HBM.
constexpr int kYAhead = 4;
constexpr int kXAhead = 8;
// offsets of the running sums are raised when an exponent (log2 units)
// exceeds this: terms stay below 2^24, sums of a row below 2^42
constexpr float kLazyRaise = 24.f;
// -offset * log2(e) before any value is seen: an offset of about -2.08e38,
// so a lane's first value above that raises it (a row whose every logit is
// below it reads as a row of -inf)
constexpr float kOffsetFloor = 3e38f;
// LDS that holds the first teacher slots between the sweeps, and the number
// of teacher slots after those that stay in registers: only the rest of the
// teacher row is read a second time.
constexpr int kYLdsBytes = 144 * 1024;
// Twelve registers per lane hold three bf16 slots (1.5 of fp32) with no
// spill in any variant; sixteen spill in the fp32 build.
constexpr int kYRegVgprs = 12;

template <class TI, class TO, int EST, int NSLOT, bool TAIL>
__global__ void __launch_bounds__(kRowThreads) k_row_dense_resident(Args a) {
  constexpr int NT = kRowThreads, NW = NT / 64, EPV = TI::EPV;
  typedef typename TI::Vec Vec;
  constexpr int YL_CAP = kYLdsBytes / (NT * (int)sizeof(Vec));
  constexpr int YL = YL_CAP < NSLOT ? YL_CAP : NSLOT;  // teacher slots kept in LDS
  // teacher slots kept in registers (after the LDS ones)
  constexpr int YR_WANT = kYRegVgprs / (int)(sizeof(Vec) / 4);
  constexpr int YR = YL + YR_WANT < NSLOT ? YR_WANT : NSLOT - YL;
  constexpr int YK = YL + YR;  // slots not read a second time
  __shared__ Stats s_st[NW];
  __shared__ Vec s_y[YL][NT];
  const int tid = threadIdx.x;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const void* yrow = (const char*)a.teacher + row * a.ld * TI::BYTES;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  if (a.mask && a.mask[row] == 0) {
    masked_row<TI, TO, NT>(a, row, grow, 0, a.nvec, true);
    return;
  }
  const uint32_t nvec = (uint32_t)a.nvec;  // <= NSLOT * NT
  // Every dense row costs the same, so the CUs would fall into step (see
  // k_row_resident): a wait of 0..7 x 4096 cycles, a hash of the row.
  if (a.N >= kJitterMinRows) {
    const uint32_t n = ((uint32_t)row * 0x9E3779B1u) >> 29;
    for (uint32_t i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(64);
  }
  // Slot s of a lane is vector s * NT + tid of the row, read and written
  // through the slot's buffer resource: past the row's last vector, loads
  // return zeros (replaced by -inf below) and gradient stores are dropped.
  constexpr uint32_t kSlotIn = NT * sizeof(Vec), kSlotOut = NT * EPV * TO::BYTES;
  const uint32_t in_bytes = nvec * (uint32_t)sizeof(Vec);
  auto z_slot = [&](int s) { return slot_rsrc(zrow, in_bytes, s * kSlotIn); };
  auto y_slot = [&](int s) { return slot_rsrc(yrow, in_bytes, s * kSlotIn); };
  auto g_slot = [&](int s) {
    return slot_rsrc(grow, nvec * (uint32_t)(EPV * TO::BYTES), s * kSlotOut);
  };
  // the large variant takes only rows longer than the small one holds, so its
  // first slots_small slots are always whole
  constexpr int DT = TI::BYTES == 2 ? BF16 : F32;
  constexpr int FULL = NSLOT == slots_large(DT) ? slots_small(DT) : 0;
  auto in_row = [](int s, int t, uint32_t nv) {
    return s < FULL || (uint32_t)(s * NT + t) < nv;
  };

  // sweep 1, one pass over both rows: per-lane sums of exp(z - oz) and
  // exp(y - oy) and the estimator's cross term, at offsets oz, oy that start
  // at a finite floor and are raised (with a rescale of the sums) only when
  // an exponent exceeds kLazyRaise: a wave-uniform branch, taken for the
  // first slot and rarely after.  The sums are exact at any offset; the
  // margin bounds each term by 2^kLazyRaise.  The student row fills its
  // registers kXAhead slots ahead of use and the teacher row streams through
  // a ring kYAhead slots deep, so the first slot starts as soon as its own
  // data has landed.  The scheduling barriers keep the loads in this order.
  Vec x[NSLOT];
  Vec yq[kYAhead];
  Vec yr[YR > 0 ? YR : 1];
  Stats st;
  {
    const uint32_t nvec1 = fresh_s(nvec);
    const int tid1 = fresh_v(tid);
    const uint32_t vo1 = fresh_v((uint32_t)tid * (uint32_t)sizeof(Vec));
#pragma unroll
    for (int j = 0; j < kXAhead && j < NSLOT; ++j) {
      x[j] = buf_ld<TI, kAuxNt>(z_slot(j), vo1);
      if (j < kYAhead) yq[j] = buf_ld<TI, 0>(y_slot(j), vo1);
    }
    // -offset * log2(e) of each row, from the floor
    float nz = kOffsetFloor, ny = kOffsetFloor;
    float sz = 0.f, sy = 0.f, tx = 0.f;  // tx: E_p[z - y] (reverse) or E_q[y - z] (forward)
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      if (s + kXAhead < NSLOT) x[s + kXAhead] = buf_ld<TI, kAuxNt>(z_slot(s + kXAhead), vo1);
      Vec yv = yq[s % kYAhead];
      if (s + kYAhead < NSLOT) yq[s % kYAhead] = buf_ld<TI, 0>(y_slot(s + kYAhead), vo1);
      if (s < YL) s_y[s][tid1] = yv;  // kept for sweep 2 (each lane reads back its own entry)
      else if (s < YK) yr[s - YL] = yv;
      if (!in_row(s, tid1, nvec1)) {
        x[s] = neg_inf_vec<TI>();
        yv = neg_inf_vec<TI>();
      }
      if constexpr (TAIL)
        if ((uint32_t)(s * NT + tid1) == nvec1 - 1) {  // the row's last vector, past V
          mask_tail<TI>(x[s], a.tail);
          mask_tail<TI>(yv, a.tail);
        }
      float fz[EPV], fy[EPV], az[EPV], ay[EPV];
      unpack<TI>(x[s], fz);
      unpack<TI>(yv, fy);
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        az[e] = fmaf(fz[e], kLog2e, nz);
        ay[e] = fmaf(fy[e], kLog2e, ny);
      }
      float hz = az[0], hy = ay[0];
#pragma unroll
      for (int e = 1; e < EPV; ++e) {
        hz = fmaxf(hz, az[e]);
        hy = fmaxf(hy, ay[e]);
      }
      if (__builtin_amdgcn_ballot_w64(hz > kLazyRaise || hy > kLazyRaise) != 0) {
        // raise each offset to the slot's maximum where that is higher
        float vz = fz[0], vy = fy[0];
#pragma unroll
        for (int e = 1; e < EPV; ++e) {
          vz = fmaxf(vz, fz[e]);
          vy = fmaxf(vy, fy[e]);
        }
        const float nz2 = fminf(nz, -vz * kLog2e), ny2 = fminf(ny, -vy * kLog2e);
        const float cz = fast_exp2(nz2 - nz), cy = fast_exp2(ny2 - ny);
        sz *= cz;
        sy *= cy;
        tx *= EST == RKL_DENSE ? cz : cy;
        nz = nz2;
        ny = ny2;
#pragma unroll
        for (int e = 0; e < EPV; ++e) {
          az[e] = fmaf(fz[e], kLog2e, nz);
          ay[e] = fmaf(fy[e], kLog2e, ny);
        }
      }
      // entries of zero weight (-inf, or an underflow) may have a NaN
      // difference d: the legacy multiply gives 0 * d = 0 for any d
#pragma unroll
      for (int e = 0; e < EPV; ++e) {
        const float pz = fast_exp2(az[e]);
        const float py = fast_exp2(ay[e]);
        const float d = fz[e] - fy[e];
        sz += pz;
        sy += py;
        if constexpr (EST == RKL_DENSE)
          tx += mul_zero_safe(pz, d);
        else
          tx -= mul_zero_safe(py, d);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // The offsets as values.  A lane that never left the floor reports -inf,
    // which the merge's rescale treats exactly; the opaque copy makes the
    // product a rounded value, so that the merge's offset differences are
    // exactly 0 where two offsets are equal (left to the compiler, the
    // product is fused into those differences and leaves its rounding error,
    // about 1e23 at the floor).
    constexpr float kLn2 = 0.6931471805599453f;
    const float oz = fresh_v(-nz * kLn2), oy = fresh_v(-ny * kLn2);
    st = Stats{nz == kOffsetFloor ? kNegInf : oz, sz, EST == RKL_DENSE ? tx : 0.f,
               ny == kOffsetFloor ? kNegInf : oy, sy, EST == RKL_DENSE ? 0.f : tx};
  }
  st = block_merge_tree<true, NW>(st, s_st);
  const DenseRow d = dense_row<EST>(st);
  if (tid == 0) {
    a.loss[row] = d.loss;
    if (a.lse_out) a.lse_out[row] = d.Lz;
  }

  // sweep 2: gradient from the resident z; y from LDS for the first YL slots,
  // a second read for the rest.  One copy per sign of gamma (a row-uniform
  // branch), so the sign costs no instruction per element.  Lanes past the
  // row's end compute values from -inf that their dropped stores discard.
  const DenseGrad k = dense_grad_consts(d, a.gamma);
  auto sweep2 = [&](auto neg) {
    constexpr bool NEG = decltype(neg)::value;
    const int tid2 = fresh_v(tid);
    const uint32_t vo2 = fresh_v((uint32_t)tid * (uint32_t)sizeof(Vec));
    const uint32_t vg2 = fresh_v((uint32_t)tid * (uint32_t)(EPV * TO::BYTES));
#pragma unroll
    for (int j = 0; j < kYAhead && YK + j < NSLOT; ++j)
      yq[j] = buf_ld<TI, 0>(y_slot(YK + j), vo2);
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      Vec yv;
      if (s < YL) {
        yv = s_y[s][tid2];
      } else if (s < YK) {
        yv = yr[s - YL];
      } else {
        yv = yq[(s - YK) % kYAhead];
        if (s + kYAhead < NSLOT)
          yq[(s - YK) % kYAhead] = buf_ld<TI, 0>(y_slot(s + kYAhead), vo2);
      }
      after(x[s], yv);
      float g[EPV];
      dense_grad<TI, EST, NEG>(x[s], yv, k, g);
      if (TAIL && (uint32_t)(s * NT + tid2) == nvec - 1)  // its first tail elements only
        store_vec<TI, TO>(grow, nvec - 1, g, a.tail);
      else
        buf_store<TO>(g_slot(s), vg2, g);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  if (k.neg)
    sweep2(std::true_type{});
  else
    sweep2(std::false_type{});
}

// Sweep-1 statistics of vectors [v0, v1) of a row, one lane's share
// (stride NT), with two loads in flight per step.
template <class TI, bool DENSE, int NT>
__device__ __forceinline__ Stats lane_stats(const void* zrow, const void* yrow, int64_t v0,
                                            int64_t v1, int64_t nvec, int tail) {
  constexpr int EPV = TI::EPV;
  Stats s = stats_empty();
  int64_t v = v0 + threadIdx.x;
  for (; v + NT < v1; v += 2 * NT) {
    typename TI::Vec z0 = ld_cached<TI>(zrow, v), z1 = ld_cached<TI>(zrow, v + NT);
    typename TI::Vec y0 = z0, y1 = z1;
    if constexpr (DENSE) {
      y0 = ld_cached<TI>(yrow, v);
      y1 = ld_cached<TI>(yrow, v + NT);
    }
    if (tail != EPV && v + NT == nvec - 1) {
      mask_tail<TI>(z1, tail);
      if constexpr (DENSE) mask_tail<TI>(y1, tail);
    }
    stats_add<TI, DENSE>(s, z0, y0);
    stats_add<TI, DENSE>(s, z1, y1);
  }
  if (v < v1) {
    typename TI::Vec z0 = ld_cached<TI>(zrow, v), y0 = z0;
    if constexpr (DENSE) y0 = ld_cached<TI>(yrow, v);
    if (tail != EPV && v == nvec - 1) {
      mask_tail<TI>(z0, tail);
      if constexpr (DENSE) mask_tail<TI>(y0, tail);
    }
    stats_add<TI, DENSE>(s, z0, y0);
  }
  return s;
}

// One 1024-lane workgroup per row, streaming: sweep 1 reads the row(s),
// sweep 2 reads them again (plain loads, so the second read can hit L2 or the
// Infinity Cache).  For rows wider than the registers hold, and for the dense
// estimators, which read two rows.
template <class TI, class TO, int EST>
__global__ void __launch_bounds__(kRowThreads) k_row_stream(Args a) {
  constexpr int NT = kRowThreads, NW = NT / 64, EPV = TI::EPV;
  constexpr bool DENSE = is_dense(EST);
  __shared__ Stats s_red[NW];
  __shared__ CacheLds c;
  const int tid = threadIdx.x;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const void* yrow = DENSE ? (const char*)a.teacher + row * a.ld * TI::BYTES : nullptr;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  if (a.mask && a.mask[row] == 0) {
    masked_row<TI, TO, NT>(a, row, grow, 0, a.nvec, true);
    return;
  }
  if constexpr (!DENSE) {
    for (int w = tid; w < kFilterWords; w += NT) c.filter[w] = 0u;
    if (tid < 64) load_cache<TI>(a, row, zrow, c);
  }
  Stats st = lane_stats<TI, DENSE, NT>(zrow, yrow, 0, a.nvec, a.nvec, a.tail);
  st = block_merge<DENSE, NW>(st, s_red);
  const float L = st.mz + logf(st.sz);

  if constexpr (DENSE) {
    const DenseRow d = dense_row<EST>(st);
    if (tid == 0) {
      a.loss[row] = d.loss;
      if (a.lse_out) a.lse_out[row] = d.Lz;
    }
    const DenseGrad dk = dense_grad_consts(d, a.gamma);
    for (int64_t v = tid; v < a.nvec; v += NT) {
      float g[EPV];
      dense_grad<TI, EST>(ld_cached<TI>(zrow, v), ld_cached<TI>(yrow, v), dk, g);
      store_vec<TI, TO>(grow, v, g, v == a.nvec - 1 ? a.tail : EPV);
    }
  } else {
    if (tid < 64) finish_row<TI, EST>(a, row, L, true, c);
    __syncthreads();
    const float C = c.C;
    const bool bad = c.bad != 0;
    const float nL = -L * kLog2e;
    for (int64_t v = tid; v < a.nvec; v += NT) {
      float g[EPV];
      if constexpr (is_mc(EST)) {
        float f[EPV];
        unpack<TI>(ld_cached<TI>(zrow, v), f);
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = C * fast_exp2(fmaf(f[e], kLog2e, nL));
      } else {
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = 0.f;
      }
      apply_spikes<EPV>(v, g, a.K, c);
      if (bad)
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = __builtin_nanf("");
      store_vec<TI, TO>(grow, v, g, v == a.nvec - 1 ? a.tail : EPV);
    }
  }
}

// ---------------------------------------------------------------- split-vocabulary kernels
// For small N a row is cut into P chunks of whole 16-byte vectors, one
// 256-lane workgroup each.  Pass 1 writes per-chunk statistics; pass 2
// merges the P records of its row in a fixed order (the same in every chunk
// of the row, so every chunk sees bit-identical row constants), repeats the
// K-entry estimator, and writes its chunk of the gradient.

template <class TI, bool DENSE>
__global__ void __launch_bounds__(kSplitThreads) k_split_stats(Args a) {
  constexpr int NT = kSplitThreads, NW = NT / 64;
  __shared__ Stats s_red[NW];
  const int64_t bi = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row = bi / a.P;
  const int chunk = (int)(bi % a.P);
  if (a.mask && a.mask[row] == 0) return;
  const int64_t v0 = (int64_t)chunk * a.chunk_vec;
  const int64_t v1 = v0 + a.chunk_vec < a.nvec ? v0 + a.chunk_vec : a.nvec;
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const void* yrow = DENSE ? (const char*)a.teacher + row * a.ld * TI::BYTES : nullptr;
  Stats st = lane_stats<TI, DENSE, NT>(zrow, yrow, v0, v1, a.nvec, a.tail);
  st = block_merge<DENSE, NW>(st, s_red);
  if (threadIdx.x == 0) {
    float* p = a.ws + ((size_t)row * a.P + chunk) * kPartialFloats;
    p[0] = st.mz; p[1] = st.sz; p[2] = st.tr;
    p[3] = st.my; p[4] = st.sy; p[5] = st.tf;
  }
}

template <class TI, class TO, int EST>
__global__ void __launch_bounds__(kSplitThreads) k_split_write(Args a) {
  constexpr int NT = kSplitThreads, EPV = TI::EPV;
  constexpr bool DENSE = is_dense(EST);
  __shared__ CacheLds c;
  __shared__ Stats s_row;
  const int tid = threadIdx.x;
  const int64_t bi = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t row = bi / a.P;
  const int chunk = (int)(bi % a.P);
  const int64_t v0 = (int64_t)chunk * a.chunk_vec;
  const int64_t v1 = v0 + a.chunk_vec < a.nvec ? v0 + a.chunk_vec : a.nvec;
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const void* yrow = DENSE ? (const char*)a.teacher + row * a.ld * TI::BYTES : nullptr;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  if (a.mask && a.mask[row] == 0) {
    masked_row<TI, TO, NT>(a, row, grow, v0, v1, chunk == 0);
    return;
  }
  if constexpr (!DENSE) {
    for (int w = tid; w < kFilterWords; w += NT) c.filter[w] = 0u;
  }
  if (tid < 64) {
    if constexpr (!DENSE) load_cache<TI>(a, row, zrow, c);
    Stats s = stats_empty();
    if (tid < a.P) {
      const float* p = a.ws + ((size_t)row * a.P + tid) * kPartialFloats;
      s = Stats{p[0], p[1], p[2], p[3], p[4], p[5]};
    }
    s = wave_merge<DENSE>(s);
    if (tid == 0) s_row = s;
  }
  __syncthreads();
  const Stats st = s_row;
  const float L = st.mz + logf(st.sz);
  if constexpr (DENSE) {
    const DenseRow d = dense_row<EST>(st);
    if (chunk == 0 && tid == 0) {
      a.loss[row] = d.loss;
      if (a.lse_out) a.lse_out[row] = d.Lz;
    }
    const DenseGrad dk = dense_grad_consts(d, a.gamma);
    for (int64_t v = v0 + tid; v < v1; v += NT) {
      float g[EPV];
      dense_grad<TI, EST>(ld_cached<TI>(zrow, v), ld_cached<TI>(yrow, v), dk, g);
      store_vec<TI, TO>(grow, v, g, v == a.nvec - 1 ? a.tail : EPV);
    }
  } else {
    if (tid < 64) finish_row<TI, EST>(a, row, L, chunk == 0, c);
    __syncthreads();
    const float C = c.C;
    const bool bad = c.bad != 0;
    const float nL = -L * kLog2e;
    for (int64_t v = v0 + tid; v < v1; v += NT) {
      float g[EPV];
      if constexpr (is_mc(EST)) {
        float f[EPV];
        unpack<TI>(ld_cached<TI>(zrow, v), f);
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = C * fast_exp2(fmaf(f[e], kLog2e, nL));
      } else {
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = 0.f;
      }
      apply_spikes<EPV>(v, g, a.K, c);
      if (bad)
#pragma unroll
        for (int e = 0; e < EPV; ++e) g[e] = __builtin_nanf("");
      store_vec<TI, TO>(grow, v, g, v == a.nvec - 1 ? a.tail : EPV);
    }
  }
}

// ---------------------------------------------------------------- top-k write-only path
// Renormalised on S, the top-k gradient is zero off the cached support and
// does not depend on any other logit, so without lse_out nothing of the row
// is read.  The zeros are written by a one-shot grid of short workgroups,
// one 16-byte store per lane, each XCD filling one contiguous eighth of the
// grid: measured on MI355X at [8192, 151936] fp32, that pattern writes at
// about 6.7 TB/s, against about 5.7 TB/s for workgroups that each sweep a
// whole row (and 5.9 TB/s for the same grid placed round-robin over the
// XCDs by the dispatcher).  A second, small launch (one wavefront per
// row) evaluates the k-entry estimator and writes the loss and the support
// entries over the zeros; stream order puts it after the fill.
constexpr int kFillThreads = 1024;
constexpr int kSparseRowsPerBlock = 4;

// Workgroup b writes 16 KiB of zeros: chunk (b' % bpr) of row row0 + b' / bpr,
// with b' the XCD placement of b.
template <class TO>
__global__ void __launch_bounds__(kFillThreads) k_fill_zero(Args a, int64_t row0,
                                                            uint32_t blocks_per_row) {
  const uint32_t bi = xcd_eighths(blockIdx.x, gridDim.x);
  const int64_t row = row0 + bi / blocks_per_row;
  const uint32_t v = (bi % blocks_per_row) * kFillThreads + threadIdx.x;
  if (row >= a.N || (int64_t)v >= a.nvec) return;
  if (a.skip_masked && a.mask && a.mask[row] == 0) return;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  if ((int64_t)v == a.nvec - 1 && a.tail != 4) {
    const float g[4] = {0.f, 0.f, 0.f, 0.f};
    store_vec<InF32, TO>(grow, v, g, a.tail);
  } else if constexpr (TO::BYTES == 4) {
    __builtin_nontemporal_store(f32x4{0.f, 0.f, 0.f, 0.f}, (f32x4*)grow + v);
  } else {
    __builtin_nontemporal_store(u32x2{0u, 0u}, (u32x2*)grow + v);
  }
}

// Wave 0: the support entries of a row over its zeros.  Ids are distinct by
// precondition; should one repeat, its first occurrence writes the sum over
// its occurrences in cache order, so the result stays deterministic.
template <class TO>
__device__ __forceinline__ void write_support(void* grow, int K, const CacheLds& c) {
  const int lane = threadIdx.x & 63;
  for (int i = lane; i < K; i += 64) {
    const int id = c.id[i];
    bool first = true;
    for (int j = 0; j < i; ++j) first = first && c.id[j] != id;
    if (!first) continue;
    float g = 0.f;
    for (int j = i; j < K; ++j)
      if (c.id[j] == id) g += c.w[j];
    if constexpr (TO::BYTES == 4)
      ((float*)grow)[id] = g;
    else
      ((uint16_t*)grow)[id] = __builtin_bit_cast(uint16_t, (__bf16)g);
  }
}

// One value in every element of a gradient row of nvec vectors (the last
// holding tail elements), lanes striding by NT.
template <class TO, int NT>
__device__ __forceinline__ void fill_row(void* grow, int64_t nvec, int tail, float x) {
  const float g[4] = {x, x, x, x};
  for (int64_t v = threadIdx.x; v < nvec; v += NT) {
    if (v == nvec - 1 && tail != 4) {
      store_vec<InF32, TO>(grow, v, g, tail);
    } else if constexpr (TO::BYTES == 4) {
      __builtin_nontemporal_store(f32x4{x, x, x, x}, (f32x4*)grow + v);
    } else {
      const uint32_t h = pack_bf16x2(x, x);
      __builtin_nontemporal_store(u32x2{h, h}, (u32x2*)grow + v);
    }
  }
}

// The write-only top-k form in one launch, for calls whose gradient is
// small enough that a second launch costs more than the one-shot fill gains
// over a row per workgroup: the workgroup writes its row's zeros, wave 0
// meanwhile evaluates the estimator, and after a barrier (which waits for
// every store of the workgroup) wave 0 writes the support entries over the
// zeros, or every lane NaN over the row if its cache was bad.
template <class TI, class TO, int EST>
__global__ void __launch_bounds__(kFillThreads) k_topk_fused(Args a) {
  __shared__ CacheLds c;
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  const int K = a.K;
  const bool masked = a.mask && a.mask[row] == 0;
  if (!(masked && a.skip_masked)) fill_row<TO, kFillThreads>(grow, a.nvec, a.tail, 0.f);
  if (masked) {  // (workgroup-uniform, before any barrier)
    if (tid == 0) a.loss[row] = 0.f;
    if (a.gathered_out)
      for (int i = tid; i < K; i += kFillThreads) a.gathered_out[row * K + i] = 0.f;
    return;
  }
  if (tid < 64) {
    load_cache<TI>(a, row, zrow, c);
    const float loss = estimate<EST>(K, 0.f, a.gamma, 0, 0.f, c);
    if (tid == 0) a.loss[row] = c.bad ? __builtin_nanf("") : loss;
    if (a.gathered_out)
      for (int i = tid; i < K; i += 64) a.gathered_out[row * K + i] = c.z[i];
  }
  __syncthreads();
  if (c.bad)
    fill_row<TO, kFillThreads>(grow, a.nvec, a.tail, __builtin_nanf(""));
  else if (tid < 64)
    write_support<TO>(grow, K, c);
}

template <class TI, class TO, int EST>
__global__ void __launch_bounds__(64 * kSparseRowsPerBlock) k_topk_sparse(Args a) {
  __shared__ CacheLds cs[kSparseRowsPerBlock];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kSparseRowsPerBlock + w;
  if (row >= a.N) return;  // whole wavefront; no workgroup barrier below
  CacheLds& c = cs[w];
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  void* grow = (char*)a.dlogits + row * a.ld * TO::BYTES;
  const int K = a.K;
  if (a.mask && a.mask[row] == 0) {
    if (lane == 0) a.loss[row] = 0.f;
    if (a.gathered_out)
      for (int i = lane; i < K; i += 64) a.gathered_out[row * K + i] = 0.f;
    return;
  }
  // every LDS entry a lane reads below was written by that same lane
  load_cache<TI>(a, row, zrow, c);
  const float loss = estimate<EST>(K, 0.f, a.gamma, 0, 0.f, c);
  const bool bad = c.bad != 0;
  if (lane == 0) a.loss[row] = bad ? __builtin_nanf("") : loss;
  if (a.gathered_out)
    for (int i = lane; i < K; i += 64) a.gathered_out[row * K + i] = c.z[i];
  if (bad) {
    const float g[4] = {__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""),
                        __builtin_nanf("")};
    for (int64_t v = lane; v < a.nvec; v += 64)
      store_vec<InF32, TO>(grow, v, g, v == a.nvec - 1 ? a.tail : 4);
    return;
  }
  write_support<TO>(grow, K, c);
}

// ---------------------------------------------------------------- cache validation

__global__ void __launch_bounds__(256) k_validate(const int32_t* ids, const float* tau,
                                                  const float* beta, int64_t V, int K,
                                                  int check_dups, int32_t* violations) {
  __shared__ int32_t s_ids[kKMax];
  __shared__ int s_red[4];
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x;
  int bad = 0;
  for (int i = tid; i < K; i += 256) {
    const int32_t id = ids[row * K + i];
    s_ids[i] = id;
    bad += (id < 0 || (int64_t)id >= V) ? 1 : 0;
    bad += isfinite(tau[row * K + i]) ? 0 : 1;
    if (beta) bad += isfinite(beta[row * K + i]) ? 0 : 1;
  }
  __syncthreads();
  if (check_dups)
    for (int i = tid; i < K; i += 256)
      for (int j = i + 1; j < K; ++j) bad += s_ids[j] == s_ids[i] ? 1 : 0;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) bad += __shfl_xor(bad, o, 64);
  if ((tid & 63) == 0) s_red[tid >> 6] = bad;
  __syncthreads();
  if (tid == 0) {
    const int total = s_red[0] + s_red[1] + s_red[2] + s_red[3];
    if (total) atomicAdd(violations, total);
  }
}

// ---------------------------------------------------------------- dispatch

template <class TI, class TO, int EST>
hipError_t row_t(const Args& a, Path path, bool read, hipStream_t s) {
  const dim3 grid((unsigned)a.N), block(kRowThreads);
  if constexpr (is_dense(EST)) {
    if (a.tail != TI::EPV && path != Path::RowStream) {
      // a partial last vector (see k_row_resident's TAIL); the fp32 variant
      // would spill, so fp32 rows of that kind stream
      // (the large variant assumes its first slots_small slots whole, so
      // the path's own size class is kept)
      if constexpr (TI::BYTES == 2) {
        if (path == Path::RowResidentSmall)
          hipLaunchKernelGGL((k_row_dense_resident<TI, TO, EST, slots_small(BF16), true>), grid,
                             block, 0, s, a);
        else
          hipLaunchKernelGGL((k_row_dense_resident<TI, TO, EST, slots_large(BF16), true>), grid,
                             block, 0, s, a);
      } else {
        hipLaunchKernelGGL((k_row_stream<TI, TO, EST>), grid, block, 0, s, a);
      }
    } else if (path == Path::RowResidentSmall) {
      constexpr int NS = slots_small(TI::BYTES == 2 ? BF16 : F32);
      hipLaunchKernelGGL((k_row_dense_resident<TI, TO, EST, NS, false>), grid, block, 0, s, a);
    } else if (path == Path::RowResidentLarge) {
      constexpr int NS = slots_large(TI::BYTES == 2 ? BF16 : F32);
      hipLaunchKernelGGL((k_row_dense_resident<TI, TO, EST, NS, false>), grid, block, 0, s, a);
    } else {
      hipLaunchKernelGGL((k_row_stream<TI, TO, EST>), grid, block, 0, s, a);
    }
  } else {
    if (!read) {
      return hipErrorInvalidValue;  // the write-only top-k form runs launch_topk_sparse
    } else if (a.tail != TI::EPV && path != Path::RowStream) {
      // a partial last vector: the variant that masks and stores it element
      // by element (the others keep whole-vector code)
      constexpr int NS = slots_large(TI::BYTES == 2 ? BF16 : F32);
      hipLaunchKernelGGL((k_row_resident<TI, TO, EST, NS, true>), grid, block, 0, s, a);
    } else if (path == Path::RowResidentSmall) {
      constexpr int NS = slots_small(TI::BYTES == 2 ? BF16 : F32);
      hipLaunchKernelGGL((k_row_resident<TI, TO, EST, NS, false>), grid, block, 0, s, a);
    } else if (path == Path::RowResidentLarge) {
      constexpr int NS = slots_large(TI::BYTES == 2 ? BF16 : F32);
      hipLaunchKernelGGL((k_row_resident<TI, TO, EST, NS, false>), grid, block, 0, s, a);
    } else {
      hipLaunchKernelGGL((k_row_stream<TI, TO, EST>), grid, block, 0, s, a);
    }
  }
  return hipGetLastError();
}

template <class TI, class TO, int EST>
hipError_t split_t(const Args& a, bool read, hipStream_t s) {
  const dim3 grid((unsigned)(a.N * a.P)), block(kSplitThreads);
  if (!read) return hipErrorInvalidValue;  // the write-only top-k form runs launch_topk_sparse
  hipLaunchKernelGGL((k_split_stats<TI, is_dense(EST)>), grid, block, 0, s, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_split_write<TI, TO, EST>), grid, block, 0, s, a);
  return hipGetLastError();
}

template <class TI, class TO, class F>
hipError_t by_est(int est, F&& f) {
  switch (est) {
    case FKL_TOPK: return f.template operator()<TI, TO, FKL_TOPK>();
    case RKL_TOPK: return f.template operator()<TI, TO, RKL_TOPK>();
    case RKL_MC1:
    case RKL_MC: return f.template operator()<TI, TO, RKL_MC>();
    case FKL_DENSE: return f.template operator()<TI, TO, FKL_DENSE>();
    case RKL_DENSE: return f.template operator()<TI, TO, RKL_DENSE>();
  }
  return hipErrorInvalidValue;
}

template <class F>
hipError_t by_types(int est, int in_dt, int out_dt, F&& f) {
  if (in_dt == BF16)
    return out_dt == BF16 ? by_est<InBf16, OutBf16>(est, f) : by_est<InBf16, OutF32>(est, f);
  return out_dt == BF16 ? by_est<InF32, OutBf16>(est, f) : by_est<InF32, OutF32>(est, f);
}

// Calls whose gradient rows total at most this many bytes take k_topk_fused.
// Measured with fp32 gradients: one launch 0.019 ms against 0.022 ms for the
// two at 65.5 MB (512 x 32,000), the same time at 155 and 262 MB, and 0.124
// against 0.109 ms at 622 MB (1,024 x 151,936).
#ifndef OPD_FUSED_TOPK_MAX_BYTES
#define OPD_FUSED_TOPK_MAX_BYTES (128ll << 20)
#endif
constexpr int64_t kFusedTopkMaxBytes = OPD_FUSED_TOPK_MAX_BYTES;

template <class TI, class TO, int EST>
hipError_t topk_sparse_t(const Args& a, hipStream_t s) {
  if constexpr (is_topk(EST)) {
    if (a.N * a.nvec * 4 * TO::BYTES <= kFusedTopkMaxBytes) {
      hipLaunchKernelGGL((k_topk_fused<TI, TO, EST>), dim3((unsigned)a.N), dim3(kFillThreads), 0,
                         s, a);
      return hipGetLastError();
    }
    const int64_t bpr = (a.nvec + kFillThreads - 1) / kFillThreads;
    // row chunks keep every grid under 2^32 work-items
    const int64_t rows_per_launch = (int64_t)0xFFFFFFFFll / (bpr * kFillThreads);
    for (int64_t r0 = 0; r0 < a.N; r0 += rows_per_launch) {
      const int64_t n = a.N - r0 < rows_per_launch ? a.N - r0 : rows_per_launch;
      hipLaunchKernelGGL((k_fill_zero<TO>), dim3((unsigned)(n * bpr)), dim3(kFillThreads), 0, s, a,
                         r0, (uint32_t)bpr);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    const unsigned blocks = (unsigned)((a.N + kSparseRowsPerBlock - 1) / kSparseRowsPerBlock);
    hipLaunchKernelGGL((k_topk_sparse<TI, TO, EST>), dim3(blocks), dim3(64 * kSparseRowsPerBlock),
                       0, s, a);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_topk_sparse(const Args& a, int est, int in_dt, int out_dt, hipStream_t stream) {
  return by_types(est, in_dt, out_dt, [&]<class TI, class TO, int EST>() {
    return topk_sparse_t<TI, TO, EST>(a, stream);
  });
}

hipError_t launch_rowwise(const Args& a, int est, int in_dt, int out_dt, Path path, bool read_row,
                          hipStream_t stream) {
  return by_types(est, in_dt, out_dt, [&]<class TI, class TO, int EST>() {
    return row_t<TI, TO, EST>(a, path, read_row, stream);
  });
}

hipError_t launch_split(const Args& a, int est, int in_dt, int out_dt, bool read_row,
                        hipStream_t stream) {
  return by_types(est, in_dt, out_dt, [&]<class TI, class TO, int EST>() {
    return split_t<TI, TO, EST>(a, read_row, stream);
  });
}

hipError_t launch_validate(const int32_t* ids, const float* tau, const float* beta, int64_t N,
                           int64_t V, int K, int check_dups, int32_t* violations,
                           hipStream_t stream) {
  hipLaunchKernelGGL(k_validate, dim3((unsigned)N), dim3(256), 0, stream, ids, tau, beta, V, K,
                     check_dups, violations);
  return hipGetLastError();
}

}  // namespace opd
