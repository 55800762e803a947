// HIP kernels that build the teacher-score cache for gfx950 (MI355X).
//
// Sec. 4.1 splits the pipeline into Stage 1, where rollout draws actions
// from the stale student p_old and records their rollout-time
// log-probabilities (or keeps its top-k support), and Stage 2, where the
// teacher scores the cached actions.  Three row operations cover it:
//   sample  M draws from softmax(z) by inversion of its index-order CDF at
//           caller-supplied uniforms (rollout at temperature 1 with no top-p
//           or top-k truncation, App. B), plus log softmax(z) at the draws;
//   top-k   the k largest logits (descending, equal values by lower index),
//           plus log softmax(z) there;
//   score   log softmax(z) at given ids.
// One 1024-lane workgroup per token row.  A row that fits the registers
// (bf16 up to 155,648 entries, fp32 up to 77,824) is loaded once and kept
// there; wider rows are streamed.
#include <math.h>

#include <type_traits>

#include "opd_device.h"

namespace opd {
namespace {

constexpr int NT = kRowThreads;
constexpr int NW = NT / 64;
// ids_out[row * k] of a row the streamed top-k kernel leaves to the resident one
constexpr int32_t kTopkRedo = -2;

// ---------------------------------------------------------------- rows

// max of three fp32 values by the hardware instruction, without the quieting
// of signalling NaNs that fmaxf adds for inputs of unknown origin (where it
// is used, a NaN input is caught another way)
__device__ __forceinline__ float max3_raw(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}


// Elements [valid, 4) of a vector replaced by -inf, without branches (the
// masks depend only on the wave-uniform count).
template <class TI>
__device__ __forceinline__ typename TI::Vec tail_masked(typename TI::Vec x, int valid) {
  if constexpr (TI::BYTES == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const uint32_t keep = (2 * d < valid ? 0x0000FFFFu : 0u) | (2 * d + 1 < valid ? 0xFFFF0000u : 0u);
      x[d] = (x[d] & keep) | (0xFF80FF80u & ~keep);
    }
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d) x[d] = d < valid ? x[d] : 0xFF800000u;
  }
  return x;
}

// Resident row in the slot layout of the loss kernels.  Lanes outside the
// row, and elements of the last vector past V, read as -inf.
template <class TI, int NSLOT>
__device__ __forceinline__ void load_row(const void* zrow, uint32_t nvec, int tail, int tid,
                                         typename TI::Vec (&x)[NSLOT]) {
#pragma unroll
  for (int s = 0; s < NSLOT; ++s) {
    const uint32_t b = slot_base<NT>(s, nvec);
    x[s] = ld_nt<TI>((const typename TI::Vec*)zrow + b, slot_off<NT>(s, b, tid, nvec));
  }
#pragma unroll
  for (int s = 0; s < NSLOT; ++s)
    if ((uint32_t)(s * NT + NT) > nvec && !slot_owns<NT>(s, slot_base<NT>(s, nvec), tid, nvec))
      x[s] = neg_inf_vec<TI>();
  if (tail != TI::EPV) {
    // the one slot that owns the last vector (a wave-uniform test), and in
    // it the one lane that holds it
    const uint32_t vt = nvec - 1;
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      const uint32_t b = slot_base<NT>(s, nvec);
      if (vt >= b && vt < b + NT && vt >= (uint32_t)(s * NT) && (uint32_t)tid == vt - b)
        x[s] = tail_masked<TI>(x[s], tail);
    }
  }
}

// One vector of a streamed row, with the tail past V read as -inf.
template <class TI>
__device__ __forceinline__ typename TI::Vec load_vec(const void* zrow, uint32_t v, uint32_t nvec,
                                                     int tail) {
  const typename TI::Vec x = ld_cached<TI>(zrow, v);
  return v == nvec - 1 ? tail_masked<TI>(x, tail) : x;
}

// exp(z - m) with nm = -m log2(e): the one expression every pass uses, so a
// value recomputed later is bit-identical to the one summed earlier.
__device__ __forceinline__ float ez(float f, float nm) { return fast_exp2(fmaf(f, kLog2e, nm)); }

template <class TI, int NSLOT>
__device__ __forceinline__ float lane_max(const typename TI::Vec (&x)[NSLOT]) {
  float mx = kNegInf;
#pragma unroll
  for (int s = 0; s < NSLOT; ++s) {
    float f[4];
    unpack<TI>(x[s], f);
#pragma unroll
    for (int e = 0; e < 4; ++e) mx = fmaxf(mx, f[e]);
  }
  return mx;
}

template <class TI, int NSLOT>
__device__ __forceinline__ float lane_sumexp(const typename TI::Vec (&x)[NSLOT], float nm) {
  float sm = 0.f;
#pragma unroll
  for (int s = 0; s < NSLOT; ++s) {
    float f[4];
    unpack<TI>(x[s], f);
#pragma unroll
    for (int e = 0; e < 4; ++e) sm += ez(f[e], nm);
  }
  return sm;
}

// Sum of exp(z - m) over one vector, added left to right onto acc.
template <class TI>
__device__ __forceinline__ float vec_sumexp(const typename TI::Vec& x, float nm, float acc) {
  float f[4];
  unpack<TI>(x, f);
#pragma unroll
  for (int e = 0; e < 4; ++e) acc += ez(f[e], nm);
  return acc;
}

// Inclusive prefix sum over the 64 lanes of a wavefront (DPP row shifts,
// then the row broadcasts of lanes 15 and 31).
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ uint32_t block_add_u32(uint32_t v, uint32_t* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) r += red[w];
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------- sampling
// Draws by inversion of the index-order CDF of softmax(z) (Sec. 4.1, Stage 1:
// the rollout samples at temperature 1 with no top-p or top-k truncation,
// App. B): draw i is the first index whose cumulative probability exceeds
// u_i.  The CDF is evaluated in double precision, so a draw is the one exact
// arithmetic gives unless u_i lies within about 1e-14 of a cumulative value.
//
// One 256-lane workgroup per row, several per CU; the row is read once.  It
// is cut into at most 2048 chunks of CV = G * 128 consecutive vectors (G * 512
// elements; G = 1 up to V = 1,048,576).  The 16 lanes of one DPP row take one
// chunk in steps of 128 vectors, eight coalesced loads per lane per step
// (each instruction covers 16 consecutive vectors).  A chunk's record is its
// maximum m_q (fp32, exact) and s_q = sum exp(z - m_q) in double.  After the
// row, each record is scaled to the row maximum M (s'_q = s_q f_q, f_q =
// exp(m_q - M)), each thread sums a run of C consecutive chunks, and a block
// scan gives the run prefixes.  One wavefront per draw then finds the run
// (a ballot over the prefixes), the chunk (a wave scan of the run's records)
// and the element (wave scans over the chunk in index order, two vectors per
// lane, with the very terms the record summed).  Where rounding leaves no
// crossing at a level, the nearest entry of nonzero mass is taken, so a drawn
// id always has positive probability.
constexpr int kSmpThreads = 256;
constexpr int kSmpWaves = kSmpThreads / 64;
constexpr int kSmpLoads = 8;                   // loads per lane per step
constexpr int kSmpStepVecs = 16 * kSmpLoads;   // vectors per DPP-row step (128)
constexpr int kSmpMaxChunks = 2048;            // records per row

// exp(z - m) in double for a logit z <= m, table-driven (Tang, ACM TOMS
// 15(2), 1989): d = z - m (exact in double) = (n / 512) ln 2 + r with |r|
// at most about ln 2 / 1024, exp(d) = 2^(n >> 9) 2^((n & 511) / 512) exp(r),
// and exp(r) by a cubic: the interpolant of exp at the four Chebyshev nodes
// of [-1.002 ln 2 / 1024, 1.002 ln 2 / 1024], computed in 50-digit decimal
// arithmetic and rounded to double (within 1.2e-15 relative of exp there).
// d is first raised to at least -2000, which keeps the reduction in range
// (-inf and far negative terms come out as 0).  n = round(d 512 / ln 2)
// comes from one fused multiply-add onto 1.5 * 2^52, whose low word is then
// n and whose value less 1.5 * 2^52 is n as a double; ln 2 / 512 is split in
// the Cody-Waite way (the high part's 32 significant bits make n times it
// exact for |n| < 2^21).  2^(n >> 9) is applied by ldexp, which rounds
// through double's gradual underflow (a term below about 4.9e-324 of the
// chunk max is 0).  The clamp also turns a NaN d into 0: NaN logits and
// infinite maxima are caught by the chunk max instead (chunk_record), whose
// record is then NaN, and so the row undefined.
constexpr int kExpTab = 512;
constexpr int kExpTabBits = 9;
constexpr double kDeadArg = -2000.0;
constexpr double kInvStep = 738.6598609351493;             // 512 / ln 2
constexpr double kShift52 = 6755399441055744.0;            // 1.5 * 2^52
constexpr double kStepHi = 6.93147180369123816490e-01 / kExpTab;
constexpr double kStepLo = 1.90821492927058770002e-10 / kExpTab;
constexpr double kQ3 = 0.16666667050025266, kQ2 = 0.50000001916793,
                 kQ1 = 0.9999999999999998, kQ0 = 0.9999999999999989;

struct SmpLds {
  double s[kSmpMaxChunks];  // chunk sum at its max; then at the row max
  float m[kSmpMaxChunks];   // chunk max
  double p[kSmpThreads];    // inclusive prefix of the runs
  double tab[kExpTab];      // 2^(j / 512)
  double wt[kSmpWaves];
  float red[kSmpWaves];
};

// (c2 is kQ2, passed in a vector register: one instruction cannot read two
// scalar constants, and a register the caller holds is not re-materialised
// per call)
__device__ __forceinline__ double exp_reduced(double d, const double* tab, double c2) {
  d = fmax(d, kDeadArg);
  const double xs = fma(d, kInvStep, kShift52);
  const double nd = xs - kShift52;
  const int n = (int)(uint32_t)__builtin_bit_cast(uint64_t, xs);
  double r = fma(-nd, kStepHi, d);
  r = fma(-nd, kStepLo, r);
  double p = fma(r, kQ3, c2);
  p = fma(p, r, kQ1);
  p = fma(p, r, kQ0);
  return ldexp(tab[n & (kExpTab - 1)] * p, n >> kExpTabBits);
}

// kQ2 in a vector register (see exp_reduced)
__device__ __forceinline__ double c2_reg() {
  double c = kQ2;
  asm volatile("" : "+v"(c));
  return c;
}

// The term for one fp32 logit z against the chunk max (md, in double).  The
// single expression both the chunk records and the draws use, so the draws
// recompute bit for bit the terms the records summed.
__device__ __forceinline__ double term(float z, double md, const double* tab, double c2) {
  return exp_reduced((double)z - md, tab, c2);
}

// exp(x) for one double x <= 0 (the row-max scale of a chunk record)
__device__ __forceinline__ double exp_neg(double x, const double* tab) {
  return exp_reduced(x, tab, c2_reg());
}

// max that propagates NaN (IEEE 754-2019 maximum; v_maximum3_f32 on gfx950)
__device__ __forceinline__ float max_nan(float a, float b) {
  return __builtin_elementwise_maximum(a, b);
}
__device__ __forceinline__ float max3_nan(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

// max over the 16 lanes of a DPP row, in every lane of the row (NaN if any
// lane holds NaN)
__device__ __forceinline__ float row16_max(float x) {
  x = max_nan(x, dpp_move<0x140>(x));  // row_mirror
  x = max_nan(x, dpp_move<0x141>(x));  // row_half_mirror
  x = max_nan(x, dpp_move<0xB1>(x));   // quad_perm [1,0,3,2]
  x = max_nan(x, dpp_move<0x4E>(x));   // quad_perm [2,3,0,1]
  return x;
}
// a double moved across lanes by one DPP pattern (both halves)
template <int CTRL>
__device__ __forceinline__ double dpp_move_f64(double v) {
  u32x2 h = __builtin_bit_cast(u32x2, v);
  h[0] = (uint32_t)__builtin_amdgcn_mov_dpp((int)h[0], CTRL, 0xF, 0xF, false);
  h[1] = (uint32_t)__builtin_amdgcn_mov_dpp((int)h[1], CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(double, h);
}
// sum over the 16 lanes of a DPP row, in every lane of the row: the same
// four patterns as row16_max; each step adds two values that every lane of a
// pair holds in swapped order, so all 16 lanes end with the same sum
__device__ __forceinline__ double row16_sum(double x) {
  x += dpp_move_f64<0x140>(x);  // row_mirror
  x += dpp_move_f64<0x141>(x);  // row_half_mirror
  x += dpp_move_f64<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp_move_f64<0x4E>(x);   // quad_perm [2,3,0,1]
  return x;
}
// inclusive prefix sum over the 64 lanes of a wavefront, in double
__device__ __forceinline__ double wave_incl_scan_f64(double x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(x, o, 64);
    if (lane >= o) x += t;
  }
  return x;
}

__device__ __forceinline__ int first_lane(uint64_t b) { return b ? __ffsll((long long)b) - 1 : -1; }
__device__ __forceinline__ int last_lane(uint64_t b) { return b ? 63 - __clzll((long long)b) : -1; }

enum Pick : int { kCross = 0, kFirst = 1, kLast = 2 };

// First (or last) chunk in [lo, hi) with positive mass, by wave ballots; -1 if none.
__device__ __forceinline__ int64_t chunk_positive(const SmpLds& c, int64_t lo, int64_t hi,
                                                  bool last) {
  const int lane = threadIdx.x & 63;
  if (!last) {
    for (int64_t b = lo; b < hi; b += 64) {
      const int64_t q = b + lane;
      const int f = first_lane(__ballot(q < hi && c.s[q] > 0.0));
      if (f >= 0) return b + f;
    }
  } else {
    for (int64_t b = hi; b > lo; b -= 64) {
      const int64_t q = b - 64 + lane;
      const int l = last_lane(__ballot(q >= lo && q < b && c.s[q] > 0.0));
      if (l >= 0) return b - 64 + l;
    }
  }
  return -1;
}

// The eight terms of this lane's two vectors of the 128-vector step that
// starts at vector v0 (vectors at or past the chunk end c1 give 0).
template <class TI>
__device__ __forceinline__ void step_terms(const void* zrow, uint32_t v0, uint32_t c1,
                                           uint32_t nvec, int tail, float mq, const double* tab,
                                           double (&w)[8]) {
  const double md = (double)mq, c2 = c2_reg();
  const uint32_t v = v0 + 2u * (uint32_t)(threadIdx.x & 63);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const bool in = v + h < c1;  // inside the chunk (and so the row)
    float f[4];
    unpack<TI>(in ? load_vec<TI>(zrow, v + h, nvec, tail) : neg_inf_vec<TI>(), f);
#pragma unroll
    for (int e = 0; e < 4; ++e) w[4 * h + e] = in ? term(f[e], md, tab, c2) : 0.0;
  }
}

// One draw by one wavefront (the result is wave-uniform): the first element
// whose cumulative mass exceeds t = u * S.
template <class TI>
__device__ int64_t smp_draw(const SmpLds& c, const void* zrow, uint32_t nvec, int tail,
                            uint32_t CV, uint32_t nchunk, uint32_t C, double t, double S,
                            double Md) {
  const int lane = threadIdx.x & 63;
  int64_t q = -1;
  double r = 0.0;
  int pick = kLast;
  if (t < S) {
    // run: the first i with p[i] > t (each lane looks at 4 entries)
    int li = -1;
#pragma unroll
    for (int k = 3; k >= 0; --k)
      if (c.p[4 * lane + k] > t) li = 4 * lane + k;
    const int fl = first_lane(__ballot(li >= 0));
    const int i = __shfl(li, fl < 0 ? 0 : fl, 64);  // fl >= 0: p[255] = S > t
    r = fmax(t - (i ? c.p[i - 1] : 0.0), 0.0);
    // chunk within the run (C <= 8 chunks, one per lane)
    const uint32_t r0 = min((uint32_t)i * C, nchunk), r1 = min(r0 + C, nchunk);
    const uint32_t qq = r0 + (uint32_t)lane;
    const double sq = qq < r1 ? c.s[qq] : 0.0;
    const double incl = wave_incl_scan_f64(sq);
    const int cl = first_lane(__ballot(qq < r1 && incl > r));
    if (cl >= 0) {
      const double before = cl > 0 ? __shfl(incl, cl - 1, 64) : 0.0;
      q = r0 + cl;
      r = fmax(r - before, 0.0);
      pick = kCross;
    } else {
      const int ll = last_lane(__ballot(qq < r1 && sq > 0.0));
      if (ll >= 0) {
        q = r0 + ll;
      } else {
        q = chunk_positive(c, r1, nchunk, false);
        pick = kFirst;
        if (q < 0) {
          q = chunk_positive(c, 0, r0, true);
          pick = kLast;
        }
      }
    }
  } else {
    q = chunk_positive(c, 0, nchunk, true);
  }
  if (q < 0) return -1;  // no chunk of positive mass (excluded by S > 0)
  // element within chunk q, in steps of 128 vectors: lane l holds vectors
  // 2l and 2l + 1 of the step (elements 8l .. 8l + 7, in index order)
  const float mq = c.m[q];
  const double fq = exp_neg((double)mq - Md, c.tab);
  const uint32_t c0 = (uint32_t)q * CV, c1 = min(c0 + CV, nvec);
  if (pick == kCross) {
    double acc = 0.0;  // unscaled mass of the earlier steps
    for (uint32_t v0 = c0; v0 < c1; v0 += kSmpStepVecs) {
      double w[8];
      step_terms<TI>(zrow, v0, c1, nvec, tail, mq, c.tab, w);
      double lsum = 0.0;
#pragma unroll
      for (int e = 0; e < 8; ++e) lsum += w[e];
      const double incl = acc + wave_incl_scan_f64(lsum);
      const int vl = first_lane(__ballot(incl * fq > r));
      if (vl >= 0) {
        double cum = vl > 0 ? __shfl(incl, vl - 1, 64) : acc;
        int ec = -1;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          cum += w[e];
          if (ec < 0 && cum * fq > r) ec = e;
        }
        const int el = __shfl(ec, vl, 64);
        if (el >= 0) return ((int64_t)v0 + 2 * vl) * 4 + el;
        break;  // rounding: no element crossing in that lane
      }
      acc = __shfl(incl, 63, 64);
    }
    pick = kLast;  // rounding left no crossing: the last entry of mass
  }
  // first (or last) element of positive mass in the chunk
  const bool last = pick == kLast;
  const uint32_t nsteps = (c1 - c0 + kSmpStepVecs - 1) / kSmpStepVecs;
  for (uint32_t k = 0; k < nsteps; ++k) {
    const uint32_t v0 = c0 + (last ? nsteps - 1 - k : k) * kSmpStepVecs;
    double w[8];
    step_terms<TI>(zrow, v0, c1, nvec, tail, mq, c.tab, w);
    int ef = -1, eb = -1;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (w[e] > 0.0) {
        if (ef < 0) ef = e;
        eb = e;
      }
    const int vl = last ? last_lane(__ballot(eb >= 0)) : first_lane(__ballot(ef >= 0));
    if (vl >= 0) return ((int64_t)v0 + 2 * vl) * 4 + __shfl(last ? eb : ef, vl, 64);
  }
  return -1;
}

// The chunk pass of one DPP row over chunk q (vectors [q CV, q CV + CV)): the
// chunk max and the double sum of exp(z - max), in every lane of the row.
// WIDE (more than one step per chunk) takes a max pass and a term pass over
// the chunk; otherwise the step's eight vectors stay in registers, loaded
// through one buffer resource that starts at the wave's first chunk qw
// (wave-uniform): the lane offset is fixed and each load's step an
// immediate.  A q past the last chunk gives the record (-inf, 0).
template <class TI, bool WIDE>
__device__ __forceinline__ void chunk_record(const void* zrow, uint32_t q, uint32_t qw,
                                             uint32_t CV, uint32_t nvec, int tail,
                                             const double* tab, float& mq_out, double& sq_out) {
  typedef typename TI::Vec Vec;
  constexpr int R = kSmpLoads;
  const uint32_t rl = threadIdx.x & 15;
  const bool ragged = tail != TI::EPV;
  const uint32_t c0 = q * CV, c1 = min(c0 + CV, nvec);
  Vec x[R];
  // (unused when WIDE)
  const uint32_t wv = (uint32_t)__builtin_amdgcn_readfirstlane((int)(qw * CV));
  const Rsrc wr = slot_rsrc(zrow, nvec * (uint32_t)sizeof(Vec), wv * (uint32_t)sizeof(Vec));
  uint32_t loff = (c0 - wv + rl) * (uint32_t)sizeof(Vec);
  asm("" : "+v"(loff));  // (kept whole, so each load's step is its immediate offset)
  // all R loads are issued before any is used; lanes past the chunk, and
  // elements past V, then become -inf through per-dword selects
  auto load_step = [&](uint32_t s0) {
#pragma unroll
    for (int b = 0; b < R; ++b) {
      if constexpr (WIDE) {
        x[b] = ld_cached<TI>(zrow, min(s0 + rl + 16u * b, nvec - 1));
      } else {
        // (s0 is c0 here; lanes past the row read zeros, replaced below)
        x[b] = buf_ld<TI, kAuxNt>(wr, loff + 16u * (uint32_t)sizeof(Vec) * b);
      }
    }
    // (a step wholly inside the chunk and clear of a ragged last vector
    // needs no selects)
    if (!(s0 + kSmpStepVecs <= c1 && !(ragged && s0 + kSmpStepVecs >= nvec))) {
#pragma unroll
      for (int b = 0; b < R; ++b) {
        const uint32_t v = s0 + rl + 16u * b;
        const Vec t = tail_masked<TI>(x[b], tail);
        const Vec n = neg_inf_vec<TI>();
        const bool out = v >= c1, last = ragged && v == nvec - 1;
#pragma unroll
        for (int d = 0; d < (int)(sizeof(Vec) / 4); ++d)
          x[b][d] = out ? n[d] : (last ? t[d] : x[b][d]);
      }
    }
  };
  // (the max propagates NaN; a NaN or +inf chunk max makes the record NaN:
  // the row then has no distribution)
  auto step_max = [&]() {
    float lm = kNegInf;
#pragma unroll
    for (int b = 0; b < R; ++b) {
      float f[4];
      unpack<TI>(x[b], f);
      lm = max3_nan(max3_nan(lm, f[0], f[1]), f[2], f[3]);
    }
    return lm;
  };
  const double c2 = c2_reg();
  auto step_sum = [&](double md, double acc) {
#pragma unroll
    for (int b = 0; b < R; ++b) {
      float f[4];
      unpack<TI>(x[b], f);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc += term(f[e], md, tab, c2);
    }
    return acc;
  };
  float lm = kNegInf;
  if constexpr (!WIDE) {
    load_step(c0);
    lm = step_max();
  } else {
    for (uint32_t s0 = c0; s0 < c1; s0 += kSmpStepVecs) {
      load_step(s0);
      lm = max_nan(lm, step_max());
    }
  }
  const float mq = row16_max(lm);
  double ls = 0.0;
  if (mq != kNegInf) {  // an all -inf chunk has no mass
    const double md = (double)mq;
    if constexpr (!WIDE) {
      ls = step_sum(md, 0.0);
    } else {
      for (uint32_t s0 = c0; s0 < c1; s0 += kSmpStepVecs) {
        load_step(s0);
        ls = step_sum(md, ls);
      }
    }
  }
  const double sum = row16_sum(ls);
  mq_out = mq;
  sq_out = mq < __builtin_huge_valf() ? sum : __builtin_nan("");  // NaN or +inf max: NaN
}

template <class TI, bool WIDE>
__global__ void __launch_bounds__(kSmpThreads) k_sample(CacheArgs a) {
  constexpr int T = kSmpThreads, W = kSmpWaves;
  __shared__ SmpLds c;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const int M = a.K;
  if (a.mask && a.mask[row] == 0) {
    for (int i = tid; i < M; i += T) {
      a.ids_out[row * M + i] = 0;
      if (a.logp) a.logp[row * M + i] = 0.f;
    }
    if (tid == 0 && a.lse_out) a.lse_out[row] = 0.f;
    return;
  }
  for (int j = tid; j < kExpTab; j += kSmpThreads) c.tab[j] = exp2((double)j / kExpTab);
  __syncthreads();
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec;
  const uint32_t steps = (nvec + kSmpStepVecs - 1) / kSmpStepVecs;
  const uint32_t G = (steps + kSmpMaxChunks - 1) / kSmpMaxChunks;  // steps per chunk
  const uint32_t CV = G * kSmpStepVecs;
  const uint32_t nchunk = (nvec + CV - 1) / CV;  // <= kSmpMaxChunks

  // one pass over the row: DPP row k of wave w takes chunks 4 w + k,
  // 4 w + k + 4 W, ...
  const uint32_t rowk = (uint32_t)lane >> 4, rl = (uint32_t)lane & 15;
  float lmax = kNegInf;
  for (uint32_t q0 = 4u * w; q0 < nchunk; q0 += 4u * W) {  // wave-uniform
    const uint32_t q = q0 + rowk;
    float mq;
    double sq;
    chunk_record<TI, WIDE>(zrow, q, q0, CV, nvec, a.tail, c.tab, mq, sq);
    if (rl == 15 && q < nchunk) {
      c.m[q] = mq;
      c.s[q] = sq;
    }
    if (q < nchunk) lmax = max_nan(lmax, mq);
  }
  const float Mx = block_max<W>(lmax, c.red);  // ends with a barrier: records visible
  const double Md = (double)Mx;
  // records at the row max; runs of C consecutive chunks per thread
  const uint32_t C = (nchunk + T - 1) / T;
  {
    const uint32_t r0 = min((uint32_t)tid * C, nchunk), r1 = min(r0 + C, nchunk);
    double run = 0.0;
    for (uint32_t q = r0; q < r1; ++q) {
      const float mq = c.m[q];
      const double sq = mq == kNegInf ? 0.0 : c.s[q] * exp_neg((double)mq - Md, c.tab);
      // (a NaN record keeps S NaN: the row has no distribution)
      c.s[q] = sq;
      run += sq;
    }
    const double incl = wave_incl_scan_f64(run);
    if (lane == 63) c.wt[w] = incl;
    __syncthreads();
    double before = 0.0;
    for (int k = 0; k < w; ++k) before += c.wt[k];
    c.p[tid] = before + incl;
  }
  double S = 0.0;
#pragma unroll
  for (int k = 0; k < W; ++k) S += c.wt[k];  // equals p[T - 1] bit for bit
  __syncthreads();

  const double L = Md + log(S);
  if (tid == 0 && a.lse_out) a.lse_out[row] = (float)L;
  // a NaN or +inf logit, or a row of -inf, leaves S NaN or 0: no distribution
  const bool defined = S > 0.0 && S <= 1.7976931348623157e308;
  for (int i = w; i < M; i += W) {  // one draw per wavefront
    const float u = a.u[row * M + i];
    int32_t id = -1;
    float lp = __builtin_nanf("");
    if (defined && u >= 0.f && u < 1.f) {
      const int64_t j = smp_draw<TI>(c, zrow, nvec, a.tail, CV, nchunk, C, (double)u * S, S, Md);
      if (j >= 0) {
        id = (int32_t)j;
        lp = (float)((double)load_elem<TI>(zrow, j) - L);
      }
    }
    if (lane == 0) {
      a.ids_out[row * M + i] = id;
      if (a.logp) a.logp[row * M + i] = lp;
    }
  }
}

// ---------------------------------------------------------------- top-k

// Sort key: the IEEE-754 total order of the fp32 bits (bf16 widened), with
// -0 taken as +0.  Larger key = larger value.
__device__ __forceinline__ uint32_t order_key(uint32_t bits) {
  bits = bits == 0x80000000u ? 0u : bits;
  return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

__device__ __forceinline__ uint32_t shfl_xor_u32(uint32_t v, int m) {
  return (uint32_t)__shfl_xor((int)v, m, 64);
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = shfl_xor_u32((uint32_t)v, m), hi = shfl_xor_u32((uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

// Bitonic sort of one value per lane over the workgroup, descending: lane i
// ends with the i-th largest.  Exchanges within a wavefront use lane
// shuffles; wider ones go through LDS (two buffers, one barrier each).
// Only the first P lanes (P a power of two) take part; the others keep their
// values.
template <class T, int NTH = NT>
__device__ T block_sort_desc(T v, T (*buf)[NTH], int P = NTH) {
  const int tid = threadIdx.x;
  int ping = 0;
#pragma unroll 1
  for (int size = 2; size <= P; size <<= 1) {
#pragma unroll 1
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      T pv;
      if (stride >= 64) {
        buf[ping][tid] = v;
        __syncthreads();
        pv = buf[ping][tid ^ stride];
        ping ^= 1;
      } else if constexpr (sizeof(T) == 8) {
        pv = shfl_xor_u64(v, stride);
      } else {
        pv = shfl_xor_u32(v, stride);
      }
      const bool take_max = ((tid & size) == 0) == ((tid & stride) == 0);
      v = take_max ? (v > pv ? v : pv) : (v < pv ? v : pv);
    }
  }
  return v;
}

// Bitonic sort of one value per lane within a wavefront, descending.
__device__ __forceinline__ uint32_t wave_sort_desc(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const uint32_t pv = shfl_xor_u32(v, stride);
      const bool take_max = ((lane & size) == 0) == ((lane & stride) == 0);
      v = take_max ? max(v, pv) : min(v, pv);
    }
  }
  return v;
}

// Bitonic sort, descending, of P entries held in LDS (P a power of two).
__device__ void lds_sort_desc(uint64_t* s, uint32_t P) {
  for (uint32_t size = 2; size <= P; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      for (uint32_t i = threadIdx.x; i < P / 2; i += NT) {
        const uint32_t lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
        const uint64_t x = s[lo], y = s[hi];
        if ((lo & size) == 0 ? x < y : x > y) {
          s[lo] = y;
          s[hi] = x;
        }
      }
      __syncthreads();
    }
  }
}

struct TopkLds {
  uint64_t sbuf[2][NT];
  uint64_t cand[kTopkCand];
  uint32_t cnt;
  uint32_t wbound[NW];
  uint32_t ured[NW];
  float red[NW];
  Stats st[NW];
};

// Calls f(key, j) for every element j of the row this lane holds (the
// resident slots, or a streamed pass).  The resident registers pass through
// an empty barrier first, so keys are recomputed in each pass rather than
// kept live from an earlier one.
template <class TI, int NSLOT, class F>
__device__ __forceinline__ void each_key(typename TI::Vec (&x)[NSLOT > 0 ? NSLOT : 1],
                                         const void* zrow, uint32_t nvec, int64_t V, int tail,
                                         int tid, F&& f) {
  const uint32_t V32 = (uint32_t)V;
  if constexpr (NSLOT > 0) {
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) keep_packed(x[s]);
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      const uint32_t b = slot_base<NT>(s, nvec);
      if ((uint32_t)(s * NT + NT) <= nvec || slot_owns<NT>(s, b, tid, nvec)) {
        const uint32_t v = b + (uint32_t)tid;
        float fv[4];
        unpack<TI>(x[s], fv);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t j = v * 4u + (uint32_t)e;
          if (tail == TI::EPV || j < V32) f(order_key(__float_as_uint(fv[e])), j);
        }
      }
    }
  } else {
    for (uint32_t v = tid; v < nvec; v += NT) {
      float fv[4];
      unpack<TI>(ld_cached<TI>(zrow, v), fv);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t j = v * 4u + (uint32_t)e;
        if (j < V32) f(order_key(__float_as_uint(fv[e])), j);
      }
    }
  }
}

// One row (every return below is workgroup-uniform).
template <class TI, int NSLOT, bool LSE>
__device__ __forceinline__ void topk_row(const CacheArgs& a, int64_t row, TopkLds& sh) {
  const int tid = threadIdx.x;
  const int k = a.K;
  if (a.mask && a.mask[row] == 0) {
    for (int i = tid; i < k; i += NT) {
      a.ids_out[row * k + i] = 0;
      if (a.logp) a.logp[row * k + i] = 0.f;
    }
    if (tid == 0 && a.lse_out) a.lse_out[row] = 0.f;
    return;
  }
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec;
  const int64_t V = a.V;
  typename TI::Vec x[NSLOT > 0 ? NSLOT : 1];
  if constexpr (NSLOT > 0) load_row<TI, NSLOT>(zrow, nvec, a.tail, tid, x);

  // Each lane's largest value (NaN ignored), which also starts the
  // log-partition; a lane with no element reports -inf.
  float lmx = kNegInf, L = 0.f;
  if constexpr (NSLOT > 0) {
    lmx = lane_max<TI, NSLOT>(x);
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) keep_packed(x[s]);
    if constexpr (LSE) {
      const float m = block_max<NW>(lmx, sh.red);
      L = m + logf(block_sum<NW>(lane_sumexp<TI, NSLOT>(x, -m * kLog2e), sh.red));
#pragma unroll
      for (int s = 0; s < NSLOT; ++s) keep_packed(x[s]);
    }
  } else {
    if constexpr (LSE) {
      Stats st = stats_empty();
      for (uint32_t v = tid; v < nvec; v += NT) {
        const typename TI::Vec xv = load_vec<TI>(zrow, v, nvec, a.tail);
        stats_add<TI, false>(st, xv, xv);
      }
      lmx = st.mz;
      st = block_merge<false, NW>(st, sh.st);
      L = st.mz + logf(st.sz);
    } else {
      for (uint32_t v = tid; v < nvec; v += NT) {
        float f[4];
        unpack<TI>(load_vec<TI>(zrow, v, nvec, a.tail), f);
#pragma unroll
        for (int e = 0; e < 4; ++e) lmx = fmaxf(lmx, f[e]);
      }
    }
  }

  // A lower bound on the k-th largest key: in every wave, r = ceil(k / 16)
  // lanes hold a value at least that wave's r-th largest lane maximum, so
  // 16 r >= k elements are at least the smallest of those 16 values.  A lane
  // whose maximum overstates its elements (none, or only NaN) can only
  // lower the bound to -inf or below, where every element is collected.
  {
    const uint32_t lkey = (uint32_t)tid < nvec ? order_key(__float_as_uint(lmx)) : 0u;
    const uint32_t srt = wave_sort_desc(lkey);
    const int r = (k + NW - 1) / NW;
    const uint32_t wb = (uint32_t)__shfl((int)srt, r - 1, 64);
    if ((tid & 63) == 0) sh.wbound[tid >> 6] = wb;
    if (tid == 0) sh.cnt = 0u;
  }
  __syncthreads();
  uint32_t bound = sh.wbound[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) bound = min(bound, sh.wbound[w]);
  // Candidates: every element not below the bound's value, and every NaN
  // (!(v < b) holds for both); their exact keys decide the order.
  const float bval = key_value(bound);
  auto take = [&](float v, uint32_t j) {
    if (!(v < bval)) {
      const uint32_t pos = atomicAdd(&sh.cnt, 1u);
      if (pos < (uint32_t)kTopkCand)
        sh.cand[pos] = ((uint64_t)order_key(__float_as_uint(v)) << 32) | (0xFFFFFFFFu - j);
    }
  };
  if constexpr (NSLOT > 0) {
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      const uint32_t b = slot_base<NT>(s, nvec);
      if ((uint32_t)(s * NT + NT) <= nvec || slot_owns<NT>(s, b, tid, nvec)) {
        const uint32_t v = b + (uint32_t)tid;
        float f[4];
        unpack<TI>(x[s], f);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (a.tail == TI::EPV || v * 4u + e < (uint32_t)V) take(f[e], v * 4u + e);
      }
    }
  } else {
    for (uint32_t v = tid; v < nvec; v += NT) {
      float f[4];
      unpack<TI>(ld_cached<TI>(zrow, v), f);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (v * 4u + e < (uint32_t)V) take(f[e], v * 4u + e);
    }
  }
  __syncthreads();
  const uint32_t cnt = sh.cnt;

  uint64_t mine = 0;  // after sorting: this lane's rank in the support
  if (cnt >= (uint32_t)k && cnt <= (uint32_t)NT) {
    int P = 2;
    while (P < (int)cnt) P <<= 1;
    mine = block_sort_desc<uint64_t>(tid < (int)cnt ? sh.cand[tid] : 0ull, sh.sbuf, P);
  } else if (cnt >= (uint32_t)k && cnt <= (uint32_t)kTopkCand) {
    uint32_t P = NT;
    while (P < cnt) P <<= 1;
    for (uint32_t i = cnt + tid; i < P; i += NT) sh.cand[i] = 0ull;
    __syncthreads();
    lds_sort_desc(sh.cand, P);
    mine = sh.cand[tid];
  } else {
    // Too many candidates (a row with many equal large values): find the
    // k-th largest key th by bisection over key bits, then the need-th
    // lowest index among the elements equal to th, by counting passes.
    // These passes re-read the row from memory (a rare path; compact code).
    typename TI::Vec none[1];
    auto count = [&](auto&& pred) {
      uint32_t n = 0;
      each_key<TI, 0>(none, zrow, nvec, V, a.tail, tid, [&](uint32_t key, uint32_t j) { n += pred(key, j) ? 1u : 0u; });
      return block_add_u32(n, sh.ured);
    };
    uint32_t th = 0;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t t = th | (1u << bit);
      if (count([&](uint32_t key, uint32_t) { return key >= t; }) >= (uint32_t)k) th = t;
    }
    const uint32_t gt = th == 0xFFFFFFFFu ? 0u : count([&](uint32_t key, uint32_t) { return key > th; });
    const uint32_t need = (uint32_t)k - gt;
    uint32_t y = 0;
    for (int bit = 30; bit >= 0; --bit) {
      const uint32_t t = y | (1u << bit);
      if (count([&](uint32_t key, uint32_t j) { return key == th && j < t; }) < need) y = t;
    }
    if (tid == 0) sh.cnt = 0u;
    __syncthreads();
    each_key<TI, 0>(none, zrow, nvec, V, a.tail, tid, [&](uint32_t key, uint32_t j) {
      if (key > th || (key == th && j <= y)) {
        const uint32_t pos = atomicAdd(&sh.cnt, 1u);
        if (pos < (uint32_t)kTopkCand) sh.cand[pos] = ((uint64_t)key << 32) | (0xFFFFFFFFu - j);
      }
    });
    __syncthreads();
    mine = block_sort_desc<uint64_t>(tid < k ? sh.cand[tid] : 0ull, sh.sbuf);
  }

  if (tid < k) {
    const uint32_t j = 0xFFFFFFFFu - (uint32_t)mine;
    a.ids_out[row * k + tid] = (int32_t)j;
    if (a.logp) a.logp[row * k + tid] = key_value((uint32_t)(mine >> 32)) - L;
  }
  if (tid == 0 && a.lse_out) a.lse_out[row] = L;
}

// The top-k of a row per workgroup (register-resident for NSLOT > 0); and,
// after the streamed kernel, a short grid whose workgroups walk the rows and
// redo only those the streamed kernel marked (reading them from memory), so
// that the usual case, no marked row, costs a few hundred workgroups rather
// than one per row.
constexpr int kTopkRedoGroups = 512;
template <class TI, int NSLOT, bool LSE>
__global__ void __launch_bounds__(NT) k_topk(CacheArgs a) {
  __shared__ TopkLds sh;
  topk_row<TI, NSLOT, LSE>(a, xcd_remap(blockIdx.x, gridDim.x), sh);
}
template <class TI, int NSLOT, bool LSE>
__global__ void __launch_bounds__(NT) k_topk_redo(CacheArgs a) {
  __shared__ TopkLds sh;
  __shared__ uint32_t s_n;
  __shared__ int64_t s_rows[NT];
  const int64_t stride = (int64_t)gridDim.x;
  // the workgroup's rows are blockIdx.x + i * stride; a lane reads one row's
  // mark, so a batch of NT rows costs one round trip, and only the marked
  // rows are redone
  for (int64_t base = blockIdx.x; base < a.N; base += stride * NT) {  // workgroup-uniform
    if (threadIdx.x == 0) s_n = 0u;
    __syncthreads();
    const int64_t row = base + (int64_t)threadIdx.x * stride;
    if (row < a.N && a.ids_out[row * a.K] == kTopkRedo) s_rows[atomicAdd(&s_n, 1u)] = row;
    __syncthreads();
    const uint32_t n = s_n;
    for (uint32_t i = 0; i < n; ++i) {
      topk_row<TI, NSLOT, LSE>(a, s_rows[i], sh);
      __syncthreads();  // the next row's writes to LDS wait for this row's reads
    }
  }
}

// ---------------------------------------------------------------- top-k, streamed

// The top-k support of rows of at least 16,384 entries, for k <= 64, reads
// each row once: 256-lane workgroups with about 34 KiB of LDS, four per CU.
// Each lane keeps the running maximum of the values it has seen.  After each
// tile of 8 coalesced loads per lane, and before any of the tile's elements
// is kept, the wave recomputes the ceil(k / 4)-th largest of its 64 running
// maxima (a radix select over order keys with ballots, 16 key bits for bf16
// rows) and publishes it in LDS; the bound in use is the smallest of the
// four waves' published values (on a wave's first tile, the k-th largest of
// its own maxima), a lower bound on the row's k-th largest, and it only
// rises.  Only lanes whose tile maximum reaches the bound look at the tile
// again, vector by vector, and keep the elements at or above it in their
// own LDS slots: no cross-lane compaction in the stream.  The next tile's
// loads are issued before the current tile is processed.  Since no bound
// exceeded the row's k-th largest key, the slots hold every element at or
// above it; at the end the largest known bound filters them, and a block
// sort of those (at most 256) gives the support.  A row
// whose lane slots overflow (many equal large values), that leaves more
// than 256 candidates, or that holds a NaN is marked, and a second launch
// runs the resident kernel on the marked rows only.
constexpr int kTkThreads = 256;
constexpr int kTkWaves = kTkThreads / 64;
constexpr int kTkLoads = 8;    // vector loads per lane per tile
constexpr int kTkSlots = 16;   // candidate slots per lane (a power of two)
constexpr int kTkMaxK = 64;    // one running maximum per lane bounds k
constexpr int64_t kTkMinVec = 4096;

struct TkLds {
  uint64_t buf[kTkSlots][kTkThreads];  // lane-private candidates: (value bits, ~index)
  uint64_t sel[kTkThreads];            // survivors: (order key, ~index)
  uint32_t theta[kTkWaves];            // published wave bounds (order keys)
  uint32_t nsel;
  uint32_t over;
  Stats st[kTkWaves];
};

// The largest key t (low KEEP bits zero) with at least k of the wave's rk
// >= t: the k-th largest rk, rounded down to the key bits that vary.
template <int LOWBITS>
__device__ __forceinline__ uint32_t wave_kth_key(uint32_t rk, int k) {
  uint32_t t = 0;
#pragma unroll
  for (int bit = 31; bit >= LOWBITS; --bit) {
    const uint32_t c = t | (1u << bit);
    if ((uint32_t)__popcll(__ballot(rk >= c)) >= (uint32_t)k) t = c;
  }
  return t;
}

template <class TI, bool LSE>
__global__ void __launch_bounds__(kTkThreads) k_topk_stream(CacheArgs a) {
  constexpr int T = kTkThreads, W = kTkWaves, B = kTkLoads;
  // bf16 values widened to fp32 have 16 zero low bits, so their order keys
  // vary in the top 16 bits only (a negative value's low key bits are ones,
  // which a threshold with zero low bits still admits)
  constexpr int LOWBITS = TI::BYTES == 2 ? 16 : 0;
  typedef typename TI::Vec Vec;
  __shared__ TkLds sh;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const int k = a.K;  // <= kTkMaxK
  if (a.mask && a.mask[row] == 0) {
    for (int i = tid; i < k; i += T) {
      a.ids_out[row * k + i] = 0;
      if (a.logp) a.logp[row * k + i] = 0.f;
    }
    if (tid == 0 && a.lse_out) a.lse_out[row] = 0.f;
    return;
  }
  if (lane == 0) sh.theta[w] = 0u;
  if (tid == 0) {
    sh.nsel = 0u;
    sh.over = 0u;
  }
  __syncthreads();
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec;  // >= kTkMinVec: every wave's first tile is full
  const uint32_t V32 = (uint32_t)a.V;
  constexpr uint32_t TILE = 64u * B, STRIDE = W * TILE;
  // tiles wholly inside the row (and clear of a ragged last vector) take
  // the path without per-element checks
  const uint32_t nclean = a.tail == TI::EPV ? nvec : nvec - 1;
  const uint32_t nfull = nclean / TILE * TILE;
  float run = kNegInf;  // this lane's running maximum (NaN ignored)
  // The bound.  Each wave publishes the ceil(k / 4)-th largest of its 64
  // running maxima (as an order key): that many of its lanes have each seen
  // an element at least that large, so the smallest of the four published
  // values has k distinct elements at or above it and is a lower bound on
  // the row's k-th largest.  Published values only rise, so a stale read
  // is still a lower bound.
  const int kq = (k + W - 1) / W;
  uint32_t qown = 0;    // this wave's published value (wave-uniform)
  uint32_t theta = 0;   // the bound in use (wave-uniform)
  bool first = true;    // this wave's first tile
  uint32_t cnt = 0;     // this lane's candidates so far
  float m = kNegInf, sum = 0.f, chk = 0.f;

  // One tile of B vectors per lane at vector t0 (lane l holds t0 + 64 b + l).
  // Pass A, for every lane: the tile's maximum (and its share of the
  // log-partition); then the bound; then pass B, in the lanes whose tile
  // maximum reaches the bound only, the elements kept.  A NaN anywhere in
  // the row (and, when the log-partition is wanted, a lane that sees no
  // finite value) sends the row to the exact fallback, so the bound and the
  // comparisons here need only order the numbers.
  auto process = [&](const Vec (&x)[B], uint32_t t0, auto full_tag) {
    constexpr bool FULL = decltype(full_tag)::value;
    auto vals = [&](int b, float (&f)[4]) {
      unpack<TI>(x[b], f);
      if constexpr (!FULL) {
        const uint32_t v = t0 + 64u * b + lane;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!(v < nvec && v * 4u + e < V32)) f[e] = kNegInf;
      }
    };
    // the tile's maximum; with LSE (registers to spare) each vector's
    // maximum is also kept, so pass B skips vectors below the bound unread
    static_assert(B == 8, "the tile maximum below folds eight vectors");
    float vmx[B];
    float tmx = kNegInf;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float f[4];
      vals(b, f);
      if constexpr (LSE) {
        vmx[b] = max3_raw(max3_raw(f[0], f[1], f[2]), f[3], f[3]);
      } else {
        tmx = max3_raw(max3_raw(tmx, f[0], f[1]), f[2], f[3]);
        chk += (f[0] + f[1]) + (f[2] + f[3]);
      }
    }
    if constexpr (LSE)
      tmx = max3_raw(max3_raw(vmx[0], vmx[1], vmx[2]), max3_raw(vmx[3], vmx[4], vmx[5]),
                     max3_raw(vmx[6], vmx[7], vmx[7]));
    if constexpr (LSE) {
      const float mn = fmaxf(m, tmx);
      if (mn != kNegInf) {  // (a lane that never sees a finite value sends its row to the fallback)
        const float nm = -mn * kLog2e;
        float ex[B * 4];
#pragma unroll
        for (int b = 0; b < B; ++b) {
          float f[4];
          vals(b, f);
#pragma unroll
          for (int e = 0; e < 4; ++e) ex[4 * b + e] = fast_exp2(fmaf(f[e], kLog2e, nm));
        }
#pragma unroll
        for (int h = B * 2; h >= 1; h >>= 1)
#pragma unroll
          for (int i = 0; i < h; ++i) ex[i] += ex[i + h];
        sum = fmaf(sum, rescale(m, mn), ex[0]);  // NaN from a NaN element
        m = mn;
      }
    }
    run = fmaxf(run, tmx);
    // raise the bound before keeping any of the tile's elements
    const uint32_t rk = order_key(__float_as_uint(run));
    if ((uint32_t)__popcll(__ballot(rk > qown)) >= (uint32_t)kq) {  // wave-uniform
      qown = wave_kth_key<LOWBITS>(rk, kq);
      if (lane == 0) sh.theta[w] = qown;
    }
    if (first) {  // until the other waves have published: the k-th of this wave's maxima
      theta = wave_kth_key<LOWBITS>(rk, k);
      first = false;
    }
    uint32_t pub = sh.theta[0];
#pragma unroll
    for (int q = 1; q < W; ++q) pub = min(pub, sh.theta[q]);
    theta = max(theta, (uint32_t)__builtin_amdgcn_readfirstlane(pub));
    const float thf = key_value(theta);
    // for numbers, f >= thf exactly when order_key(f) >= theta (a bf16
    // bound's zero low key bits sit below every widened value's)
    if (__ballot(tmx >= thf) != 0) {  // wave-uniform
      // the lane's vectors whose maximum reaches the bound, one bit each
      uint32_t rm = 0u;
      if (tmx >= thf) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
          bool reach;
          if constexpr (LSE) {
            reach = vmx[b] >= thf;
          } else {
            Vec xv = x[b];
            keep_packed(xv);  // unpacked again here rather than held since pass A
            float f[4];
            unpack<TI>(xv, f);
            reach = max3_raw(max3_raw(f[0], f[1], f[2]), f[3], f[3]) >= thf;
          }
          rm |= reach ? 1u << b : 0u;
        }
      }
      // One reaching vector per lane per round, in index order within the
      // lane, for as many rounds as the busiest lane needs (usually one):
      // a body per vector position instead would run whenever any lane's
      // vector at that position reaches.
      while (__ballot(rm != 0u) != 0) {  // wave-uniform
        if (rm != 0u) {
          const int b = __builtin_ctz(rm);
          rm &= rm - 1u;
          Vec xv = x[0];
#pragma unroll
          for (int j = 1; j < B; ++j) xv = b == j ? x[j] : xv;
          keep_packed(xv);  // selected packed, then unpacked
          float f[4];
          unpack<TI>(xv, f);
          const uint32_t v = t0 + 64u * (uint32_t)b + lane;
          // each element is written to the lane's next free slot, which
          // only a kept element then claims (a lane that reaches the last
          // slot overflows, and its row goes to the fallback)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool keep = f[e] >= thf && (FULL || (v < nvec && v * 4u + e < V32));
            sh.buf[cnt & (kTkSlots - 1)][tid] =
                ((uint64_t)__float_as_uint(f[e]) << 32) | (0xFFFFFFFFu - (v * 4u + e));
            cnt += keep ? 1u : 0u;
          }
        }
      }
    }
  };
  // full tiles through a buffer resource that starts at the tile (scalar
  // arithmetic): the lane offset is fixed and each load's step an immediate
  const uint32_t loff = (uint32_t)lane * (uint32_t)sizeof(Vec);
  auto load = [&](Vec (&x)[B], uint32_t t0) {
    const uint64_t off = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)t0) * sizeof(Vec);
    const Rsrc r = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>((const char*)zrow + off), 0,
                                                     (int)(TILE * sizeof(Vec)), kRsrcWord3);
#pragma unroll
    for (int b = 0; b < B; ++b) {
      if constexpr (TI::BYTES == 2)
        x[b] = __builtin_amdgcn_raw_buffer_load_b64(r, (int)(loff + 64u * sizeof(Vec) * b), 0,
                                                    kAuxNt);
      else
        x[b] = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(loff + 64u * sizeof(Vec) * b), 0,
                                                     kAuxNt);
    }
  };
  typedef std::integral_constant<bool, true> Full;
  typedef std::integral_constant<bool, false> Partial;
  // the wave's full tiles, two buffers: the next tile's loads are in flight
  // while the current one is processed
  Vec xa[B], xb[B];
  uint32_t t0 = (uint32_t)w * TILE;
  if (t0 < nfull) {  // wave-uniform
    load(xa, t0);
    while (t0 + 2 * STRIDE < nfull) {
      load(xb, t0 + STRIDE);
      process(xa, t0, Full());
      load(xa, t0 + 2 * STRIDE);
      process(xb, t0 + STRIDE, Full());
      t0 += 2 * STRIDE;
    }
    if (t0 + STRIDE < nfull) {
      load(xb, t0 + STRIDE);
      process(xa, t0, Full());
      process(xb, t0 + STRIDE, Full());
      t0 += 2 * STRIDE;
    } else {
      process(xa, t0, Full());
      t0 += STRIDE;
    }
  }
  // the one tile that reaches past the clean vectors (the wave whose turn it is)
  if (t0 < nvec) {
#pragma unroll
    for (int b = 0; b < B; ++b) xa[b] = ld_nt<TI>(zrow, min(t0 + 64u * b + lane, nvec - 1));
    process(xa, t0, Partial());
  }
  bool nan_seen;
  if constexpr (LSE) nan_seen = sum != sum || m == kNegInf;
  else nan_seen = chk != chk;
  if (cnt >= (uint32_t)kTkSlots || nan_seen) sh.over = 1u;
  float L = 0.f;
  if constexpr (LSE) {
    Stats st = stats_empty();
    st.mz = m;
    st.sz = sum;
    st = block_merge<false, W>(st, sh.st);  // barriers: bounds and slots visible
    L = st.mz + logf(st.sz);
  } else {
    __syncthreads();
  }
  // every bound in use was at most the row's k-th largest key, so the slots
  // hold every element at or above it; the largest bound known filters them
  uint32_t tstar = sh.theta[0];
#pragma unroll
  for (int q = 1; q < W; ++q) tstar = min(tstar, sh.theta[q]);
  tstar = max(tstar, theta);
  const bool overflow = sh.over != 0u;
  if (!overflow) {
    for (uint32_t i = 0; i < cnt; ++i) {
      const uint64_t e = sh.buf[i][tid];  // (value bits, ~index)
      const uint32_t key = order_key((uint32_t)(e >> 32));
      if (key >= tstar) {
        const uint32_t pos = atomicAdd(&sh.nsel, 1u);
        if (pos < (uint32_t)T) sh.sel[pos] = ((uint64_t)key << 32) | (uint32_t)e;
      }
    }
  }
  __syncthreads();
  const uint32_t nsel = sh.nsel;
  if (overflow || nsel > (uint32_t)T || nsel < (uint32_t)k) {  // workgroup-uniform
    if (tid == 0) a.ids_out[row * k] = kTopkRedo;
    return;
  }
  // Each survivor's rank is the number of survivors above it (the entries
  // are distinct); the k of rank below k are the top k, each written at its
  // rank.  Every lane reads the same entry at a time (an LDS broadcast), and
  // the reads do not depend on each other, unlike the exchanges of a sort.
  if (tid < (int)nsel) {
    const uint64_t mine = sh.sel[tid];
    uint32_t rank = 0;
#pragma unroll 8
    for (uint32_t i = 0; i < nsel; ++i) rank += sh.sel[i] > mine ? 1u : 0u;
    if (rank < (uint32_t)k) {
      const uint32_t j = 0xFFFFFFFFu - (uint32_t)mine;
      a.ids_out[row * k + rank] = (int32_t)j;
      if (a.logp) a.logp[row * k + rank] = key_value((uint32_t)(mine >> 32)) - L;
    }
  }
  if (tid == 0 && a.lse_out) a.lse_out[row] = L;
}

// ---------------------------------------------------------------- scoring

// Scoring reads each row once and writes a handful of values, so it is
// organised for overlap rather than residency: 256-lane workgroups with a
// small register footprint (several per CU), each lane loading batches of
// kScoreBatch vectors and folding them into a running (max, sum-exp) with
// one rescale per batch.
constexpr int kScoreThreads = 256;
constexpr int kScoreBatch = 8;

template <class TI>
__global__ void __launch_bounds__(kScoreThreads) k_score(CacheArgs a) {
  constexpr int T = kScoreThreads, W = T / 64, B = kScoreBatch;
  typedef typename TI::Vec Vec;
  __shared__ Stats s_st[W];
  const int tid = threadIdx.x;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const int K = a.K;  // <= OPD_K_MAX == T: one id per lane
  if (a.mask && a.mask[row] == 0) {
    if (tid < K) a.logp[row * K + tid] = 0.f;
    if (tid == 0 && a.lse_out) a.lse_out[row] = 0.f;
    return;
  }
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec;
  const bool ragged = a.tail != TI::EPV;
  // the ids are requested before the row, so the gather does not wait behind it
  const int32_t id = tid < K ? a.ids[row * K + tid] : 0;
  float m = kNegInf, sum = 0.f;
  for (uint32_t v0 = 0; v0 < nvec; v0 += T * B) {
    Vec xb[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const uint32_t v = v0 + (uint32_t)(b * T + tid);
      xb[b] = ld_nt<TI>(zrow, min(v, nvec - 1));  // clamped: every lane loads
    }
    float f[B][4];
    float bm = kNegInf;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const uint32_t v = v0 + (uint32_t)(b * T + tid);
      Vec xv = xb[b];
      if (v >= nvec) xv = neg_inf_vec<TI>();
      else if (ragged && v == nvec - 1) xv = tail_masked<TI>(xv, a.tail);
      unpack<TI>(xv, f[b]);
#pragma unroll
      for (int e = 0; e < 4; ++e) bm = fmaxf(bm, f[b][e]);
    }
    const float mn = fmaxf(m, bm);
    if (mn != kNegInf) {
      float acc = sum * rescale(m, mn);
      const float nm = -mn * kLog2e;
#pragma unroll
      for (int b = 0; b < B; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc += ez(f[b][e], nm);
      sum = acc;
      m = mn;
    }
  }
  Stats st = stats_empty();
  st.mz = m;
  st.sz = sum;
  st = block_merge<false, W>(st, s_st);
  const float L = st.mz + logf(st.sz);
  if (tid < K) {
    const bool ok = id >= 0 && (int64_t)id < a.V;
    a.logp[row * K + tid] = ok ? load_elem<TI>(zrow, id) - L : __builtin_nanf("");
  }
  if (tid == 0 && a.lse_out) a.lse_out[row] = L;
}

// ---------------------------------------------------------------- dispatch

template <class TI, int NSLOT>
hipError_t launch_op(const CacheArgs& a, CacheOp op, hipStream_t stream) {
  const dim3 grid((unsigned)a.N), block(NT);
  const dim3 rgrid((unsigned)min(a.N, (int64_t)kTopkRedoGroups));
  switch (op) {
    case CacheOp::Sample:
      break;
    case CacheOp::Topk:
      if constexpr (NSLOT == 0) {
        if (a.redo) {
          if (a.logp || a.lse_out)
            hipLaunchKernelGGL((k_topk_redo<TI, 0, true>), rgrid, block, 0, stream, a);
          else
            hipLaunchKernelGGL((k_topk_redo<TI, 0, false>), rgrid, block, 0, stream, a);
          break;
        }
      }
      if (a.logp || a.lse_out) {
        hipLaunchKernelGGL((k_topk<TI, NSLOT, true>), grid, block, 0, stream, a);
      } else {
        hipLaunchKernelGGL((k_topk<TI, NSLOT, false>), grid, block, 0, stream, a);
      }
      break;
    case CacheOp::Score:
      break;
  }
  return hipGetLastError();
}

template <class TI>
hipError_t launch_dt(const CacheArgs& a, CacheOp op, bool resident, hipStream_t stream) {
  if (op == CacheOp::Sample) {
    // more than one 128-vector step per chunk above 2048 steps per row
    if ((a.nvec + kSmpStepVecs - 1) / kSmpStepVecs <= (int64_t)kSmpMaxChunks)
      hipLaunchKernelGGL((k_sample<TI, false>), dim3((unsigned)a.N), dim3(kSmpThreads), 0,
                         stream, a);
    else
      hipLaunchKernelGGL((k_sample<TI, true>), dim3((unsigned)a.N), dim3(kSmpThreads), 0,
                         stream, a);
    return hipGetLastError();
  }
  if (op == CacheOp::Score) {
    hipLaunchKernelGGL((k_score<TI>), dim3((unsigned)a.N), dim3(kScoreThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (op == CacheOp::Topk && a.K <= kTkMaxK && a.nvec >= kTkMinVec) {
    if (a.logp || a.lse_out)
      hipLaunchKernelGGL((k_topk_stream<TI, true>), dim3((unsigned)a.N), dim3(kTkThreads), 0,
                         stream, a);
    else
      hipLaunchKernelGGL((k_topk_stream<TI, false>), dim3((unsigned)a.N), dim3(kTkThreads), 0,
                         stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    CacheArgs b = a;
    b.redo = 1;  // the rows the streamed kernel left (rare: re-read, not held in registers)
    return launch_op<TI, 0>(b, op, stream);
  }
  if (!resident) return launch_op<TI, 0>(a, op, stream);
  constexpr int big = TI::BYTES == 2 ? 38 : 19, small = TI::BYTES == 2 ? 16 : 8;
  if (a.nvec <= (int64_t)small * NT) return launch_op<TI, small>(a, op, stream);
  return launch_op<TI, big>(a, op, stream);
}

}  // namespace

hipError_t launch_cache(const CacheArgs& a, CacheOp op, int in_dt, bool resident,
                        hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  return in_dt == BF16 ? launch_dt<InBf16>(a, op, resident, stream)
                       : launch_dt<InF32>(a, op, resident, stream);
}

}  // namespace opd
