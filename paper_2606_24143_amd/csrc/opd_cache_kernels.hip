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

#include "opd_device.h"

namespace opd {
namespace {

constexpr int NT = kRowThreads;
constexpr int NW = NT / 64;
// ids_out[row * k] of a row the streamed top-k kernel leaves to the resident one
constexpr int32_t kTopkRedo = -2;

// ---------------------------------------------------------------- rows

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
__device__ __forceinline__ float wave_incl_scan(float x) {
  const int lane = threadIdx.x & 63, rl = lane & 15;
  float t;
  t = dpp_move<0x111>(x);  // row_shr:1
  if (rl >= 1) x += t;
  t = dpp_move<0x112>(x);  // row_shr:2
  if (rl >= 2) x += t;
  t = dpp_move<0x114>(x);  // row_shr:4
  if (rl >= 4) x += t;
  t = dpp_move<0x118>(x);  // row_shr:8
  if (rl >= 8) x += t;
  t = dpp_move<0x142>(x);  // row_bcast:15
  if ((lane & 31) >= 16) x += t;
  t = dpp_move<0x143>(x);  // row_bcast:31
  if (lane >= 32) x += t;
  return x;
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

// Chunk sums of exp(z - m) in index order (chunk = G consecutive vectors),
// the inclusive prefix of each thread's run of C consecutive chunks, and
// the wave totals of the runs.
struct CdfLds {
  float ls[kCdfChunks];
  float p[NT];
  float wt[NW];
  float red[NW];
};

enum Pick : int { kCross = 0, kFirst = 1, kLast = 2 };

__device__ __forceinline__ int64_t last_positive(const CdfLds& c, uint32_t lo, uint32_t hi) {
  for (uint32_t q = hi; q > lo; --q)
    if (c.ls[q - 1] > 0.f) return q - 1;
  return -1;
}
__device__ __forceinline__ int64_t first_positive(const CdfLds& c, uint32_t lo, uint32_t hi) {
  for (uint32_t q = lo; q < hi; ++q)
    if (c.ls[q] > 0.f) return q;
  return -1;
}

// One draw: the first element whose cumulative mass exceeds t, located run
// -> chunk -> element.  Each level subtracts the mass before the chosen
// entry; where rounding leaves no crossing at a level, the nearest entry of
// nonzero mass is taken instead, so a drawn element always has positive
// probability.
template <class TI>
__device__ int64_t draw_one(const CdfLds& c, const void* zrow, uint32_t nvec, int tail, uint32_t G,
                            uint32_t nchunk, uint32_t C, float t, float S, float nm) {
  int64_t ch;
  float r = 0.f;
  int pick = kLast;
  if (t < S) {
    // The run prefixes come from a parallel scan and need not be monotone to
    // the last bit; this bisection keeps p[hi] > t and p[lo - 1] <= t, so it
    // ends on a crossing either way.
    uint32_t lo = 0, hi = NT - 1;
    while (lo < hi) {
      const uint32_t mid = (lo + hi) >> 1;
      if (c.p[mid] > t)
        hi = mid;
      else
        lo = mid + 1;
    }
    r = fmaxf(t - (lo ? c.p[lo - 1] : 0.f), 0.f);
    const uint32_t r0 = min(lo * C, nchunk), r1 = min(r0 + C, nchunk);
    float cum = 0.f;
    uint32_t q = r0;
    for (; q < r1; ++q) {
      const float nc = cum + c.ls[q];
      if (nc > r) break;
      cum = nc;
    }
    if (q < r1) {
      ch = q;
      r = fmaxf(r - cum, 0.f);
      pick = kCross;
    } else {
      ch = last_positive(c, r0, r1);
      if (ch < 0) {
        ch = first_positive(c, r1, nchunk);
        pick = kFirst;
        if (ch < 0) {
          ch = last_positive(c, 0, r0);
          pick = kLast;
        }
      }
    }
  } else {
    ch = last_positive(c, 0, nchunk);
  }
  // element level, with the same sums as the chunk level
  const uint32_t v0 = (uint32_t)ch * G, v1 = min(v0 + G, nvec);
  float cum = 0.f;
  int64_t first = -1, last = -1, cross = -1;
  for (uint32_t v = v0; v < v1; ++v) {
    float f[4];
    unpack<TI>(load_vec<TI>(zrow, v, nvec, tail), f);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float w = ez(f[e], nm);
      const int64_t j = (int64_t)v * 4 + e;
      if (w > 0.f) {
        if (first < 0) first = j;
        last = j;
      }
      const float nc = cum + w;
      if (cross < 0 && nc > r) cross = j;
      cum = nc;
    }
  }
  if (pick == kFirst) return first;
  if (pick == kCross && cross >= 0) return cross;
  return last;
}

template <class TI, int NSLOT>
__global__ void __launch_bounds__(NT) k_sample(CacheArgs a) {
  __shared__ CdfLds c;
  const int tid = threadIdx.x;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const int M = a.K;
  if (a.mask && a.mask[row] == 0) {
    for (int i = tid; i < M; i += NT) {
      a.ids_out[row * M + i] = 0;
      if (a.logp) a.logp[row * M + i] = 0.f;
    }
    if (tid == 0 && a.lse_out) a.lse_out[row] = 0.f;
    return;
  }
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec, G = (uint32_t)a.G, nchunk = (uint32_t)a.nchunk;
  float m, nm;
  if constexpr (NSLOT > 0) {
    // G == 1: chunk q is vector q
    typename TI::Vec x[NSLOT];
    load_row<TI, NSLOT>(zrow, nvec, a.tail, tid, x);
    m = block_max<NW>(lane_max<TI, NSLOT>(x), c.red);
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) keep_packed(x[s]);
    nm = -m * kLog2e;
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
      const uint32_t b = slot_base<NT>(s, nvec);
      if ((uint32_t)(s * NT + NT) <= nvec || slot_owns<NT>(s, b, tid, nvec))
        c.ls[b + tid] = vec_sumexp<TI>(x[s], nm, 0.f);
    }
  } else {
    float mx = kNegInf;
    for (uint32_t v = tid; v < nvec; v += NT) {
      float f[4];
      unpack<TI>(load_vec<TI>(zrow, v, nvec, a.tail), f);
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, f[e]);
    }
    m = block_max<NW>(mx, c.red);
    nm = -m * kLog2e;
    for (uint32_t q = tid; q < nchunk; q += NT) {
      const uint32_t v1 = min(q * G + G, nvec);
      float acc = 0.f;
      for (uint32_t v = q * G; v < v1; ++v) acc = vec_sumexp<TI>(load_vec<TI>(zrow, v, nvec, a.tail), nm, acc);
      c.ls[q] = acc;
    }
  }
  __syncthreads();

  // runs of C consecutive chunks per thread, and their block-wide prefix
  const uint32_t C = (nchunk + NT - 1) / NT;
  {
    const uint32_t r0 = min((uint32_t)tid * C, nchunk), r1 = min(r0 + C, nchunk);
    float run = 0.f;
    for (uint32_t q = r0; q < r1; ++q) run += c.ls[q];
    const float incl = wave_incl_scan(run);
    if ((tid & 63) == 63) c.wt[tid >> 6] = incl;
    __syncthreads();
    float before = 0.f;
    for (int w = 0; w < (tid >> 6); ++w) before += c.wt[w];
    c.p[tid] = before + incl;
  }
  float S = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) S += c.wt[w];  // equals p[NT - 1] bit for bit
  __syncthreads();

  const float L = m + logf(S);
  if (tid == 0 && a.lse_out) a.lse_out[row] = L;
  // a NaN or +inf logit, or a row of -inf, leaves S NaN: no distribution
  const bool defined = S > 0.f && S <= 3.4028235e38f;
  for (int i = tid; i < M; i += NT) {
    const float u = a.u[row * M + i];
    int32_t id = -1;
    float lp = __builtin_nanf("");
    if (defined && u >= 0.f && u < 1.f) {
      const int64_t j = draw_one<TI>(c, zrow, nvec, a.tail, G, nchunk, C, u * S, S, nm);
      id = (int32_t)j;
      lp = load_elem<TI>(zrow, j) - L;
    }
    a.ids_out[row * M + i] = id;
    if (a.logp) a.logp[row * M + i] = lp;
  }
}

// ---------------------------------------------------------------- sampling, streamed

// Draws read each row once, so the common case is organised for overlap
// rather than residency: 256-lane workgroups with about 17 KiB of LDS,
// several per CU, so one row's prefix and draws overlap other rows' reads.
// The index-order CDF is kept as chunk records.  A chunk is 128 consecutive
// vectors (512 elements); the 16 lanes of one DPP row load it with eight
// instructions, each covering 16 consecutive vectors (128 bytes of bf16), so
// every load is coalesced.  Its record is the chunk max m_q (a DPP row max)
// and s_q = sum exp(z - m_q) (per-lane sums in load order, then a DPP row
// scan).  After the row, each record is scaled to the row max M
// (s'_q = s_q f_q, f_q = exp(m_q - M)), each thread sums its run of C
// consecutive chunks in order, and a block scan gives the run prefixes.  One
// wavefront per draw then finds the run (ballot over the prefixes), the
// chunk (a wave scan of the run's records and a ballot), and the element (a
// wave scan over the chunk in index order, two vectors per lane, at the same
// weights exp(z - m_q) f_q).  Where rounding leaves no crossing at a level,
// the nearest entry of nonzero mass is taken, as in the resident kernel.
constexpr int kSmpThreads = 256;
constexpr int kSmpWaves = kSmpThreads / 64;
constexpr int kSmpLoads = 8;                          // loads per lane per chunk
constexpr int kSmpChunkVecs = 16 * kSmpLoads;         // vectors per chunk (128)
constexpr int kSmpMaxChunks = 2048;                   // records per row: V <= 1,048,576

struct SmpLds {
  float m[kSmpMaxChunks];  // chunk max
  float s[kSmpMaxChunks];  // chunk sum at its max; then at the row max
  float p[kSmpThreads];    // inclusive prefix of the runs
  float wt[kSmpWaves];
  float red[kSmpWaves];
};

// max over the 16 lanes of a DPP row, in every lane of the row
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_move<0x140>(x));  // row_mirror
  x = fmaxf(x, dpp_move<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dpp_move<0xB1>(x));   // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp_move<0x4E>(x));   // quad_perm [2,3,0,1]
  return x;
}
// inclusive prefix sum within each DPP row of 16 lanes
__device__ __forceinline__ float row16_scan(float x) {
  const int rl = threadIdx.x & 15;
  float t;
  t = dpp_move<0x111>(x);  // row_shr:1
  if (rl >= 1) x += t;
  t = dpp_move<0x112>(x);  // row_shr:2
  if (rl >= 2) x += t;
  t = dpp_move<0x114>(x);  // row_shr:4
  if (rl >= 4) x += t;
  t = dpp_move<0x118>(x);  // row_shr:8
  if (rl >= 8) x += t;
  return x;
}

__device__ __forceinline__ int first_lane(uint64_t b) { return b ? __ffsll((long long)b) - 1 : -1; }
__device__ __forceinline__ int last_lane(uint64_t b) { return b ? 63 - __clzll((long long)b) : -1; }

// First (or last) chunk in [lo, hi) with positive mass, by wave ballots; -1 if none.
__device__ __forceinline__ int64_t chunk_positive(const SmpLds& c, int64_t lo, int64_t hi,
                                                  bool last) {
  const int lane = threadIdx.x & 63;
  if (!last) {
    for (int64_t b = lo; b < hi; b += 64) {
      const int64_t q = b + lane;
      const int f = first_lane(__ballot(q < hi && c.s[q] > 0.f));
      if (f >= 0) return b + f;
    }
  } else {
    for (int64_t b = hi; b > lo; b -= 64) {
      const int64_t q = b - 64 + lane;
      const int l = last_lane(__ballot(q >= lo && q < b && c.s[q] > 0.f));
      if (l >= 0) return b - 64 + l;
    }
  }
  return -1;
}

// One draw by one wavefront (the result is wave-uniform): the first element
// whose cumulative mass exceeds t = u * S.
template <class TI>
__device__ int64_t smp_draw(const SmpLds& c, const void* zrow, uint32_t nvec, int tail,
                            uint32_t nchunk, uint32_t C, float t, float S, float nM) {
  const int lane = threadIdx.x & 63;
  int64_t q = -1;
  float r = 0.f;
  int pick = kLast;
  if (t < S) {
    // run: the first i with p[i] > t (each lane looks at 4 entries)
    int li = -1;
#pragma unroll
    for (int k = 3; k >= 0; --k)
      if (c.p[4 * lane + k] > t) li = 4 * lane + k;
    const int fl = first_lane(__ballot(li >= 0));
    const int i = __shfl(li, fl < 0 ? 0 : fl, 64);  // fl >= 0: p[255] = S > t
    r = fmaxf(t - (i ? c.p[i - 1] : 0.f), 0.f);
    // chunk within the run (C <= 8 chunks, one per lane)
    const uint32_t r0 = min((uint32_t)i * C, nchunk), r1 = min(r0 + C, nchunk);
    const uint32_t qq = r0 + (uint32_t)lane;
    const float sq = qq < r1 ? c.s[qq] : 0.f;
    const float incl = wave_incl_scan(sq);
    const int cl = first_lane(__ballot(qq < r1 && incl > r));
    if (cl >= 0) {
      const float before = cl > 0 ? __shfl(incl, cl - 1, 64) : 0.f;
      q = r0 + cl;
      r = fmaxf(r - before, 0.f);
      pick = kCross;
    } else {
      const int ll = last_lane(__ballot(qq < r1 && sq > 0.f));
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
  // element within chunk q: lane l holds vectors 2l and 2l + 1 of the chunk
  // (elements 8l .. 8l + 7, in index order)
  const float mq = c.m[q];
  const float nmq = -mq * kLog2e, fq = fast_exp2(fmaf(mq, kLog2e, nM));
  const uint32_t v = (uint32_t)q * kSmpChunkVecs + 2u * (uint32_t)lane;
  float wl[8];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const bool in = v + h < nvec;
    float f[4];
    unpack<TI>(in ? load_vec<TI>(zrow, v + h, nvec, tail) : neg_inf_vec<TI>(), f);
#pragma unroll
    for (int e = 0; e < 4; ++e) wl[4 * h + e] = in ? ez(f[e], nmq) : 0.f;
  }
  float lsum = 0.f;
  int e_first = -1, e_last = -1;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    lsum += wl[e];
    if (wl[e] > 0.f) {
      if (e_first < 0) e_first = e;
      e_last = e;
    }
  }
  int vl = -1, el = -1;  // chosen lane and element in it
  if (pick == kCross) {
    const float incl = wave_incl_scan(lsum);
    vl = first_lane(__ballot(incl * fq > r));
    if (vl >= 0) {
      float cum = vl > 0 ? __shfl(incl, vl - 1, 64) : 0.f;
      int ec = -1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        cum += wl[e];
        if (ec < 0 && cum * fq > r) ec = e;
      }
      el = __shfl(ec, vl, 64);
      if (el < 0) vl = -1;  // rounding: no element crossing in that lane
    }
    if (vl < 0) pick = kLast;
  }
  if (pick == kFirst) {
    vl = first_lane(__ballot(e_first >= 0));
    el = __shfl(e_first, vl < 0 ? 0 : vl, 64);
  } else if (pick == kLast) {
    vl = last_lane(__ballot(e_last >= 0));
    el = __shfl(e_last, vl < 0 ? 0 : vl, 64);
  }
  if (vl < 0 || el < 0) return -1;
  return ((int64_t)q * kSmpChunkVecs + 2 * vl) * 4 + el;
}

template <class TI>
__global__ void __launch_bounds__(kSmpThreads) k_sample_stream(CacheArgs a) {
  constexpr int T = kSmpThreads, W = kSmpWaves, R = kSmpLoads, CV = kSmpChunkVecs;
  typedef typename TI::Vec Vec;
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
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec;
  const uint32_t nchunk = (nvec + CV - 1) / CV;  // <= kSmpMaxChunks
  const bool ragged = a.tail != TI::EPV;

  // one pass over the row: DPP row k of wave w takes chunks 4 w + k,
  // 4 w + k + 4 W, ...; its lane l loads vectors 16 b + l of the chunk
  const uint32_t rowk = (uint32_t)lane >> 4, rl = (uint32_t)lane & 15;
  float lmax = kNegInf;
  for (uint32_t q0 = 4u * w; q0 < nchunk; q0 += 4u * W) {  // wave-uniform
    const uint32_t q = q0 + rowk;
    const uint32_t v0 = q * CV + rl;
    Vec x[R];
#pragma unroll
    for (int b = 0; b < R; ++b) x[b] = ld_nt<TI>(zrow, min(v0 + 16u * b, nvec - 1));
    float lm = kNegInf;
#pragma unroll
    for (int b = 0; b < R; ++b) {
      const uint32_t v = v0 + 16u * b;
      if (v >= nvec) x[b] = neg_inf_vec<TI>();
      else if (ragged && v == nvec - 1) x[b] = tail_masked<TI>(x[b], a.tail);
      float f[4];
      unpack<TI>(x[b], f);
      lm = fmaxf(lm, fmaxf(fmaxf(f[0], f[1]), fmaxf(f[2], f[3])));
    }
    const float mq = row16_max(lm);
    float ls = 0.f;
    if (mq != kNegInf) {  // an all -inf chunk has no mass (and no NaN)
      const float nm = -mq * kLog2e;
#pragma unroll
      for (int b = 0; b < R; ++b) {
        float f[4];
        unpack<TI>(x[b], f);
#pragma unroll
        for (int e = 0; e < 4; ++e) ls += ez(f[e], nm);
      }
    }
    const float sq = row16_scan(ls);
    if (rl == 15 && q < nchunk) {
      c.m[q] = mq;
      c.s[q] = sq;
    }
    lmax = fmaxf(lmax, lm);
  }
  const float Mx = block_max<W>(lmax, c.red);  // ends with a barrier: records visible
  const float nM = -Mx * kLog2e;
  // records at the row max; runs of C consecutive chunks per thread
  const uint32_t C = (nchunk + T - 1) / T;
  {
    const uint32_t r0 = min((uint32_t)tid * C, nchunk), r1 = min(r0 + C, nchunk);
    float run = 0.f;
    for (uint32_t q = r0; q < r1; ++q) {
      const float mq = c.m[q];
      const float sq = mq == kNegInf ? 0.f : c.s[q] * fast_exp2(fmaf(mq, kLog2e, nM));
      c.s[q] = sq;
      run += sq;
    }
    const float incl = wave_incl_scan(run);
    if (lane == 63) c.wt[w] = incl;
    __syncthreads();
    float before = 0.f;
    for (int k = 0; k < w; ++k) before += c.wt[k];
    c.p[tid] = before + incl;
  }
  float S = 0.f;
#pragma unroll
  for (int k = 0; k < W; ++k) S += c.wt[k];  // equals p[T - 1] bit for bit
  __syncthreads();

  const float L = Mx + logf(S);
  if (tid == 0 && a.lse_out) a.lse_out[row] = L;
  // a NaN or +inf logit, or a row of -inf, leaves S NaN or 0: no distribution
  const bool defined = S > 0.f && S <= 3.4028235e38f;
  for (int i = w; i < M; i += W) {  // one draw per wavefront
    const float u = a.u[row * M + i];
    int32_t id = -1;
    float lp = __builtin_nanf("");
    if (defined && u >= 0.f && u < 1.f) {
      const int64_t j = smp_draw<TI>(c, zrow, nvec, a.tail, nchunk, C, u * S, S, nM);
      if (j >= 0) {
        id = (int32_t)j;
        lp = load_elem<TI>(zrow, j) - L;
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

template <class TI, int NSLOT, bool LSE>
__global__ void __launch_bounds__(NT) k_topk(CacheArgs a) {
  __shared__ TopkLds sh;
  const int tid = threadIdx.x;
  const int64_t row = xcd_remap(blockIdx.x, gridDim.x);
  const int k = a.K;
  // after the streamed kernel: only the rows it left to this one
  if (a.redo && a.ids_out[row * k] != kTopkRedo) return;
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

// ---------------------------------------------------------------- top-k, streamed

// The top-k support of rows of at least 16,384 entries, for k <= 64, reads
// each row once: 256-lane workgroups with about 38 KiB of LDS, four per CU.
// Each lane keeps the running maximum of the values it has seen.  After each
// tile of 8 coalesced loads per lane, the k-th largest of the wave's 64
// running maxima (a radix select over their order keys by ballots) is a
// lower bound on the row's k-th largest (k lanes have each seen an element
// at least that large), updated every fourth tile; the bound only rises.
// Elements not below the wave's current bound, and NaNs, are appended to
// its LDS buffer by ballot compaction, skipping every vector whose maximum
// is below the bound in all lanes.  At the end the largest of the four wave
// bounds is still a lower bound, every element at or above it is in some
// buffer, and a block sort of those (at most 256) gives the support.  A row
// whose buffers overflow (many equal large values) or that leaves more than
// 256 candidates is marked, and a second launch runs the resident kernel on
// the marked rows only.
constexpr int kTkThreads = 256;
constexpr int kTkWaves = kTkThreads / 64;
constexpr int kTkLoads = 8;    // vector loads per lane per tile
constexpr int kTkCap = 1024;   // candidates per wave
constexpr int kTkMaxK = 64;    // one running maximum per lane bounds k
constexpr int64_t kTkMinVec = 4096;

struct TkLds {
  uint64_t buf[kTkWaves][kTkCap];
  uint64_t sbuf[2][kTkThreads];
  uint64_t sel[kTkThreads];
  uint32_t cnt[kTkWaves];
  uint32_t theta[kTkWaves];
  uint32_t nsel;
  Stats st[kTkWaves];
};

template <class TI, bool LSE>
__global__ void __launch_bounds__(kTkThreads) k_topk_stream(CacheArgs a) {
  constexpr int T = kTkThreads, W = kTkWaves, B = kTkLoads;
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
  const void* zrow = (const char*)a.logits + row * a.ld * TI::BYTES;
  const uint32_t nvec = (uint32_t)a.nvec;  // >= kTkMinVec: every wave's first tile is full
  const uint32_t V32 = (uint32_t)a.V;
  float run = kNegInf;  // this lane's running maximum (NaN ignored)
  uint32_t theta = 0;   // the wave's bound as an order key (wave-uniform)
  float thf = kNegInf;  // the same bound as a value
  uint32_t nb = 0;      // the wave's candidates so far (wave-uniform)
  float m = kNegInf, sum = 0.f;
  uint32_t tile = 0;
  for (uint32_t t0 = (uint32_t)w * 64 * B; t0 < nvec; t0 += W * 64 * B) {  // wave-uniform
    Vec xb[B];
#pragma unroll
    for (int b = 0; b < B; ++b) xb[b] = ld_nt<TI>(zrow, min(t0 + 64u * b + lane, nvec - 1));
    // a whole tile inside the row needs no per-element checks (wave-uniform)
    const bool full = t0 + 64u * B <= nvec && a.tail == TI::EPV;
    auto vals = [&](int b, float (&f)[4]) {
      unpack<TI>(xb[b], f);
      if (!full) {
        const uint32_t v = t0 + 64u * b + lane;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!(v < nvec && v * 4u + e < V32)) f[e] = kNegInf;
      }
    };
    // pass 1: vector maxima (NaN ignored) and the tile's
    float vm[B];
    float tmx = kNegInf;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float f[4];
      vals(b, f);
      vm[b] = fmaxf(fmaxf(f[0], f[1]), fmaxf(f[2], f[3]));
      tmx = fmaxf(tmx, vm[b]);
    }
    // NaN (or +inf) in this lane's part of the tile: the tile's sum of
    // exponentials is NaN; without the sums, tested element by element
    bool nan = false;
    if constexpr (LSE) {
      const float mn = fmaxf(m, tmx);
      if (mn != kNegInf) {
        float acc = 0.f;
        const float nm = -mn * kLog2e;
#pragma unroll
        for (int b = 0; b < B; ++b) {
          float f[4];
          vals(b, f);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc += fast_exp2(fmaf(f[e], kLog2e, nm));
        }
        nan = acc != acc;
        sum = fmaf(sum, rescale(m, mn), acc);
        m = mn;
      }
    } else {
#pragma unroll
      for (int b = 0; b < B; ++b) {
        float f[4];
        vals(b, f);
#pragma unroll
        for (int e = 0; e < 4; ++e) nan = nan || f[e] != f[e];
      }
    }
    run = fmaxf(run, tmx);
    // every fourth tile: k lanes of this wave have each seen a value at
    // least the k-th largest running maximum, found bit by bit with ballots
    // (the bound only rises)
    if ((tile++ & 3) == 0) {
      const uint32_t rk = order_key(__float_as_uint(run));
      if ((uint32_t)__popcll(__ballot(rk > theta)) >= (uint32_t)k) {
        uint32_t t = 0;
        for (int bit = 31; bit >= 0; --bit) {
          const uint32_t c = t | (1u << bit);
          if ((uint32_t)__popcll(__ballot(rk >= c)) >= (uint32_t)k) t = c;
        }
        theta = t;
        thf = key_value(t);
      }
    }
    // candidates: every element not below the bound, and every NaN
    // (!(x < bound) holds for both); vectors whose maximum is below the
    // bound and that hold no NaN are skipped by the whole wave
#pragma unroll
    for (int b = 0; b < B; ++b) {
      if (__ballot(!(vm[b] < thf) || nan)) {  // wave-uniform
        const uint32_t v = t0 + 64u * b + lane;
        float f[4];
        vals(b, f);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool take = !(f[e] < thf) && (full || (v < nvec && v * 4u + e < V32));
          const uint64_t mask = __ballot(take);
          if (mask) {  // wave-uniform
            const uint32_t pos = nb + (uint32_t)__popcll(mask & ((1ull << lane) - 1ull));
            if (take && pos < (uint32_t)kTkCap)
              sh.buf[w][pos] = ((uint64_t)order_key(__float_as_uint(f[e])) << 32) |
                               (0xFFFFFFFFu - (v * 4u + e));
            nb += (uint32_t)__popcll(mask);
          }
        }
      }
    }
  }
  if (lane == 0) {
    sh.cnt[w] = nb;
    sh.theta[w] = theta;
  }
  if (tid == 0) sh.nsel = 0u;
  float L = 0.f;
  if constexpr (LSE) {
    Stats st = stats_empty();
    st.mz = m;
    st.sz = sum;
    st = block_merge<false, W>(st, sh.st);  // barriers: counts and bounds visible
    L = st.mz + logf(st.sz);
  } else {
    __syncthreads();
  }
  uint32_t tstar = 0;
  bool overflow = false;
#pragma unroll
  for (int q = 0; q < W; ++q) {
    tstar = max(tstar, sh.theta[q]);
    overflow = overflow || sh.cnt[q] > (uint32_t)kTkCap;
  }
  if (!overflow) {
    // every element with key >= tstar is in some buffer: each wave's bound
    // never exceeded tstar while it appended
#pragma unroll
    for (int q = 0; q < W; ++q) {
      const uint32_t n = sh.cnt[q];
      for (uint32_t i = tid; i < n; i += T) {
        const uint64_t e = sh.buf[q][i];
        if ((uint32_t)(e >> 32) >= tstar) {
          const uint32_t pos = atomicAdd(&sh.nsel, 1u);
          if (pos < (uint32_t)T) sh.sel[pos] = e;
        }
      }
    }
  }
  __syncthreads();
  const uint32_t nsel = sh.nsel;
  if (overflow || nsel > (uint32_t)T || nsel < (uint32_t)k) {  // workgroup-uniform
    if (tid == 0) a.ids_out[row * k] = kTopkRedo;
    return;
  }
  int P = 2;
  while (P < (int)nsel) P <<= 1;
  const uint64_t mine =
      block_sort_desc<uint64_t, T>(tid < (int)nsel ? sh.sel[tid] : 0ull, sh.sbuf, P);
  if (tid < k) {
    const uint32_t j = 0xFFFFFFFFu - (uint32_t)mine;
    a.ids_out[row * k + tid] = (int32_t)j;
    if (a.logp) a.logp[row * k + tid] = key_value((uint32_t)(mine >> 32)) - L;
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
  switch (op) {
    case CacheOp::Sample:
      hipLaunchKernelGGL((k_sample<TI, NSLOT>), grid, block, 0, stream, a);
      break;
    case CacheOp::Topk:
      if (a.logp || a.lse_out)
        hipLaunchKernelGGL((k_topk<TI, NSLOT, true>), grid, block, 0, stream, a);
      else
        hipLaunchKernelGGL((k_topk<TI, NSLOT, false>), grid, block, 0, stream, a);
      break;
    case CacheOp::Score:
      break;
  }
  return hipGetLastError();
}

template <class TI>
hipError_t launch_dt(const CacheArgs& a, CacheOp op, bool resident, hipStream_t stream) {
  if (op == CacheOp::Sample &&
      (a.nvec + kSmpChunkVecs - 1) / kSmpChunkVecs <= (int64_t)kSmpMaxChunks) {
    hipLaunchKernelGGL((k_sample_stream<TI>), dim3((unsigned)a.N), dim3(kSmpThreads), 0, stream,
                       a);
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
    b.redo = 1;  // the rows the streamed kernel left
    if (!resident) return launch_op<TI, 0>(b, op, stream);
    constexpr int big = TI::BYTES == 2 ? 38 : 19, small = TI::BYTES == 2 ? 16 : 8;
    if (b.nvec <= (int64_t)small * NT) return launch_op<TI, small>(b, op, stream);
    return launch_op<TI, big>(b, op, stream);
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
