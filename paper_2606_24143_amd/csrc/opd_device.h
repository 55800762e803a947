// Device helpers shared by the HIP kernels of libopd: element types and
// their packing, wide loads, deterministic wave and workgroup reductions,
// running softmax statistics, and the register-slot layout of a resident
// row.  Internal; included by the .hip sources only.
#pragma once

#include <math.h>

#include "opd_internal.h"

namespace opd {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
// Each lane handles vectors of 4 consecutive elements: 8-byte loads of bf16,
// 16-byte loads of fp32.  The fp32 gradient of a vector is then one 16-byte
// store, and a wavefront's store instruction covers one contiguous 1 KiB span
// (a lane holding 8 bf16 would write 32 bytes as two half-filled stores).
struct InBf16 {
  static constexpr int EPV = 4;  // elements per vector
  static constexpr int BYTES = 2;
  typedef u32x2 Vec;
};
struct InF32 {
  static constexpr int EPV = 4;
  static constexpr int BYTES = 4;
  typedef u32x4 Vec;
};
struct OutF32 {
  static constexpr int BYTES = 4;
};
struct OutBf16 {
  static constexpr int BYTES = 2;
};

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// a * b with 0 * x = 0 for every x (NaN and infinities included): the
// legacy multiply, for weights of zero times differences that may be NaN.
// Bound to the compiler intrinsic rather than written as inline asm, so that
// the wait state a VALU read of a fresh v_exp_f32 result needs on gfx950 is
// inserted by the compiler (it does not inspect inline asm for that hazard).
extern "C" __device__ float opd_fmul_legacy(float, float) __asm("llvm.amdgcn.fmul.legacy");
__device__ __forceinline__ float mul_zero_safe(float a, float b) { return opd_fmul_legacy(a, b); }

// ---------------------------------------------------------------- XCD-aware placement
// The MI355X dispatcher hands workgroup b of a grid to XCD b % 8.  Remapping
// b so that each XCD works through blocks of kXcdBlock consecutive rows (in
// its own dispatch order) keeps every XCD's concurrent rows adjacent in
// memory; measured on the row-per-workgroup read+write pattern at
// V = 151,936 this cuts the time by about 6% against the identity mapping.
// Blocks, rather than one contiguous eighth per XCD, keep the XCDs balanced
// when the valid rows of a masked batch cluster.  Workgroups past the last
// whole round of 8 blocks keep their place, so the map is a permutation of
// [0, G).
constexpr int kXcds = 8;
#ifndef OPD_XCD_BLOCK
#define OPD_XCD_BLOCK 64
#endif
constexpr int64_t kXcdBlock = OPD_XCD_BLOCK;

__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t G) {
  const int64_t B = G / kXcds < kXcdBlock ? G / kXcds : kXcdBlock;
  if (B == 0) return b;
  const int64_t span = B * kXcds;
  if (b >= G - G % span) return b;
  const int64_t q = b / kXcds;  // b's place in its XCD's dispatch order
  return (q / B) * span + (b % kXcds) * B + q % B;
}

// One contiguous eighth of a one-shot grid per XCD (32-bit indices).  For
// grids of short workgroups that each write one 16 KiB piece; measured on a
// zero fill of an [8192, 151936] fp32 gradient this beat both the identity
// and the 64-row blocks above.
__device__ __forceinline__ uint32_t xcd_eighths(uint32_t b, uint32_t G) {
  const uint32_t g8 = G - G % kXcds;
  return b < g8 ? (b % kXcds) * (g8 / kXcds) + b / kXcds : b;
}

// ---------------------------------------------------------------- dtype helpers

template <class TI>
__device__ __forceinline__ void unpack(const typename TI::Vec& x, float (&f)[4]) {
  if constexpr (TI::BYTES == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      f[2 * d] = __uint_as_float(x[d] << 16);              // element 2d: low half
      f[2 * d + 1] = __uint_as_float(x[d] & 0xFFFF0000u);  // element 2d+1: high half
    }
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d) f[d] = __uint_as_float(x[d]);
  }
}

template <class TI>
__device__ __forceinline__ float load_elem(const void* row, int64_t j) {
  if constexpr (TI::BYTES == 2)
    return __uint_as_float((uint32_t)((const uint16_t*)row)[j] << 16);
  else
    return ((const float*)row)[j];
}

template <class TI>
__device__ __forceinline__ typename TI::Vec neg_inf_vec() {
  typename TI::Vec x;
  const uint32_t w = TI::BYTES == 2 ? 0xFF80FF80u : 0xFF800000u;
#pragma unroll
  for (int d = 0; d < (int)(sizeof(x) / 4); ++d) x[d] = w;
  return x;
}

// Elements [valid, EPV) of a loaded vector become -inf, so they drop out of
// the max and the sum without a branch in the hot loop.
template <class TI>
__device__ __forceinline__ void mask_tail(typename TI::Vec& x, int valid) {
  if constexpr (TI::BYTES == 2) {
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      if (2 * d >= valid)
        x[d] = 0xFF80FF80u;
      else if (2 * d + 1 >= valid)
        x[d] = (x[d] & 0x0000FFFFu) | 0xFF800000u;
    }
  } else {
#pragma unroll
    for (int d = 0; d < 4; ++d)
      if (d >= valid) x[d] = 0xFF800000u;
  }
}

// Empty register barrier: the compiler must assume x changed, so it re-derives
// fp32 values from the packed row instead of keeping an unpacked copy alive
// across sweeps (which would double the registers the row occupies).
template <class VecT>
__device__ __forceinline__ void keep_packed(VecT& x) { asm volatile("" : "+v"(x)); }

template <class TI, class IdxT>
__device__ __forceinline__ typename TI::Vec ld_nt(const void* row, IdxT v) {
  return __builtin_nontemporal_load((const typename TI::Vec*)row + v);
}
template <class TI, class IdxT>
__device__ __forceinline__ typename TI::Vec ld_cached(const void* row, IdxT v) {
  return ((const typename TI::Vec*)row)[v];
}

// ---------------------------------------------------------------- buffer access
// A buffer resource for one slot of a row: its base is the slot's first
// vector and its byte count what remains of the row from there (0 for a slot
// wholly past the end).  The hardware checks each lane's offset against that
// count: loads past the end return zeros, stores past the end are dropped.
// The check covers the lane offset only, not the scalar offset operand, so
// the slot's position goes into the base (scalar arithmetic) and the scalar
// offset stays 0.  A lane then addresses every slot with one fixed offset and
// no arithmetic or bounds test of its own.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;  // raw access, 32-bit data format
constexpr int kAuxNt = 2;              // cache policy: non-temporal
// (row bytes < 2^31; the count is clamped with a signed max, which has a
// scalar instruction, and read back as a scalar so the resource stays in
// scalar registers)
__device__ __forceinline__ Rsrc slot_rsrc(const void* row, uint32_t row_bytes, uint32_t off) {
  const int left = (int)row_bytes - (int)off;
  const int count = __builtin_amdgcn_readfirstlane(left > 0 ? left : 0);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>((const char*)row + off), 0, count,
                                           kRsrcWord3);
}
template <class TI, int AUX>
__device__ __forceinline__ typename TI::Vec buf_ld(Rsrc r, uint32_t voff) {
  if constexpr (TI::BYTES == 2)
    return __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, 0, AUX);
  else
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, AUX);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const uint32_t a = __builtin_bit_cast(uint16_t, (__bf16)lo);
  const uint32_t b = __builtin_bit_cast(uint16_t, (__bf16)hi);
  return a | (b << 16);
}

// Store the gradient values of vector v (elements [4v, 4v + valid)).
// IdxT = uint32_t lets the compiler address with a uniform row base plus a
// 32-bit lane offset instead of a 64-bit address per vector.
template <class TI, class TO, class IdxT>
__device__ __forceinline__ void store_vec(void* grow, IdxT v, const float (&g)[4], int valid) {
  if constexpr (TO::BYTES == 4) {
    float* p = (float*)grow + v * 4;
    if (valid == 4)
      __builtin_nontemporal_store(f32x4{g[0], g[1], g[2], g[3]}, (f32x4*)p);
    else
      for (int e = 0; e < valid; ++e) p[e] = g[e];
  } else {
    uint16_t* p = (uint16_t*)grow + v * 4;
    if (valid == 4)
      __builtin_nontemporal_store(u32x2{pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3])},
                                  (u32x2*)p);
    else
      for (int e = 0; e < valid; ++e) p[e] = __builtin_bit_cast(uint16_t, (__bf16)g[e]);
  }
}

// Store the four gradient values of a vector through a slot's buffer resource
// (non-temporal; a store past the row's end is dropped).
template <class TO>
__device__ __forceinline__ void buf_store(Rsrc r, uint32_t voff, const float (&g)[4]) {
  if constexpr (TO::BYTES == 4)
    __builtin_amdgcn_raw_buffer_store_b128(
        u32x4{__float_as_uint(g[0]), __float_as_uint(g[1]), __float_as_uint(g[2]),
              __float_as_uint(g[3])},
        r, (int)voff, 0, kAuxNt);
  else
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3])},
                                          r, (int)voff, 0, kAuxNt);
}

// ---------------------------------------------------------------- reductions
// Butterfly reductions: every lane ends with the same value (each pairwise
// step is commutative), and the order is fixed, so results are reproducible.

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <int NW>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) r = fmaxf(r, red[w]);
  __syncthreads();
  return r;
}
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) r += red[w];
  __syncthreads();
  return r;
}

// Running (max, sum of exp(x - max)) statistics of a row, plus, for the dense
// estimators, those of the teacher row and the two cross sums
//   tr = sum_j e^{z_j - mz} (z_j - y_j),   tf = sum_j e^{y_j - my} (y_j - z_j),
// which give E_p[z - y] = tr / sz and E_q[y - z] = tf / sy.
struct Stats {
  float mz, sz, tr;
  float my, sy, tf;
};

__device__ __forceinline__ Stats stats_empty() { return Stats{kNegInf, 0.f, 0.f, kNegInf, 0.f, 0.f}; }

// factor exp(m_old - m_new) for rescaling a running sum; 0 for an empty sum.
__device__ __forceinline__ float rescale(float m_old, float m_new) {
  return m_old == kNegInf ? 0.f : fast_exp2((m_old - m_new) * kLog2e);
}

template <bool DENSE>
__device__ __forceinline__ Stats stats_merge(const Stats& a, const Stats& b) {
  Stats r;
  r.mz = fmaxf(a.mz, b.mz);
  {
    const float fa = rescale(a.mz, r.mz), fb = rescale(b.mz, r.mz);
    r.sz = a.sz * fa + b.sz * fb;
    r.tr = DENSE ? a.tr * fa + b.tr * fb : 0.f;
  }
  if constexpr (DENSE) {
    r.my = fmaxf(a.my, b.my);
    const float fa = rescale(a.my, r.my), fb = rescale(b.my, r.my);
    r.sy = a.sy * fa + b.sy * fb;
    r.tf = a.tf * fa + b.tf * fb;
  } else {
    r.my = kNegInf;
    r.sy = 0.f;
    r.tf = 0.f;
  }
  return r;
}

template <bool DENSE>
__device__ __forceinline__ Stats wave_merge(Stats s) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    Stats t;
    t.mz = __shfl_xor(s.mz, o, 64);
    t.sz = __shfl_xor(s.sz, o, 64);
    t.tr = __shfl_xor(s.tr, o, 64);
    t.my = __shfl_xor(s.my, o, 64);
    t.sy = __shfl_xor(s.sy, o, 64);
    t.tf = __shfl_xor(s.tf, o, 64);
    s = stats_merge<DENSE>(s, t);
  }
  return s;
}

template <bool DENSE, int NW>
__device__ __forceinline__ Stats block_merge(Stats s, Stats* red) {
  s = wave_merge<DENSE>(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  Stats r = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) r = stats_merge<DENSE>(r, red[w]);
  __syncthreads();
  return r;
}

// The same merge with the NW wave results combined by a butterfly over NW
// lanes of every wave (log2(NW) steps instead of NW - 1 in sequence).  The
// pairing, and so the rounding, is fixed.  NW is a power of two up to 64.
template <bool DENSE, int NW>
__device__ __forceinline__ Stats block_merge_tree(Stats s, Stats* red) {
  static_assert((NW & (NW - 1)) == 0 && NW <= 64, "NW: a power of two up to 64");
  s = wave_merge<DENSE>(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  Stats r = red[threadIdx.x & (NW - 1)];
#pragma unroll
  for (int o = NW / 2; o >= 1; o >>= 1) {
    Stats t;
    t.mz = __shfl_xor(r.mz, o, 64);
    t.sz = __shfl_xor(r.sz, o, 64);
    t.tr = __shfl_xor(r.tr, o, 64);
    t.my = __shfl_xor(r.my, o, 64);
    t.sy = __shfl_xor(r.sy, o, 64);
    t.tf = __shfl_xor(r.tf, o, 64);
    r = stats_merge<DENSE>(r, t);
  }
  __syncthreads();
  return r;
}

// Fold one 16-byte vector of z (and y) into a lane's running statistics.
template <class TI, bool DENSE>
__device__ __forceinline__ void stats_add(Stats& s, const typename TI::Vec& xz,
                                          const typename TI::Vec& xy) {
  constexpr int EPV = TI::EPV;
  float fz[EPV];
  unpack<TI>(xz, fz);
  float vm = fz[0];
#pragma unroll
  for (int e = 1; e < EPV; ++e) vm = fmaxf(vm, fz[e]);
  if constexpr (!DENSE) {
    const float mn = fmaxf(s.mz, vm);
    if (mn != kNegInf) {
      float acc = s.sz * rescale(s.mz, mn);
      const float nm = -mn * kLog2e;
#pragma unroll
      for (int e = 0; e < EPV; ++e) acc += fast_exp2(fmaf(fz[e], kLog2e, nm));
      s.sz = acc;
      s.mz = mn;
    }
  } else {
    float fy[EPV];
    unpack<TI>(xy, fy);
    float vmy = fy[0];
#pragma unroll
    for (int e = 1; e < EPV; ++e) vmy = fmaxf(vmy, fy[e]);
    // each row on its own: while a row's maximum is -inf its terms are 0
    // (offset 0 keeps exp(-inf) = 0 instead of exp(-inf + inf))
    const float mnz = fmaxf(s.mz, vm), mny = fmaxf(s.my, vmy);
    const float cz = rescale(s.mz, mnz), cy = rescale(s.my, mny);
    float sz = s.sz * cz, tr = s.tr * cz, sy = s.sy * cy, tf = s.tf * cy;
    const float nmz = mnz != kNegInf ? -mnz * kLog2e : 0.f;
    const float nmy = mny != kNegInf ? -mny * kLog2e : 0.f;
#pragma unroll
    for (int e = 0; e < EPV; ++e) {
      const float pz = fast_exp2(fmaf(fz[e], kLog2e, nmz));
      const float py = fast_exp2(fmaf(fy[e], kLog2e, nmy));
      const float d = fz[e] - fy[e];
      // an element that is -inf in both rows has weight 0 but d = NaN: the
      // legacy multiply gives 0 * d = 0
      tr += mul_zero_safe(pz, d);
      tf -= mul_zero_safe(py, d);
      sz += pz;
      sy += py;
    }
    s.mz = mnz; s.sz = sz; s.tr = tr;
    s.my = mny; s.sy = sy; s.tf = tf;
  }
}

// Register slot s of a resident row covers vectors [s*NT, s*NT + NT).  A slot
// that would run past the row end is moved back to end at it, [nvec - NT,
// nvec), so every lane loads a vector inside the row; lanes of a moved slot
// whose vector an earlier slot already holds are masked (slot_owns false).
// Rows narrower than one slot use base 0 with lane offsets clamped.
template <int NT>
__device__ __forceinline__ uint32_t slot_base(int s, uint32_t nvec) {
  const uint32_t b = (uint32_t)(s * NT);
  if (b + NT <= nvec) return b;
  return nvec >= (uint32_t)NT ? nvec - NT : 0u;
}
template <int NT>
__device__ __forceinline__ bool slot_owns(int s, uint32_t base, int tid, uint32_t nvec) {
  if ((uint32_t)(s * NT + NT) <= nvec) return true;  // a full slot: wave-uniform
  const uint32_t v = base + (uint32_t)tid;
  return v >= (uint32_t)(s * NT) && v < nvec;
}

// Lane offset of this lane's vector within slot s (base b): the lane id for a
// full slot, clamped to the row end for a moved or narrow one.
template <int NT>
__device__ __forceinline__ uint32_t slot_off(int s, uint32_t b, int tid, uint32_t nvec) {
  if ((uint32_t)(s * NT + NT) <= nvec) return (uint32_t)tid;
  return min((uint32_t)tid, nvec - 1 - b);
}

// Empty asm that takes y as an input and claims to modify x: work on x is
// not started before y has arrived, so the compiler cannot compute the
// student-only terms of every slot early and hold them until the teacher
// data lands.
template <class VecT>
__device__ __forceinline__ void after(VecT& x, const VecT& y) {
  asm volatile("" : "+v"(x) : "v"(y));
}

// Opaque copy: values derived from it in a later sweep are recomputed there
// (a few scalar and lane operations) instead of being kept live from an
// earlier sweep, which would cost registers the resident row needs.
template <class T>
__device__ __forceinline__ T fresh_s(T x) {
  asm volatile("" : "+s"(x));
  return x;
}
template <class T>
__device__ __forceinline__ T fresh_v(T x) {
  asm volatile("" : "+v"(x));
  return x;
}

}  // namespace
}  // namespace opd
