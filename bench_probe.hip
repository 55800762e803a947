// Read-bandwidth probe for bench.py: the device's plain read rate, measured
// in the same process as the kernels it is compared with.  Not part of the
// library; built beside it by __graft_entry__.build().
//
// One pass over a buffer, each workgroup streaming its own contiguous share
// with non-temporal 16-byte loads (consecutive lanes on consecutive vectors,
// eight loads in flight per lane).  Nothing depends on the data but a
// never-taken store, so the only HBM traffic is the read.  On the MI355X this
// pattern read 7.0-7.07 TB/s with 1,024 to 8,192 workgroups, against
// 5.8-6.3 TB/s for a grid-stride loop over the whole buffer.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kThreads = 256;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t fold(u32x4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

__global__ void __launch_bounds__(kThreads) k_read_probe(const u32x4* __restrict__ p, uint64_t n,
                                                       uint32_t* out) {
  constexpr int U = 8;
  const uint64_t share = (n + gridDim.x - 1) / gridDim.x;
  const uint64_t c0 = (uint64_t)blockIdx.x * share;
  const uint64_t c1 = c0 + share < n ? c0 + share : n;
  uint64_t i = c0 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (U - 1) * kThreads < c1; i += U * kThreads) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + i + u * kThreads);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= fold(v[u]);
  }
  for (; i < c1; i += kThreads) acc ^= fold(__builtin_nontemporal_load(p + i));
  if (acc == 0x9E3779B9u) out[blockIdx.x] = acc;  // keeps the loads (the bench fills the buffer with words of 1: never taken)
}

}  // namespace

// Reads bytes / 16 vectors of buf (device memory, 16-byte aligned) once with
// `groups` workgroups of 256 lanes; out holds `groups` words (device).  The
// call is asynchronous on `stream`; returns the launch's hipError_t.
extern "C" int bench_read_probe(const void* buf, uint64_t bytes, uint32_t* out, int groups,
                                hipStream_t stream) {
  if (buf == nullptr || out == nullptr || groups <= 0 || bytes < 16) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_read_probe, dim3((unsigned)groups), dim3(kThreads), 0, stream,
                     (const u32x4*)buf, bytes / 16, out);
  return (int)hipGetLastError();
}
