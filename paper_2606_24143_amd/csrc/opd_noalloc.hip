// The loss entry point for callers that cannot allocate device memory (code
// under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc).  It runs exactly what opd_loss_fwd_bwd runs; the only kernels
// that need memory beyond inputs and outputs are the split-vocabulary ones,
// whose per-(row, chunk) statistics records go to a static device array held
// by the library instead of a caller workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/opd.h"
#include "opd_internal.h"

namespace {

constexpr size_t kScratchBytes = OPD_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch holds whole 256-byte blocks");

// One copy per GPU, alive until the process ends.  In host code this name is
// a host-side stand-in: kernels get the device address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, once looked up

// The current device's address of `scratch`, looked up on the first call on
// that device (with it current).  Returns nullptr if HIP reports an error.
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> g(g_lock);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" {

size_t opd_noalloc_scratch_bytes(void) { return kScratchBytes; }

int opd_loss_fwd_bwd_noalloc(const void* logits, int32_t dtype, int64_t N, int64_t V, int64_t ld,
                             const opd_cache* cache, int32_t estimator, int32_t k, int32_t M,
                             const uint8_t* mask, const opd_opts* opts, float* loss,
                             void* dlogits, float* lse_out, float* gathered_out,
                             float* coverage_out, void* stream) {
  return opd::loss_call(logits, dtype, N, V, ld, cache, estimator, k, M, mask, opts, loss, dlogits,
                        lse_out, gathered_out, coverage_out, nullptr, 0, scratch_ptr,
                        kScratchBytes, stream);
}

}  // extern "C"
