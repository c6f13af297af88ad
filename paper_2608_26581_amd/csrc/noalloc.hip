// rfq_gemm_split without a workspace argument, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid allocation): the split product's fp32 partials go to
// a file-scope device array of kScratchBytes instead.  Every GPU the library
// runs on holds its own copy of the array from the module's load until the
// process ends.  Calls that overlap on one GPU (other streams, other host
// threads) share the array and race; calls in one stream are ordered.  The
// split kernel writes every partial it later adds, so nothing needs clearing
// between calls.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "rfq_internal.h"

namespace {

// The largest workspace the split plan asks for (parts x tiles <= 512 tiles
// of 128 x 128 fp32 partials).
constexpr int64_t kScratchBytes = int64_t(32) << 20;

static __device__ __align__(256) float scratch[kScratchBytes / 4];

// Device address of `scratch` per device, looked up on the first call on
// that device (with it current).  In host code the array's name is only a
// handle for the lookup, never an address to pass on.
std::atomic<void *> g_scratch[rfq::kMaxDevices];

hipError_t scratch_address(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= rfq::kMaxDevices) return hipErrorInvalidDevice;
  void *p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return hipSuccess;
}

}  // namespace

namespace rfq {

int64_t static_scratch_bytes() { return kScratchBytes; }

hipError_t launch_gemm_static_scratch(const uint8_t *q_codes, const uint8_t *q_scales,
                                      const uint8_t *r_codes, const uint8_t *r_scales,
                                      const uint8_t *w_codes, const uint8_t *w_scales,
                                      int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                                      hipStream_t stream) {
  void *p = nullptr;
  const hipError_t e = scratch_address(&p);
  if (e != hipSuccess) return e;
  return launch_gemm(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, z_bf16,
                     stream, static_cast<float *>(p), kScratchBytes);
}

}  // namespace rfq
