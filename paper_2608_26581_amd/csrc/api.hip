// C ABI of librfq: host-side argument validation and kernel dispatch.
// Every check that can be made on the host runs before the first HIP call,
// so argument errors are reported without touching a device.  Order: dtype,
// shape, empty work (a no-op whose pointers are not read and may be NULL),
// pointers, alignment, device.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#include "rfq.h"
#include "rfq_internal.h"

namespace {

constexpr int kAbiVersion = 1;
using rfq::kMaxDevices;

// Per-device result of the architecture check: 0 unknown, 1 gfx950, 2 other.
std::atomic<int> g_arch_state[kMaxDevices];

bool aligned(const void *p, uintptr_t a) {
  return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0;
}

bool valid_dtype(rfq_dtype d) { return d == RFQ_F32 || d == RFQ_BF16; }

// Size limits.  K is capped so that every byte count and stage counter below
// stays in range; a launch's work-item count (grid times workgroup) must fit
// 32 bits; dequantization and the phi map loop over their grid, so only
// int64 overflow bounds them.
constexpr int64_t kMaxK = int64_t(1) << 31;
constexpr int64_t kMaxWorkItems = UINT32_MAX;
constexpr int64_t kMaxElements = int64_t(1) << 56;

// a * b > limit for a, b >= 0, computed without overflow.
bool exceeds(int64_t a, int64_t b, int64_t limit) { return a != 0 && b > limit / a; }

rfq_status check_k(int64_t rows, int64_t K) {
  if (rows < 0 || K < 32 || (K % 32) != 0 || K > kMaxK) return RFQ_ERR_SHAPE;
  return RFQ_OK;
}

// Quantizers: one 64-lane wave per 64 MX blocks, so the launch covers the
// block count rounded up to 64.
bool quantizer_fits(int64_t rows, int64_t K) {
  return !exceeds(rows, K / 32, kMaxWorkItems - 63);
}

// Products: one workgroup per output tile, 128 x 128 tiles of 256 work items
// (general kernel) or 256 x 256 tiles of 512 (large-tile kernel).  With M
// and N below 2^31 neither product overflows.
bool product_fits(int64_t M, int64_t N) {
  if (M > INT32_MAX || N > INT32_MAX) return false;
  const int64_t general = ((M + 127) / 128) * ((N + 127) / 128) * 256;
  const int64_t large = ((M + 255) / 256) * ((N + 255) / 256) * 512;
  return general <= kMaxWorkItems && large <= kMaxWorkItems;
}

// HiF4 calls: K a positive multiple of 64 (one metadata word per 64-element
// block).  The quantizer runs 256 work items per 128 blocks.  The product
// runs one workgroup per 128 x 256 output tile (up to 768 work items: eight
// producer waves with the residual, four consumers) or per 128 x 128 tile
// (up to 640); both grids must fit, whichever the dispatch picks.
rfq_status check_k64(int64_t rows, int64_t K) {
  if (rows < 0 || K < 64 || (K % 64) != 0 || K > kMaxK) return RFQ_ERR_SHAPE;
  return RFQ_OK;
}
bool hif4_quantizer_fits(int64_t rows, int64_t K) {
  return !exceeds(rows, K / 64, (kMaxWorkItems / 256) * 128);
}
bool hif4_product_fits(int64_t M, int64_t N) {
  if (M > INT32_MAX || N > INT32_MAX) return false;
  const int64_t rows = (M + 127) / 128;
  return rows * ((N + 255) / 256) * 768 <= kMaxWorkItems &&
         rows * ((N + 127) / 128) * 640 <= kMaxWorkItems;
}

// Confirms that the current device is a gfx950 GPU (cached per device).
rfq_status check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return RFQ_ERR_DEVICE;
  if (dev >= kMaxDevices) return RFQ_ERR_DEVICE;
  int st = g_arch_state[dev].load(std::memory_order_acquire);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return RFQ_ERR_DEVICE;
    st = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    g_arch_state[dev].store(st, std::memory_order_release);
  }
  return st == 1 ? RFQ_OK : RFQ_ERR_DEVICE;
}

rfq_status launched(hipError_t e) { return e == hipSuccess ? RFQ_OK : RFQ_ERR_LAUNCH; }

}  // namespace

extern "C" {

rfq_status rfq_quantize_act(const void *x, rfq_dtype x_dtype, int64_t M, int64_t K,
                            uint8_t *q_codes, uint8_t *q_scales,
                            uint8_t *r_codes, uint8_t *r_scales,
                            void *hip_stream) {
  if (!valid_dtype(x_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (!quantizer_fits(M, K)) return RFQ_ERR_SHAPE;
  if (M == 0) return RFQ_OK;
  if (!x || !q_codes || !q_scales) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_scales == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(x, 16) || !aligned(q_codes, 16) || (r_codes && !aligned(r_codes, 16)))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_quantize(x, x_dtype == RFQ_BF16, M * K, q_codes, q_scales,
                                       r_codes, r_scales,
                                       static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_quantize_weight(const void *w, rfq_dtype w_dtype, int64_t N, int64_t K,
                               uint8_t *w_codes, uint8_t *w_scales,
                               void *hip_stream) {
  if (!valid_dtype(w_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(N, K);
  if (s != RFQ_OK) return s;
  if (!quantizer_fits(N, K)) return RFQ_ERR_SHAPE;
  if (N == 0) return RFQ_OK;
  if (!w || !w_codes || !w_scales) return RFQ_ERR_NULL;
  if (!aligned(w, 16) || !aligned(w_codes, 16)) return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_quantize(w, w_dtype == RFQ_BF16, N * K, w_codes, w_scales,
                                       nullptr, nullptr,
                                       static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_gemm(const uint8_t *q_codes, const uint8_t *q_scales,
                    const uint8_t *r_codes, const uint8_t *r_scales,
                    const uint8_t *w_codes, const uint8_t *w_scales,
                    int64_t M, int64_t N, int64_t K,
                    void *z, rfq_dtype z_dtype, void *hip_stream) {
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || !product_fits(M, N)) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_scales || !w_codes || !w_scales || !z) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_scales == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(w_codes, 16) || (r_codes && !aligned(r_codes, 16)) ||
      !aligned(z, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_gemm(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales,
                                   M, N, K, z, z_dtype == RFQ_BF16,
                                   static_cast<hipStream_t>(hip_stream)));
}

int64_t rfq_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (check_k(M, K) != RFQ_OK || N < 0 || !product_fits(M, N)) return 0;
  return rfq::gemm_split_bytes(M, N, K);
}

rfq_status rfq_gemm_split(const uint8_t *q_codes, const uint8_t *q_scales,
                          const uint8_t *r_codes, const uint8_t *r_scales,
                          const uint8_t *w_codes, const uint8_t *w_scales, int64_t M, int64_t N,
                          int64_t K, void *z, rfq_dtype z_dtype, void *workspace,
                          int64_t workspace_bytes, void *hip_stream) {
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || !product_fits(M, N) || workspace_bytes < 0) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_scales || !w_codes || !w_scales || !z) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_scales == nullptr)) return RFQ_ERR_NULL;
  if (!workspace && workspace_bytes > 0) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(w_codes, 16) || (r_codes && !aligned(r_codes, 16)) ||
      !aligned(z, 16) || !aligned(workspace, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_gemm(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales,
                                   M, N, K, z, z_dtype == RFQ_BF16,
                                   static_cast<hipStream_t>(hip_stream),
                                   static_cast<float *>(workspace), workspace_bytes));
}

rfq_status rfq_gemm_split_noalloc(const uint8_t *q_codes, const uint8_t *q_scales,
                                  const uint8_t *r_codes, const uint8_t *r_scales,
                                  const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                                  int64_t N, int64_t K, void *z, rfq_dtype z_dtype,
                                  void *hip_stream) {
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || !product_fits(M, N)) return RFQ_ERR_SHAPE;
  if (rfq::gemm_split_bytes(M, N, K) > rfq::static_scratch_bytes()) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_scales || !w_codes || !w_scales || !z) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_scales == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(w_codes, 16) || (r_codes && !aligned(r_codes, 16)) ||
      !aligned(z, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_gemm_static_scratch(q_codes, q_scales, r_codes, r_scales, w_codes,
                                                  w_scales, M, N, K, z, z_dtype == RFQ_BF16,
                                                  static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_dequant(const uint8_t *codes, const uint8_t *scales, int64_t rows,
                       int64_t K, float *out, void *hip_stream) {
  rfq_status s = check_k(rows, K);
  if (s != RFQ_OK) return s;
  if (exceeds(rows, K, kMaxElements)) return RFQ_ERR_SHAPE;
  if (rows == 0) return RFQ_OK;
  if (!codes || !scales || !out) return RFQ_ERR_NULL;
  if (!aligned(codes, 16) || !aligned(out, 16)) return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_dequant(codes, scales, rows * K, out,
                                      static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_swiglu_quantize_act(const void *g, const void *u, rfq_dtype dt,
                                   int64_t M, int64_t Nh,
                                   uint8_t *q_codes, uint8_t *q_scales,
                                   uint8_t *r_codes, uint8_t *r_scales,
                                   void *h_out, void *hip_stream) {
  if (!valid_dtype(dt)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, Nh);
  if (s != RFQ_OK) return s;
  if (!quantizer_fits(M, Nh)) return RFQ_ERR_SHAPE;
  if (M == 0) return RFQ_OK;
  if (!g || !u || !q_codes || !q_scales) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_scales == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(g, 16) || !aligned(u, 16) || !aligned(q_codes, 16) ||
      (r_codes && !aligned(r_codes, 16)) || (h_out && !aligned(h_out, 16)))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_swiglu_quantize(g, u, dt == RFQ_BF16, M * Nh, q_codes, q_scales,
                                              r_codes, r_scales,
                                              static_cast<uint16_t *>(h_out),
                                              static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_gemm_phi(const uint8_t *q_codes, const uint8_t *q_scales,
                        const uint8_t *r_codes, const uint8_t *r_scales,
                        const uint8_t *w_codes, const uint8_t *w_scales, const uint8_t *phi,
                        int64_t M, int64_t N, int64_t K, void *z, rfq_dtype z_dtype,
                        void *hip_stream) {
  if (!phi || !r_codes)
    return rfq_gemm(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z,
                    z_dtype, hip_stream);
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || K > (int64_t(1) << 20) || !product_fits(M, N)) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_scales || !r_scales || !w_codes || !w_scales || !z) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(w_codes, 16) || !aligned(r_codes, 16) ||
      !aligned(z, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_gemm_phi(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales,
                                       phi, M, N, K, z, z_dtype == RFQ_BF16,
                                       static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_fallback_map(const uint8_t *r_codes, const uint8_t *q_scales, int64_t M,
                            int64_t K, int rule, int threshold, uint8_t *phi,
                            void *hip_stream) {
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (rule != RFQ_PHI_RESIDUAL_NONZERO && rule != RFQ_PHI_SCALE_AT_LEAST) return RFQ_ERR_SHAPE;
  if (exceeds(M, K, kMaxElements)) return RFQ_ERR_SHAPE;
  if (M == 0) return RFQ_OK;
  if (!phi || (rule == RFQ_PHI_RESIDUAL_NONZERO ? !r_codes : !q_scales)) return RFQ_ERR_NULL;
  if (rule == RFQ_PHI_RESIDUAL_NONZERO && !aligned(r_codes, 16)) return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_fallback_map(r_codes, q_scales, M, K, rule, threshold, phi,
                                           static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_gemm_swiglu_quantize(const uint8_t *q_codes, const uint8_t *q_scales,
                                    const uint8_t *r_codes, const uint8_t *r_scales,
                                    const uint8_t *wgu_codes, const uint8_t *wgu_scales,
                                    int64_t M, int64_t Nh, int64_t K,
                                    uint8_t *hq_codes, uint8_t *hq_scales,
                                    uint8_t *hr_codes, uint8_t *hr_scales,
                                    void *h_out, void *hip_stream) {
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (Nh < 0 || (Nh % 32) != 0 || (K % 512) != 0) return RFQ_ERR_SHAPE;
  if (Nh > INT32_MAX || !product_fits(M, 2 * Nh)) return RFQ_ERR_SHAPE;
  // Byte offsets inside each code tensor are 32-bit.
  const int64_t limit = int64_t(1) << 32;
  if (M * (K / 2) >= limit || 2 * Nh * (K / 2) >= limit) return RFQ_ERR_SHAPE;
  if (M == 0 || Nh == 0) return RFQ_OK;
  if (!q_codes || !q_scales || !wgu_codes || !wgu_scales || !hq_codes || !hq_scales)
    return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_scales == nullptr)) return RFQ_ERR_NULL;
  if ((hr_codes == nullptr) != (hr_scales == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(q_scales, 16) || !aligned(wgu_codes, 16) ||
      !aligned(wgu_scales, 16) || (r_codes && (!aligned(r_codes, 16) || !aligned(r_scales, 16))) ||
      !aligned(hq_codes, 16) || (hr_codes && !aligned(hr_codes, 16)) ||
      (h_out && !aligned(h_out, 16)))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_gemm_swiglu(q_codes, q_scales, r_codes, r_scales, wgu_codes,
                                          wgu_scales, M, Nh, K, hq_codes, hq_scales, hr_codes,
                                          hr_scales, static_cast<uint16_t *>(h_out),
                                          static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_gemm_stream(const void *x, rfq_dtype x_dtype, int residual,
                           const uint8_t *w_codes, const uint8_t *w_scales,
                           int64_t M, int64_t N, int64_t K,
                           void *z, rfq_dtype z_dtype, void *hip_stream) {
  if (!valid_dtype(x_dtype) || !valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || (K % 512) != 0) return RFQ_ERR_SHAPE;
  // One 256-work-item workgroup per 16 x 16 output block: N/16 along the
  // grid's x axis, M/16 along its y axis (at most 65535); buffer ranges (X
  // bytes, weight code bytes) are 31-bit.
  if (M > 65535 * 16 || N > kMaxWorkItems / 256 * 16) return RFQ_ERR_SHAPE;
  const int64_t limit = int64_t(1) << 31;
  const int64_t xbytes = x_dtype == RFQ_BF16 ? 2 : 4;
  if (M * K >= limit / xbytes || N * (K / 2) >= limit) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!x || !w_codes || !w_scales || !z) return RFQ_ERR_NULL;
  if (!aligned(x, 16) || !aligned(w_codes, 16) || !aligned(w_scales, 16) || !aligned(z, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_gemm_stream(x, x_dtype == RFQ_BF16, residual != 0, w_codes,
                                          w_scales, M, N, K, z, z_dtype == RFQ_BF16,
                                          static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_hif4_quantize(const void *x, rfq_dtype x_dtype, int64_t rows, int64_t K,
                             uint8_t *q_codes, uint32_t *q_meta,
                             uint8_t *r_codes, uint32_t *r_meta, void *hip_stream) {
  if (!valid_dtype(x_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k64(rows, K);
  if (s != RFQ_OK) return s;
  if (!hif4_quantizer_fits(rows, K)) return RFQ_ERR_SHAPE;
  if (rows == 0) return RFQ_OK;
  if (!x || !q_codes || !q_meta) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_meta == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(x, 16) || !aligned(q_codes, 4) || !aligned(q_meta, 4) ||
      (r_codes && (!aligned(r_codes, 4) || !aligned(r_meta, 4))))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_hif4_quantize(x, x_dtype == RFQ_BF16, rows * K, q_codes, q_meta,
                                            r_codes, r_meta,
                                            static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_hif4_dequant(const uint8_t *codes, const uint32_t *meta, int64_t rows, int64_t K,
                            void *out, rfq_dtype out_dtype, void *hip_stream) {
  if (!valid_dtype(out_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k64(rows, K);
  if (s != RFQ_OK) return s;
  if (exceeds(rows, K, kMaxElements)) return RFQ_ERR_SHAPE;
  if (rows == 0) return RFQ_OK;
  if (!codes || !meta || !out) return RFQ_ERR_NULL;
  if (!aligned(codes, 4) || !aligned(meta, 4) || !aligned(out, 16)) return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_hif4_dequant(codes, meta, rows * K, out, out_dtype == RFQ_BF16,
                                           static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_hif4_gemm(const uint8_t *q_codes, const uint32_t *q_meta,
                         const uint8_t *r_codes, const uint32_t *r_meta,
                         const uint8_t *w_codes, const uint32_t *w_meta,
                         int64_t M, int64_t N, int64_t K,
                         void *z, rfq_dtype z_dtype, void *hip_stream) {
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k64(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || !hif4_product_fits(M, N)) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_meta || !w_codes || !w_meta || !z) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_meta == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(w_codes, 16) || !aligned(q_meta, 4) ||
      !aligned(w_meta, 4) || (r_codes && (!aligned(r_codes, 16) || !aligned(r_meta, 4))) ||
      !aligned(z, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_hif4_gemm(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta,
                                        nullptr, M, N, K, z, z_dtype == RFQ_BF16,
                                        static_cast<hipStream_t>(hip_stream)));
}

int64_t rfq_hif4_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (check_k64(M, K) != RFQ_OK || N < 0 || !hif4_product_fits(M, N)) return 0;
  const rfq::SplitPlan p = rfq::hif4_split_plan(M, N, K);
  return (p.parts > 1 || p.decode_w) ? p.work_bytes : 0;
}

rfq_status rfq_hif4_gemm_split(const uint8_t *q_codes, const uint32_t *q_meta,
                               const uint8_t *r_codes, const uint32_t *r_meta,
                               const uint8_t *w_codes, const uint32_t *w_meta,
                               int64_t M, int64_t N, int64_t K,
                               void *z, rfq_dtype z_dtype, void *workspace,
                               int64_t workspace_bytes, void *hip_stream) {
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k64(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || !hif4_product_fits(M, N) || workspace_bytes < 0) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_meta || !w_codes || !w_meta || !z) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_meta == nullptr)) return RFQ_ERR_NULL;
  if (!workspace && workspace_bytes > 0) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(w_codes, 16) || !aligned(q_meta, 4) ||
      !aligned(w_meta, 4) || (r_codes && (!aligned(r_codes, 16) || !aligned(r_meta, 4))) ||
      !aligned(z, 16) || !aligned(workspace, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_hif4_gemm_split(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta,
                                              M, N, K, z, z_dtype == RFQ_BF16,
                                              static_cast<float *>(workspace), workspace_bytes,
                                              static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_hif4_gemm_wbf16(const uint8_t *q_codes, const uint32_t *q_meta,
                               const uint8_t *r_codes, const uint32_t *r_meta,
                               const void *w_bf16, int64_t M, int64_t N, int64_t K,
                               void *z, rfq_dtype z_dtype, void *hip_stream) {
  if (!valid_dtype(z_dtype)) return RFQ_ERR_DTYPE;
  rfq_status s = check_k64(M, K);
  if (s != RFQ_OK) return s;
  if (N < 0 || !hif4_product_fits(M, N)) return RFQ_ERR_SHAPE;
  if (M == 0 || N == 0) return RFQ_OK;
  if (!q_codes || !q_meta || !w_bf16 || !z) return RFQ_ERR_NULL;
  if ((r_codes == nullptr) != (r_meta == nullptr)) return RFQ_ERR_NULL;
  if (!aligned(q_codes, 16) || !aligned(q_meta, 4) || !aligned(w_bf16, 16) ||
      (r_codes && (!aligned(r_codes, 16) || !aligned(r_meta, 4))) || !aligned(z, 16))
    return RFQ_ERR_ALIGN;
  if ((s = check_device()) != RFQ_OK) return s;
  return launched(rfq::launch_hif4_gemm(q_codes, q_meta, r_codes, r_meta, nullptr, nullptr,
                                        static_cast<const uint16_t *>(w_bf16), M, N, K, z,
                                        z_dtype == RFQ_BF16,
                                        static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_mfma_fp4_loop(int64_t iters, int random_operands, float *sink,
                             void *hip_stream) {
  if (iters < 1 || iters > (int64_t(1) << 24)) return RFQ_ERR_SHAPE;
  if (!sink) return RFQ_ERR_NULL;
  if (!aligned(sink, 16)) return RFQ_ERR_ALIGN;
  rfq_status s = check_device();
  if (s != RFQ_OK) return s;
  return launched(rfq::launch_mfma_fp4_loop(iters, random_operands != 0, sink,
                                            static_cast<hipStream_t>(hip_stream)));
}

rfq_status rfq_mfma_bf16_loop(int64_t iters, int random_operands, float *sink,
                              void *hip_stream) {
  if (iters < 1 || iters > (int64_t(1) << 24)) return RFQ_ERR_SHAPE;
  if (!sink) return RFQ_ERR_NULL;
  if (!aligned(sink, 16)) return RFQ_ERR_ALIGN;
  rfq_status s = check_device();
  if (s != RFQ_OK) return s;
  return launched(rfq::launch_mfma_bf16_loop(iters, random_operands != 0, sink,
                                             static_cast<hipStream_t>(hip_stream)));
}

const char *rfq_status_str(rfq_status s) {
  switch (s) {
    case RFQ_OK: return "ok";
    case RFQ_ERR_NULL: return "null pointer (or half of an optional pair)";
    case RFQ_ERR_SHAPE: return "bad shape (negative size, K not a positive multiple of 32 (64 for HiF4), or a size limit)";
    case RFQ_ERR_DTYPE: return "unknown dtype";
    case RFQ_ERR_ALIGN: return "misaligned pointer";
    case RFQ_ERR_DEVICE: return "no gfx950 device current";
    case RFQ_ERR_LAUNCH: return "kernel launch failed";
  }
  return "unknown status";
}

int rfq_abi_version(void) { return kAbiVersion; }

}  // extern "C"
