// Internal declarations shared by the translation units of librfq (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace rfq {

// Devices the library tracks (the C ABI rejects higher device indices).
constexpr int kMaxDevices = 64;

// Raises a kernel's dynamic-LDS limit to `bytes` on the current device, once
// per device (`done` is the caller's per-kernel flag array).
inline hipError_t set_lds_limit(std::atomic<bool> (&done)[kMaxDevices], const void *kern,
                                int bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (!done[dev].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    done[dev].store(true, std::memory_order_release);
  }
  return hipSuccess;
}

// Elements handled by one thread of the streaming kernels (a quarter block).
constexpr int kChunk = 8;
// MX block length along K.
constexpr int kBlock = 32;

// Streaming quantizer: nelem elements (multiple of 32) of bf16 or fp32 input
// in flat row-major order.  r_codes == nullptr selects the primary code only.
hipError_t launch_quantize(const void *x, bool bf16_in, int64_t nelem,
                           uint8_t *q_codes, uint8_t *q_scales,
                           uint8_t *r_codes, uint8_t *r_scales,
                           hipStream_t stream);

// h = bf16(silu(g) * u) followed by the quantizer above.
hipError_t launch_swiglu_quantize(const void *g, const void *u, bool bf16_in,
                                  int64_t nelem, uint8_t *q_codes,
                                  uint8_t *q_scales, uint8_t *r_codes,
                                  uint8_t *r_scales, uint16_t *h_out,
                                  hipStream_t stream);

// codes/scales -> fp32, nelem a multiple of 32.
hipError_t launch_dequant(const uint8_t *codes, const uint8_t *scales,
                          int64_t nelem, float *out, hipStream_t stream);

// RFQ product (r_codes == nullptr: primary contraction only).  Picks the
// few-row, large-tile or general kernel; with a workspace (work, 16-byte
// aligned, work_bytes long) the large-tile kernel splits K where
// splitk_plan() says so and the workspace holds the partials.
hipError_t launch_gemm(const uint8_t *q_codes, const uint8_t *q_scales,
                       const uint8_t *r_codes, const uint8_t *r_scales,
                       const uint8_t *w_codes, const uint8_t *w_scales,
                       int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                       hipStream_t stream, float *work = nullptr, int64_t work_bytes = 0);
// Workspace bytes launch_gemm splits K with for this shape (0: no split),
// assuming 16-byte aligned scale tensors.
int64_t gemm_split_bytes(int64_t M, int64_t N, int64_t K);

// Large-tile product: K a multiple of 512, 16-byte aligned scale tensors and
// code tensors below 4 GiB.
bool gemm_large_applies(const uint8_t *q_scales, const uint8_t *r_scales,
                        const uint8_t *w_scales, int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_large(const uint8_t *q_codes, const uint8_t *q_scales,
                             const uint8_t *r_codes, const uint8_t *r_scales,
                             const uint8_t *w_codes, const uint8_t *w_scales,
                             int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                             hipStream_t stream);

// Split of K for the large-tile product's 128-wide tiles: `parts` ranges of
// ksplit columns (a multiple of 512), fp32 partials in work_bytes of
// workspace; parts == 1: no split.  parts_wanted <= 0 takes the library's
// choice for the shape.
struct SplitPlan {
  int parts;
  int64_t ksplit;
  int64_t work_bytes;
  bool few_rows = false;  // HiF4: the split runs the few-row kernel
  bool decode_w = false;  // HiF4: no split; W decoded to bf16 in the workspace
};
SplitPlan splitk_plan(int64_t M, int64_t N, int64_t K, int parts_wanted = 0);
// The product with the plan's split (work: plan.work_bytes of device memory,
// 16-byte aligned); with parts == 1 the same as launch_gemm_large.
hipError_t launch_gemm_large_split(const uint8_t *q_codes, const uint8_t *q_scales,
                                   const uint8_t *r_codes, const uint8_t *r_scales,
                                   const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                                   int64_t N, int64_t K, void *z, bool z_bf16,
                                   const SplitPlan &plan, float *work, hipStream_t stream);

// Z = the sum of parts fp32 partial products work[parts][mn], added in the
// order 0, 1, ..., rounded to bf16 or kept in fp32.
hipError_t launch_splitk_sum(const float *work, int parts, int64_t mn, void *z, bool z_bf16,
                             hipStream_t stream);

// launch_gemm with the library's static device scratch array as the split
// product's workspace (no allocation); static_scratch_bytes() is its size.
int64_t static_scratch_bytes();
hipError_t launch_gemm_static_scratch(const uint8_t *q_codes, const uint8_t *q_scales,
                                      const uint8_t *r_codes, const uint8_t *r_scales,
                                      const uint8_t *w_codes, const uint8_t *w_scales,
                                      int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                                      hipStream_t stream);

// Between 65 and kSkinnyMaxRows rows the large-tile kernel's 128-wide tiles
// are faster than the few-row kernel once there are at least 96 column tiles
// (N > 12160): measured 0.45-0.77 of its time at 80-128 rows and N = 12288,
// 13824 and 24576; 1.3-3x slower at N = 4096-5120, where one row of tiles
// occupies 32-40 CUs.
bool large_tiles_beat_few_rows(int64_t M, int64_t N);

// Product for few activation rows (M <= kSkinnyMaxRows, K a multiple of 512,
// 16-byte aligned scale tensors, code tensors below 2 GiB): one workgroup per
// 16, 32 or 64 weight rows and up to 64 activation rows.
constexpr int64_t kSkinnyMaxRows = 128;
// Where it runs 64 weight rows per workgroup (5-64 activation rows at
// 11264 <= N < 16384, 33-64 rows from N = 16384).
bool skinny_four_fragments(int64_t M, int64_t N);
bool gemm_skinny_applies(const uint8_t *q_scales, const uint8_t *r_scales,
                         const uint8_t *w_scales, int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_skinny(const uint8_t *q_codes, const uint8_t *q_scales,
                              const uint8_t *r_codes, const uint8_t *r_scales,
                              const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                              int64_t N, int64_t K, void *z, bool z_bf16, hipStream_t stream);
// Whether the few-row kernel's grid for this shape holds between one and two
// workgroups per CU (so some CUs run two and the rest one).
bool skinny_grid_uneven(int64_t M, int64_t N);
// Parts of K the few-row kernel splits into when given a workspace of
// parts * M * N fp32 partials (1: no split), and that split product: the
// kernel writes the partials to work, launch_splitk_sum adds them.
int skinny_split_parts(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_skinny_split(const uint8_t *q_codes, const uint8_t *q_scales,
                                    const uint8_t *r_codes, const uint8_t *r_scales,
                                    const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                                    int64_t N, int64_t K, void *z, bool z_bf16, int parts,
                                    float *work, hipStream_t stream);

// Streaming form of the product: X[M][K] (bf16 or fp32) is quantized inside
// the product's K loop (primary and, with residual, the quantized residual);
// K a multiple of 512, W's scale tensor 16-byte aligned.
hipError_t launch_gemm_stream(const void *x, bool x_bf16, bool residual, const uint8_t *w_codes,
                              const uint8_t *w_scales, int64_t M, int64_t N, int64_t K, void *z,
                              bool z_bf16, hipStream_t stream);

// RFQ product with a fallback-indicator map phi[ceil(M/64)][ceil(K/256)]
// (residual operand required; K up to 2^20): the residual term of a tile is
// included where its byte is nonzero.
hipError_t launch_gemm_phi(const uint8_t *q_codes, const uint8_t *q_scales,
                           const uint8_t *r_codes, const uint8_t *r_scales,
                           const uint8_t *w_codes, const uint8_t *w_scales, const uint8_t *phi,
                           int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                           hipStream_t stream);
hipError_t launch_gemm_large_phi(const uint8_t *q_codes, const uint8_t *q_scales,
                                 const uint8_t *r_codes, const uint8_t *r_scales,
                                 const uint8_t *w_codes, const uint8_t *w_scales,
                                 const uint8_t *phi, int64_t M, int64_t N, int64_t K, void *z,
                                 bool z_bf16, hipStream_t stream);

// phi map by rule 0 (residual codes not all zero) or 1 (a primary scale
// byte >= threshold) over the same tiles.
hipError_t launch_fallback_map(const uint8_t *r_codes, const uint8_t *q_scales, int64_t M,
                               int64_t K, int rule, int threshold, uint8_t *phi,
                               hipStream_t stream);

// Gate/up product of interleaved weights [2 Nh][K] with the SwiGLU + RFQ
// quantizer in its epilogue (large-tile conditions must hold); writes the
// codes of h [M][Nh] (hr_codes == nullptr: primary only) and optionally h.
hipError_t launch_gemm_swiglu(const uint8_t *q_codes, const uint8_t *q_scales,
                              const uint8_t *r_codes, const uint8_t *r_scales,
                              const uint8_t *wgu_codes, const uint8_t *wgu_scales,
                              int64_t M, int64_t Nh, int64_t K, uint8_t *hq_codes,
                              uint8_t *hq_scales, uint8_t *hr_codes, uint8_t *hr_scales,
                              uint16_t *h_out, hipStream_t stream);

// HiF4 quantizer (nelem a multiple of 64; r_codes == nullptr: primary only),
// dequantization and RFQ product (K a multiple of 64); metadata words are
// uint32 per 64-element block.
hipError_t launch_hif4_quantize(const void *x, bool bf16_in, int64_t nelem, uint8_t *q_codes,
                                uint32_t *q_meta, uint8_t *r_codes, uint32_t *r_meta,
                                hipStream_t stream);
hipError_t launch_hif4_dequant(const uint8_t *codes, const uint32_t *meta, int64_t nelem,
                               void *out, bool bf16_out, hipStream_t stream);
// w_bf16 != nullptr: weights given as bf16 values [N][K] (w_codes, w_meta unused).
hipError_t launch_hif4_gemm(const uint8_t *q_codes, const uint32_t *q_meta,
                            const uint8_t *r_codes, const uint32_t *r_meta,
                            const uint8_t *w_codes, const uint32_t *w_meta,
                            const uint16_t *w_bf16, int64_t M, int64_t N, int64_t K, void *z,
                            bool z_bf16, hipStream_t stream);
// Split of K for the HiF4 tile product's 128-wide tiles (ksplit a multiple
// of 64); parts == 1: no split (the shape runs the few-row kernel, or its
// tiles fill the chip, or K is short).
SplitPlan hif4_split_plan(int64_t M, int64_t N, int64_t K);
// launch_hif4_gemm (codes form) with the plan's split where work_bytes
// covers it (work: 16-byte aligned device memory), else unsplit.
hipError_t launch_hif4_gemm_split(const uint8_t *q_codes, const uint32_t *q_meta,
                                  const uint8_t *r_codes, const uint32_t *r_meta,
                                  const uint8_t *w_codes, const uint32_t *w_meta, int64_t M,
                                  int64_t N, int64_t K, void *z, bool z_bf16, float *work,
                                  int64_t work_bytes, hipStream_t stream);

// Register-only loop of FP4 scaled MFMAs (measurement support):
// kMfmaLoopWorkgroups workgroups of 512 work items, each wave issuing
// 8 * iters 32x32x64 MFMAs; sink receives one float per work item.
constexpr int kMfmaLoopWorkgroups = 256;
hipError_t launch_mfma_fp4_loop(int64_t iters, bool random_operands, float *sink,
                                hipStream_t stream);
// The same loop of bf16 MFMAs (32x32x16), same grid and sink.
hipError_t launch_mfma_bf16_loop(int64_t iters, bool random_operands, float *sink,
                                 hipStream_t stream);

}  // namespace rfq
