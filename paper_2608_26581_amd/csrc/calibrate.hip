// Measurement support: a register-only loop of FP4 scaled MFMAs on every CU,
// the sustained matrix-core rate against which the product's time is read.
// Same instruction (v_mfma_scale_f32_32x32x64_f8f6f4, E2M1 operands), same
// workgroup shape (8 waves, two per SIMD, one workgroup per CU) and the same
// accumulator pattern per wave (2 x 4 fragments of 32 x 32, each weight
// fragment meeting both activation fragments) as the large-tile product, but
// no memory traffic: the operands stay in registers.  The power drawn, and so
// the clock the chip holds, depends on the operand bits, hence two modes:
// random bits (as quantized data) or one constant code.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm_common.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

constexpr int kLoopThreads = 512;

__device__ __forceinline__ uint32_t mix(uint32_t h) {
  h ^= h >> 16;
  h *= 0x7feb352du;
  h ^= h >> 15;
  h *= 0x846ca68bu;
  h ^= h >> 16;
  return h;
}

__global__ __launch_bounds__(kLoopThreads, 2) void mfma_fp4_loop_kernel(int64_t iters, int random,
                                                                       float *__restrict__ sink) {
  const uint32_t gid = blockIdx.x * kLoopThreads + threadIdx.x;
  auto operand = [&](uint32_t salt) {
    v8i v = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] = random ? (int)mix(gid * 97u + salt * 8u + e + 1u) : 0x22222222;   // 0x2: 1.0
    return v;
  };
  v8i w[4], a[2];
#pragma unroll
  for (int j = 0; j < 4; ++j) w[j] = operand(j);
#pragma unroll
  for (int i = 0; i < 2; ++i) a[i] = operand(4 + i);
  v16f acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v16f{};
  constexpr int kScaleOne = 127;   // E8M0 byte of 1.0
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            w[j], a[i], acc[i][j], kFmtFp4, kFmtFp4, 0, kScaleOne, 0, kScaleOne);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) s += acc[i][j][e];
  sink[gid] = s;
}

// The same loop on the bf16 matrix cores that the HiF4 product runs on
// (v_mfma_f32_32x32x16_bf16, 2 x 4 accumulators of 32 x 32 per wave).  Random
// operands are finite bf16 values: random sign and 7 mantissa bits, exponent
// 0x7E or 0x7F (magnitudes in [0.5, 2)); constant operands are 1.0.
typedef __bf16 v8bf_t __attribute__((ext_vector_type(8)));

__global__ __launch_bounds__(kLoopThreads, 2) void mfma_bf16_loop_kernel(int64_t iters, int random,
                                                                        float *__restrict__ sink) {
  const uint32_t gid = blockIdx.x * kLoopThreads + threadIdx.x;
  auto operand = [&](uint32_t salt) {
    uint32_t v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t h = mix(gid * 97u + salt * 8u + e + 1u);
      // Two bf16 halves: sign, the exponent's lowest bit and the mantissa
      // from h, the exponent's upper bits 0111111 (exponent 0x7E or 0x7F).
      v[e] = random ? (h & 0x80FF80FFu) | 0x3F003F00u : 0x3F803F80u;
    }
    return __builtin_bit_cast(v8bf_t, u32x4{v[0], v[1], v[2], v[3]});
  };
  v8bf_t w[4], a[2];
#pragma unroll
  for (int j = 0; j < 4; ++j) w[j] = operand(j);
#pragma unroll
  for (int i = 0; i < 2; ++i) a[i] = operand(4 + i);
  v16f acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v16f{};
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w[j], a[i], acc[i][j], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) s += acc[i][j][e];
  sink[gid] = s;
}

}  // namespace

hipError_t launch_mfma_bf16_loop(int64_t iters, bool random_operands, float *sink,
                                 hipStream_t stream) {
  mfma_bf16_loop_kernel<<<dim3(kMfmaLoopWorkgroups), dim3(kLoopThreads), 0, stream>>>(
      iters, random_operands ? 1 : 0, sink);
  return hipGetLastError();
}

hipError_t launch_mfma_fp4_loop(int64_t iters, bool random_operands, float *sink,
                                hipStream_t stream) {
  mfma_fp4_loop_kernel<<<dim3(kMfmaLoopWorkgroups), dim3(kLoopThreads), 0, stream>>>(
      iters, random_operands ? 1 : 0, sink);
  return hipGetLastError();
}

}  // namespace rfq
