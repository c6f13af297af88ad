// MXFP4 element arithmetic shared by the quantizer kernels and the fused
// SwiGLU epilogue of the product, so that both produce the same bits.
//
// Element conversion uses the gfx950 scaled FP4 conversions: the convert to
// FP4 divides by the scale 2^(byte-127), rounds to nearest-even, saturates at
// +-6 and keeps the sign of zero; the convert from FP4 multiplies by the scale
// exactly.  Within a byte the element with the lower index is the low nibble.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rfq {

typedef float f32x2 __attribute__((ext_vector_type(2)));

// E8M0 byte of a block whose largest magnitude is amax (Eq. 3 with the OCP
// offset): floor(log2 amax) - 2 + 127 is the biased exponent field minus 2;
// blocks with amax < 2^-125 (zero and subnormal included) clamp to byte 0.
__device__ __forceinline__ uint32_t scale_byte(float amax) {
  const uint32_t e = __float_as_uint(amax) >> 23;
  return e > 2u ? e - 2u : 0u;
}

// Scale operand of the scaled conversions: a float whose exponent field is
// the E8M0 byte.
__device__ __forceinline__ float scale_operand(uint32_t byte) {
  return __uint_as_float(byte << 23);
}

// Codes of 4 consecutive elements (16 bits: byte 0 holds v[0], v[1]).
__device__ __forceinline__ uint32_t encode4(float v0, float v1, float v2, float v3, float s) {
  uint32_t c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, v0, v1, s, 0);
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, v2, v3, s, 1);
}

// Codes of 8 consecutive elements (32 bits).
__device__ __forceinline__ uint32_t encode8(const float (&v)[8], float s) {
  uint32_t c = 0;
  c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, v[0], v[1], s, 0);
  c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, v[2], v[3], s, 1);
  c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, v[4], v[5], s, 2);
  c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, v[6], v[7], s, 3);
  return c;
}

// Values of the 4 elements in the low 16 bits of c.
__device__ __forceinline__ void decode4(uint32_t c, float s, float (&d)[4]) {
  const f32x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, s, 0);
  const f32x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, s, 1);
  d[0] = p0[0]; d[1] = p0[1]; d[2] = p1[0]; d[3] = p1[1];
}

__device__ __forceinline__ void decode8(uint32_t c, float s, float (&d)[8]) {
  const f32x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, s, 0);
  const f32x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, s, 1);
  const f32x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, s, 2);
  const f32x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, s, 3);
  d[0] = p0[0]; d[1] = p0[1]; d[2] = p1[0]; d[3] = p1[1];
  d[4] = p2[0]; d[5] = p2[1]; d[6] = p3[0]; d[7] = p3[1];
}

// bf16 round to nearest even of a finite fp32 value, returned as the bf16
// value widened back to fp32 bits (low 16 bits zero).
__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
}

// SwiGLU intermediate of one element before its bf16 rounding: silu(g) * u,
// silu(g) = g / (1 + exp(-g)), fp32 arithmetic; g and u are bf16 values.
__device__ __forceinline__ float swiglu_f32(float g, float u) {
  const float silu = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
  return silu * u;
}

// bf16(silu(g) * u), returned as fp32 bits.
__device__ __forceinline__ uint32_t swiglu_bits(float g, float u) {
  return bf16_rne_bits(swiglu_f32(g, u));
}

}  // namespace rfq
