// Device helpers shared by the RFQ product kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rfq {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
// Native 16-byte vector (HIP's uint4 is a struct that copies through memcpy,
// which keeps staging arrays out of registers).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kFmtFp4 = 4;   // E2M1 operand format code of the scaled MFMA

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// bf16 round to nearest even of two finite fp32 values, a in the low half:
// one hardware conversion (v_cvt_pk_bf16_f32) for the pair.  It gives the
// same bits as rounding the fp32 pattern by integer arithmetic (checked on
// the GPU for every exponent, both signs, the patterns around every tie and
// subnormals).
__device__ __forceinline__ uint32_t bf16x2_rne(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// bf16 round to nearest even of a finite fp32 value (16-bit pattern).
__device__ __forceinline__ uint32_t bf16_rne(float f) { return bf16x2_rne(f, 0.0f) & 0xFFFFu; }

// Output-tile order: tiles handed to one XCD (workgroups are dealt to the 8
// XCDs round robin) are made contiguous, then walked in groups of GM tile
// rows so that concurrently running tiles share operand rows in that XCD's L2.
template <int GM>
__device__ __forceinline__ void tile_coords(int bid, int ntm, int ntn, int &tm, int &tn) {
  const int ntiles = ntm * ntn;
  int t = bid;
  if ((ntiles & 7) == 0) t = (t & 7) * (ntiles >> 3) + (t >> 3);
  const int group = t / (GM * ntn);
  const int first_m = group * GM;
  const int gsize = min(ntm - first_m, GM);
  const int in_group = t - group * GM * ntn;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

}  // namespace rfq
