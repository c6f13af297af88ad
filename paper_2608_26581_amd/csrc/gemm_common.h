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

// bf16 round to nearest even of a finite fp32 value (16-bit pattern).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Stores the four consecutive outputs Z[m][n .. n+3] a lane holds after a
// 16x16 block-scaled MFMA (weights as the A operand).  Bounds: m < M is the
// caller's; columns past N are dropped.
template <bool ZBF16>
__device__ __forceinline__ void store4(void *__restrict__ z, int64_t m, int64_t n,
                                       int64_t N, bool vec_ok, const v4f &a) {
  if constexpr (ZBF16) {
    uint16_t *zp = reinterpret_cast<uint16_t *>(z) + m * N + n;
    if (vec_ok && n + 3 < N) {
      uint2 w;
      w.x = bf16_rne(a[0]) | (bf16_rne(a[1]) << 16);
      w.y = bf16_rne(a[2]) | (bf16_rne(a[3]) << 16);
      *reinterpret_cast<uint2 *>(zp) = w;
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (n + v < N) zp[v] = (uint16_t)bf16_rne(a[v]);
    }
  } else {
    float *zp = reinterpret_cast<float *>(z) + m * N + n;
    if (vec_ok && n + 3 < N) {
      *reinterpret_cast<float4 *>(zp) = make_float4(a[0], a[1], a[2], a[3]);
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (n + v < N) zp[v] = a[v];
    }
  }
}

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
