// Streaming MXFP4 kernels for gfx950: the RFQ activation quantizer (primary
// code, Eq. 8, plus the quantized residual, Eq. 9-10), the weight quantizer,
// the fused SwiGLU + quantizer and dequantization (Eq. 12).
//
// Work decomposition: the tensor is treated as a flat array (K is a multiple
// of 32, so no MX block straddles a row and the scale index of a block is its
// flat block index).  One thread owns 8 consecutive elements; the four lanes
// of a DPP quad own one 32-element block, so the block maximum takes two
// quad-permute steps and no LDS.  A wave owns a span of 64 consecutive blocks
// and walks it in 4 steps; in step u the 16-lane row r holds blocks
// 16r + 4u .. 16r + 4u + 3, so every load of a row is 256 contiguous bytes
// and, after the steps, the row's 16 scale bytes are contiguous: two DPP
// row shifts gather a step's 4 bytes into the row's first lane, which then
// writes all 16 with one store (64 bytes per wave).  All loads are issued
// before any arithmetic.  bf16 inputs are read non-temporally; stores are
// plain (measured: non-temporal stores of these partial lines cost about a
// fifth more write traffic, and non-temporal fp32 loads were slower).
//
// Element arithmetic (scale byte, scaled FP4 conversions, SwiGLU) comes from
// mx_device.h.  The residual x - deq(q) is exact in fp32 (a nonzero E2M1
// rounding lies within a factor of two of x), so it is formed in registers
// only.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mx_device.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;   // steps per wave span of 64 blocks (4 blocks per row)

// Maximum over the four lanes of a quad (DPP quad_perm 1,0,3,2 then 2,3,0,1).
__device__ __forceinline__ float quad_max(float v) {
  float o = __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  v = fmaxf(v, o);
  o = __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  return fmaxf(v, o);
}

__device__ __forceinline__ float absmax8(const float (&v)[8]) {
  float a = fmaxf(fabsf(v[0]), fabsf(v[1]));
  a = fmaxf(a, fmaxf(fabsf(v[2]), fabsf(v[3])));
  a = fmaxf(a, fmaxf(fabsf(v[4]), fabsf(v[5])));
  return fmaxf(a, fmaxf(fabsf(v[6]), fabsf(v[7])));
}

// Quantize the 8 values a thread owns: primary code and scale byte and, with
// RES, the residual code and scale byte.  All four quad lanes must call it.
template <bool RES>
__device__ __forceinline__ void quantize8(const float (&v)[8], uint32_t &qc,
                                          uint32_t &qb, uint32_t &rc,
                                          uint32_t &rb) {
  qb = scale_byte(quad_max(absmax8(v)));
  const float qs = scale_operand(qb);
  qc = encode8(v, qs);
  if constexpr (RES) {
    float d[8], r[8];
    decode8(qc, qs, d);
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = v[i] - d[i];
    rb = scale_byte(quad_max(absmax8(r)));
    rc = encode8(r, scale_operand(rb));
  }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
static_assert(kUnroll == 4, "a wave span is 16 rows of 4 steps");

template <bool BF16_IN>
__device__ __forceinline__ void load8(const void *__restrict__ x, int64_t chunk,
                                      float (&v)[8]) {
  if constexpr (BF16_IN) {
    const u32x4 w = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(x) + chunk);
    v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xFFFF0000u);
    v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xFFFF0000u);
    v[4] = __uint_as_float(w.z << 16); v[5] = __uint_as_float(w.z & 0xFFFF0000u);
    v[6] = __uint_as_float(w.w << 16); v[7] = __uint_as_float(w.w & 0xFFFF0000u);
  } else {
    const u32x4 *p = reinterpret_cast<const u32x4 *>(x) + 2 * chunk;
    const u32x4 a = p[0];
    const u32x4 b = p[1];
    v[0] = __uint_as_float(a.x); v[1] = __uint_as_float(a.y);
    v[2] = __uint_as_float(a.z); v[3] = __uint_as_float(a.w);
    v[4] = __uint_as_float(b.x); v[5] = __uint_as_float(b.y);
    v[6] = __uint_as_float(b.z); v[7] = __uint_as_float(b.w);
  }
}

// Chunk (8 elements) of lane `lane` in step u of a wave span of 64 blocks:
// block 16r + 4u + q, elements 8j .. 8j+7 of it (lane = 16r + 4q + j).
__device__ __forceinline__ int span_chunk(int lane, int u) {
  return 4 * (16 * (lane >> 4) + 4 * u + ((lane >> 2) & 3)) + (lane & 3);
}

// Collects the scale bytes of the four quads of a 16-lane row into the
// row's first lane (byte q from quad q).
__device__ __forceinline__ uint32_t gather_row4(uint32_t b) {
  const uint32_t t = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)b, 0x104, 0xF, 0xF, false);
  const uint32_t v = b | (t << 8);                                  // row_shl:4
  const uint32_t t2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x108, 0xF, 0xF, false);
  return v | (t2 << 16);                                            // row_shl:8
}

// Writes the scale bytes of a wave span: sw[u] holds, in the first lane of
// row r, the bytes of blocks 16r + 4u .. +3.  Full spans with an aligned
// tensor use one 16-byte store per row; otherwise each quad leader writes its
// own byte (bytes[u] in every lane of the quad).
__device__ __forceinline__ void store_span_scales(uint8_t *__restrict__ scales,
                                                  int64_t span_block0, int64_t nblocks,
                                                  int lane, const uint32_t (&sw)[4],
                                                  const uint32_t (&bytes)[4]) {
  const bool full = span_block0 + 64 <= nblocks &&
                    (reinterpret_cast<uintptr_t>(scales) & 15) == 0;
  if (full) {
    if ((lane & 15) == 0) {
      u32x4 w = {sw[0], sw[1], sw[2], sw[3]};
      *reinterpret_cast<u32x4 *>(scales + span_block0 + (lane & 48)) = w;
    }
  } else if ((lane & 3) == 0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t b = span_block0 + 16 * (lane >> 4) + 4 * u + ((lane >> 2) & 3);
      if (b < nblocks) scales[b] = (uint8_t)bytes[u];
    }
  }
}

template <bool BF16_IN, bool RES>
__global__ __launch_bounds__(kThreads) void quantize_kernel(
    const void *__restrict__ x, int64_t nchunks, uint32_t *__restrict__ q_codes,
    uint8_t *__restrict__ q_scales, uint32_t *__restrict__ r_codes,
    uint8_t *__restrict__ r_scales) {
  const int lane = threadIdx.x & 63;
  const int64_t span0 = ((int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * 256;
  float v[kUnroll][8];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    // Lanes past the end load the last chunk (never out of bounds) and skip
    // their stores; nchunks is a multiple of 4, so quads stay whole.
    const int64_t ch = span0 + span_chunk(lane, u);
    load8<BF16_IN>(x, ch < nchunks ? ch : nchunks - 1, v[u]);
  }
  uint32_t qsw[kUnroll], rsw[kUnroll], qbytes[kUnroll], rbytes[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t ch = span0 + span_chunk(lane, u);
    uint32_t qc, qb, rc = 0, rb = 0;
    quantize8<RES>(v[u], qc, qb, rc, rb);
    qbytes[u] = qb;
    qsw[u] = gather_row4(qb);
    if constexpr (RES) {
      rbytes[u] = rb;
      rsw[u] = gather_row4(rb);
    }
    if (ch < nchunks) {
      q_codes[ch] = qc;
      if constexpr (RES) r_codes[ch] = rc;
    }
  }
  const int64_t nblocks = nchunks >> 2;
  store_span_scales(q_scales, span0 >> 2, nblocks, lane, qsw, qbytes);
  if constexpr (RES) store_span_scales(r_scales, span0 >> 2, nblocks, lane, rsw, rbytes);
}

template <bool BF16_IN, bool RES>
__global__ __launch_bounds__(kThreads) void swiglu_quantize_kernel(
    const void *__restrict__ g, const void *__restrict__ u, int64_t nchunks,
    uint32_t *__restrict__ q_codes, uint8_t *__restrict__ q_scales,
    uint32_t *__restrict__ r_codes, uint8_t *__restrict__ r_scales,
    u32x4 *__restrict__ h_out) {
  const int lane = threadIdx.x & 63;
  const int64_t span0 = ((int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * 256;
  float gv[kUnroll][8], uv[kUnroll][8];
#pragma unroll
  for (int i = 0; i < kUnroll; ++i) {
    const int64_t ch = span0 + span_chunk(lane, i);
    const int64_t c = ch < nchunks ? ch : nchunks - 1;
    load8<BF16_IN>(g, c, gv[i]);
    load8<BF16_IN>(u, c, uv[i]);
  }
  uint32_t qsw[kUnroll], rsw[kUnroll], qbytes[kUnroll], rbytes[kUnroll];
#pragma unroll
  for (int i = 0; i < kUnroll; ++i) {
    const int64_t ch = span0 + span_chunk(lane, i);
    float h[8];
    uint32_t hb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      hb[j] = swiglu_bits(gv[i][j], uv[i][j]);
      h[j] = __uint_as_float(hb[j]);
    }
    uint32_t qc, qb, rc = 0, rb = 0;
    quantize8<RES>(h, qc, qb, rc, rb);
    qbytes[i] = qb;
    qsw[i] = gather_row4(qb);
    if constexpr (RES) {
      rbytes[i] = rb;
      rsw[i] = gather_row4(rb);
    }
    if (ch < nchunks) {
      q_codes[ch] = qc;
      if constexpr (RES) r_codes[ch] = rc;
      if (h_out) {
        u32x4 w;
        w.x = (hb[0] >> 16) | hb[1];
        w.y = (hb[2] >> 16) | hb[3];
        w.z = (hb[4] >> 16) | hb[5];
        w.w = (hb[6] >> 16) | hb[7];
        h_out[ch] = w;
      }
    }
  }
  const int64_t nblocks = nchunks >> 2;
  store_span_scales(q_scales, span0 >> 2, nblocks, lane, qsw, qbytes);
  if constexpr (RES) store_span_scales(r_scales, span0 >> 2, nblocks, lane, rsw, rbytes);
}

__global__ __launch_bounds__(kThreads) void dequant_kernel(
    const uint32_t *__restrict__ codes, const uint8_t *__restrict__ scales,
    int64_t nchunks, float4 *__restrict__ out) {
  const int64_t ch = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (ch >= nchunks) return;
  float d[8];
  decode8(codes[ch], scale_operand(scales[ch >> 2]), d);
  out[2 * ch] = make_float4(d[0], d[1], d[2], d[3]);
  out[2 * ch + 1] = make_float4(d[4], d[5], d[6], d[7]);
}

// Fallback-indicator map over tiles of 64 rows by 256 reduction columns
// (one workgroup per tile): rule 0 marks tiles where a residual code has a
// nonzero magnitude, rule 1 tiles holding a primary scale byte >= threshold.
__global__ __launch_bounds__(kThreads) void fallback_map_kernel(
    const uint8_t *__restrict__ r_codes, const uint8_t *__restrict__ q_scales, int64_t M,
    int64_t K, int rule, int threshold, int pcols, uint8_t *__restrict__ phi) {
  const int64_t p = blockIdx.x / pcols, c = blockIdx.x % pcols;
  const int tid = threadIdx.x;
  const int64_t m = 64 * p + tid / 4;
  int flag = 0;
  if (m < M) {
    if (rule == 0) {
      const int64_t kb = K / 2;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int64_t b = 128 * c + 32 * (tid & 3) + 16 * h;
        if (b < kb) {
          const u32x4 v = *reinterpret_cast<const u32x4 *>(r_codes + m * kb + b);
          flag |= ((v.x | v.y | v.z | v.w) & 0x77777777u) != 0;
        }
      }
    } else {
      const int64_t nb = K / 32;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int64_t b = 8 * c + 2 * (tid & 3) + h;
        if (b < nb) flag |= (int)q_scales[m * nb + b] >= threshold;
      }
    }
  }
  flag = __syncthreads_or(flag);
  if (tid == 0) phi[blockIdx.x] = (uint8_t)(flag != 0);
}

inline unsigned grid_for(int64_t nchunks, int64_t per_block) {
  return (unsigned)((nchunks + per_block - 1) / per_block);
}

}  // namespace

hipError_t launch_quantize(const void *x, bool bf16_in, int64_t nelem,
                           uint8_t *q_codes, uint8_t *q_scales,
                           uint8_t *r_codes, uint8_t *r_scales,
                           hipStream_t stream) {
  const int64_t nchunks = nelem / kChunk;
  const dim3 grid(grid_for(nchunks, kThreads * kUnroll)), block(kThreads);
  uint32_t *qc = reinterpret_cast<uint32_t *>(q_codes);
  uint32_t *rc = reinterpret_cast<uint32_t *>(r_codes);
  if (bf16_in) {
    if (r_codes)
      quantize_kernel<true, true><<<grid, block, 0, stream>>>(x, nchunks, qc, q_scales, rc, r_scales);
    else
      quantize_kernel<true, false><<<grid, block, 0, stream>>>(x, nchunks, qc, q_scales, rc, r_scales);
  } else {
    if (r_codes)
      quantize_kernel<false, true><<<grid, block, 0, stream>>>(x, nchunks, qc, q_scales, rc, r_scales);
    else
      quantize_kernel<false, false><<<grid, block, 0, stream>>>(x, nchunks, qc, q_scales, rc, r_scales);
  }
  return hipGetLastError();
}

hipError_t launch_swiglu_quantize(const void *g, const void *u, bool bf16_in,
                                  int64_t nelem, uint8_t *q_codes,
                                  uint8_t *q_scales, uint8_t *r_codes,
                                  uint8_t *r_scales, uint16_t *h_out,
                                  hipStream_t stream) {
  const int64_t nchunks = nelem / kChunk;
  const dim3 grid(grid_for(nchunks, kThreads * kUnroll)), block(kThreads);
  uint32_t *qc = reinterpret_cast<uint32_t *>(q_codes);
  uint32_t *rc = reinterpret_cast<uint32_t *>(r_codes);
  u32x4 *h = reinterpret_cast<u32x4 *>(h_out);
  if (bf16_in) {
    if (r_codes)
      swiglu_quantize_kernel<true, true><<<grid, block, 0, stream>>>(g, u, nchunks, qc, q_scales, rc, r_scales, h);
    else
      swiglu_quantize_kernel<true, false><<<grid, block, 0, stream>>>(g, u, nchunks, qc, q_scales, rc, r_scales, h);
  } else {
    if (r_codes)
      swiglu_quantize_kernel<false, true><<<grid, block, 0, stream>>>(g, u, nchunks, qc, q_scales, rc, r_scales, h);
    else
      swiglu_quantize_kernel<false, false><<<grid, block, 0, stream>>>(g, u, nchunks, qc, q_scales, rc, r_scales, h);
  }
  return hipGetLastError();
}

hipError_t launch_dequant(const uint8_t *codes, const uint8_t *scales,
                          int64_t nelem, float *out, hipStream_t stream) {
  const int64_t nchunks = nelem / kChunk;
  dequant_kernel<<<grid_for(nchunks, kThreads), kThreads, 0, stream>>>(
      reinterpret_cast<const uint32_t *>(codes), scales, nchunks,
      reinterpret_cast<float4 *>(out));
  return hipGetLastError();
}

hipError_t launch_fallback_map(const uint8_t *r_codes, const uint8_t *q_scales, int64_t M,
                               int64_t K, int rule, int threshold, uint8_t *phi,
                               hipStream_t stream) {
  const int pcols = (int)((K + 255) / 256);
  const int64_t tiles = ((M + 63) / 64) * pcols;
  fallback_map_kernel<<<(unsigned)tiles, kThreads, 0, stream>>>(r_codes, q_scales, M, K, rule,
                                                                 threshold, pcols, phi);
  return hipGetLastError();
}

}  // namespace rfq
