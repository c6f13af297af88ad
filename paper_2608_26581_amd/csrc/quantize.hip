// Streaming MXFP4 kernels for gfx950: the RFQ activation quantizer (primary
// code, Eq. 8, plus the quantized residual, Eq. 9-10), the weight quantizer,
// the fused SwiGLU + quantizer and dequantization (Eq. 12).
//
// Work decomposition of the quantizers: the tensor is treated as a flat array
// (K is a multiple of 32, so no MX block straddles a row and the scale index
// of a block is its flat block index).  A wave owns a span of 64 consecutive
// blocks.  Every load instruction of the wave reads 1 KB of contiguous input,
// 16 bytes per lane: 8 bf16 elements (4 lanes per block, 4 steps per span) or
// 4 fp32 elements (8 lanes per block, 8 steps).  The block maximum is a DPP
// max over the block's lanes.  Each step writes its codes and scale bytes into
// a wave-private LDS area in the tensor's own order; after the last step each
// lane reads back the 16 code bytes of one block, so every code store of the
// wave writes 1 KB of contiguous codes with 16-byte stores, and the 64 scale
// bytes of a span leave as four 16-byte stores.  Inputs are read
// non-temporally.  Stores are non-temporal when the whole job moves more bytes
// than the 256 MB last-level cache holds, and plain otherwise (measured on
// MI355X: plain stores are slightly faster while everything fits, leaving the
// codes cached for the product that reads them next; streaming stores are 5-7%
// faster on larger jobs).  This layout runs 8-10% faster than one that stored
// 4 code bytes per lane straight from registers (64-byte pieces per store).
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

constexpr int kThreads = 256;        // dequantization and the phi map
// Quantizers: one wave per workgroup (measured on MI355X, 8192 x 4096 bf16:
// 18.3 us against 18.6 us with four waves per workgroup).
constexpr int kQuantThreads = 64;
constexpr int kSpanBlocks = 64;                       // blocks per wave span
constexpr int kSpanCodeBytes = kSpanBlocks * kBlock / 2;
constexpr int64_t kLastLevelCacheBytes = int64_t(256) << 20;
// Workgroups of the kernels that loop over their grid (dequantization and
// the phi map): enough to fill the GPU many times over.
constexpr int64_t kMaxLoopGrid = int64_t(1) << 16;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Maximum over aligned groups of G lanes (G = 4: quad_perm 1,0,3,2 and
// 2,3,0,1; G = 8 adds row_half_mirror, which pairs lane i with 7 - i).
template <int G>
__device__ __forceinline__ float group_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  if constexpr (G == 8) v = fmaxf(v, dpp_f<0x141>(v));
  return v;
}

template <int E>
__device__ __forceinline__ float absmax(const float (&v)[E]) {
  float a = fabsf(v[0]);
#pragma unroll
  for (int i = 1; i < E; ++i) a = fmaxf(a, fabsf(v[i]));
  return a;
}

template <int E>
__device__ __forceinline__ uint32_t encode(const float (&v)[E], float s) {
  if constexpr (E == 8) return encode8(v, s);
  else return encode4(v[0], v[1], v[2], v[3], s);
}

template <int E>
__device__ __forceinline__ void decode(uint32_t c, float s, float (&d)[E]) {
  if constexpr (E == 8) decode8(c, s, d);
  else decode4(c, s, d);
}

template <bool NT>
__device__ __forceinline__ void store16(uint8_t *p, const u32x4 &v) {
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p));
  else *reinterpret_cast<u32x4 *>(p) = v;
}

// Elements of one 16-byte input unit.
template <bool BF16_IN>
__device__ __forceinline__ void unpack(const u32x4 &w, float (&v)[BF16_IN ? 8 : 4]) {
  if constexpr (BF16_IN) {
    v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xFFFF0000u);
    v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xFFFF0000u);
    v[4] = __uint_as_float(w.z << 16); v[5] = __uint_as_float(w.z & 0xFFFF0000u);
    v[6] = __uint_as_float(w.w << 16); v[7] = __uint_as_float(w.w & 0xFFFF0000u);
  } else {
    v[0] = __uint_as_float(w.x); v[1] = __uint_as_float(w.y);
    v[2] = __uint_as_float(w.z); v[3] = __uint_as_float(w.w);
  }
}

// Wave-private staging of one code stream: the span's codes in tensor order,
// then its scale bytes.
struct alignas(16) Stage {
  uint8_t codes[kSpanCodeBytes];
  uint8_t scales[kSpanBlocks];
};

// Quantizer kernel (SWIGLU: the input is h = bf16(silu(g) u) of g = x and
// u = x2, optionally written to h_out).  nblocks = elements / 32.
template <bool BF16_IN, bool RES, bool NT_STORE, bool SWIGLU>
__global__ __launch_bounds__(kQuantThreads) void quantize_kernel(
    const void *__restrict__ x, const void *__restrict__ x2, int64_t nblocks,
    uint8_t *__restrict__ q_codes, uint8_t *__restrict__ q_scales,
    uint8_t *__restrict__ r_codes, uint8_t *__restrict__ r_scales,
    uint16_t *__restrict__ h_out) {
  constexpr int kE = BF16_IN ? 8 : 4;             // elements per lane and step
  constexpr int kLanesPerBlock = kBlock / kE;
  constexpr int kSteps = kSpanBlocks * kLanesPerBlock / 64;
  constexpr int kCodeBytes = kE / 2;              // per lane and step
  __shared__ Stage stage[kQuantThreads / 64][RES ? 2 : 1];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t blk0 = ((int64_t)blockIdx.x * (kQuantThreads / 64) + wave) * kSpanBlocks;
  const int64_t nunits = nblocks * kLanesPerBlock;   // 16-byte input units
  const u32x4 *xin = reinterpret_cast<const u32x4 *>(x);
  const u32x4 *xin2 = reinterpret_cast<const u32x4 *>(x2);

  // Unit of (step u, lane): blk0 * kLanesPerBlock + 64 u + lane.  Lanes past
  // the end load the last unit (never out of bounds); their blocks are not
  // stored, and a block is either wholly inside or wholly past the end.
  u32x4 in[kSteps], in2[SWIGLU ? kSteps : 1];
#pragma unroll
  for (int u = 0; u < kSteps; ++u) {
    int64_t unit = blk0 * kLanesPerBlock + 64 * u + lane;
    unit = unit < nunits ? unit : nunits - 1;
    in[u] = __builtin_nontemporal_load(xin + unit);
    if constexpr (SWIGLU) in2[u] = __builtin_nontemporal_load(xin2 + unit);
  }

  Stage &sq = stage[wave][0];
  Stage &sr = stage[wave][RES ? 1 : 0];
#pragma unroll
  for (int u = 0; u < kSteps; ++u) {
    const int64_t unit = blk0 * kLanesPerBlock + 64 * u + lane;
    float v[kE];
    if constexpr (SWIGLU) {
      float g[kE], w[kE];
      uint32_t hb[kE];
      unpack<BF16_IN>(in[u], g);
      unpack<BF16_IN>(in2[u], w);
#pragma unroll
      for (int j = 0; j < kE; ++j) {
        hb[j] = swiglu_bits(g[j], w[j]);
        v[j] = __uint_as_float(hb[j]);
      }
      if (h_out && unit < nunits) {
        uint32_t p[kE / 2];
#pragma unroll
        for (int j = 0; j < kE / 2; ++j) p[j] = (hb[2 * j] >> 16) | (hb[2 * j + 1] & 0xFFFF0000u);
        if constexpr (BF16_IN)
          *reinterpret_cast<u32x4 *>(h_out + kE * unit) = u32x4{p[0], p[1], p[2], p[3]};
        else
          *reinterpret_cast<uint2 *>(h_out + kE * unit) = make_uint2(p[0], p[1]);
      }
    } else {
      unpack<BF16_IN>(in[u], v);
    }
    const int pos = 64 * u + lane;                 // lane-unit within the span
    const int sblk = pos / kLanesPerBlock;         // block within the span
    const bool leader = (lane & (kLanesPerBlock - 1)) == 0;

    const uint32_t qb = scale_byte(group_max<kLanesPerBlock>(absmax(v)));
    const float qsc = scale_operand(qb);
    const uint32_t qc = encode(v, qsc);
    if constexpr (kCodeBytes == 4) *reinterpret_cast<uint32_t *>(sq.codes + 4 * pos) = qc;
    else *reinterpret_cast<uint16_t *>(sq.codes + 2 * pos) = (uint16_t)qc;
    if (leader) sq.scales[sblk] = (uint8_t)qb;
    if constexpr (RES) {
      float d[kE], r[kE];
      decode(qc, qsc, d);
#pragma unroll
      for (int j = 0; j < kE; ++j) r[j] = v[j] - d[j];
      const uint32_t rb = scale_byte(group_max<kLanesPerBlock>(absmax(r)));
      const uint32_t rc = encode(r, scale_operand(rb));
      if constexpr (kCodeBytes == 4) *reinterpret_cast<uint32_t *>(sr.codes + 4 * pos) = rc;
      else *reinterpret_cast<uint16_t *>(sr.codes + 2 * pos) = (uint16_t)rc;
      if (leader) sr.scales[sblk] = (uint8_t)rb;
    }
  }
  // The staging area is private to the wave and LDS serves a wave's
  // accesses in order, so no workgroup barrier is needed.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();

  const int64_t b = blk0 + lane;                   // block stored by this lane
  const u32x4 cq = *reinterpret_cast<const u32x4 *>(sq.codes + 16 * lane);
  if (b < nblocks) store16<NT_STORE>(q_codes + 16 * b, cq);
  if constexpr (RES) {
    const u32x4 cr = *reinterpret_cast<const u32x4 *>(sr.codes + 16 * lane);
    if (b < nblocks) store16<NT_STORE>(r_codes + 16 * b, cr);
  }
  const bool vec = blk0 + kSpanBlocks <= nblocks &&
                   ((reinterpret_cast<uintptr_t>(q_scales) |
                     reinterpret_cast<uintptr_t>(RES ? r_scales : q_scales)) & 15) == 0;
  if (vec) {
    // Lanes 0-3: primary scale bytes, lanes 4-7: residual, 16 each.
    if (lane < 4)
      store16<NT_STORE>(q_scales + blk0 + 16 * lane,
                        *reinterpret_cast<const u32x4 *>(sq.scales + 16 * lane));
    else if (RES && lane < 8)
      store16<NT_STORE>(r_scales + blk0 + 16 * (lane - 4),
                        *reinterpret_cast<const u32x4 *>(sr.scales + 16 * (lane - 4)));
  } else if (b < nblocks) {
    q_scales[b] = sq.scales[lane];
    if constexpr (RES) r_scales[b] = sr.scales[lane];
  }
}

__global__ __launch_bounds__(kThreads) void dequant_kernel(
    const uint32_t *__restrict__ codes, const uint8_t *__restrict__ scales,
    int64_t nchunks, float4 *__restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t ch = (int64_t)blockIdx.x * kThreads + threadIdx.x; ch < nchunks; ch += stride) {
    float d[8];
    decode8(codes[ch], scale_operand(scales[ch >> 2]), d);
    out[2 * ch] = make_float4(d[0], d[1], d[2], d[3]);
    out[2 * ch + 1] = make_float4(d[4], d[5], d[6], d[7]);
  }
}

// Fallback-indicator map over tiles of 64 rows by 256 reduction columns (a
// workgroup per tile, looping over the grid): rule 0 marks tiles where a
// residual code has a nonzero magnitude, rule 1 tiles holding a primary
// scale byte >= threshold.
__global__ __launch_bounds__(kThreads) void fallback_map_kernel(
    const uint8_t *__restrict__ r_codes, const uint8_t *__restrict__ q_scales, int64_t M,
    int64_t K, int rule, int threshold, int pcols, int64_t tiles, uint8_t *__restrict__ phi) {
  const int tid = threadIdx.x;
  for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
    const int64_t p = t / pcols, c = t % pcols;
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
    if (tid == 0) phi[t] = (uint8_t)(flag != 0);
  }
}

inline unsigned grid_for(int64_t n, int64_t per_block) {
  return (unsigned)((n + per_block - 1) / per_block);
}

// Streaming stores once the job's traffic exceeds the last-level cache.
inline bool nt_stores(int64_t nelem, int64_t in_bytes_per_elem, bool res) {
  const int64_t bytes = nelem * in_bytes_per_elem + (res ? 2 : 1) * (nelem / 2 + nelem / 32);
  return bytes > kLastLevelCacheBytes;
}

template <bool BF16_IN, bool RES, bool SWIGLU>
hipError_t launch_q(const void *x, const void *x2, int64_t nelem, bool nt, uint8_t *qc,
                    uint8_t *qs, uint8_t *rc, uint8_t *rs, uint16_t *h, hipStream_t stream) {
  const int64_t nblocks = nelem / kBlock;
  const dim3 grid(grid_for(nblocks, (kQuantThreads / 64) * kSpanBlocks)), block(kQuantThreads);
  if (nt)
    quantize_kernel<BF16_IN, RES, true, SWIGLU><<<grid, block, 0, stream>>>(x, x2, nblocks, qc, qs,
                                                                           rc, rs, h);
  else
    quantize_kernel<BF16_IN, RES, false, SWIGLU><<<grid, block, 0, stream>>>(x, x2, nblocks, qc, qs,
                                                                            rc, rs, h);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const void *x, bool bf16_in, int64_t nelem,
                           uint8_t *q_codes, uint8_t *q_scales,
                           uint8_t *r_codes, uint8_t *r_scales,
                           hipStream_t stream) {
  const bool res = r_codes != nullptr;
  const bool nt = nt_stores(nelem, bf16_in ? 2 : 4, res);
  if (bf16_in) {
    if (res)
      return launch_q<true, true, false>(x, nullptr, nelem, nt, q_codes, q_scales, r_codes,
                                         r_scales, nullptr, stream);
    return launch_q<true, false, false>(x, nullptr, nelem, nt, q_codes, q_scales, nullptr,
                                        nullptr, nullptr, stream);
  }
  if (res)
    return launch_q<false, true, false>(x, nullptr, nelem, nt, q_codes, q_scales, r_codes,
                                        r_scales, nullptr, stream);
  return launch_q<false, false, false>(x, nullptr, nelem, nt, q_codes, q_scales, nullptr,
                                       nullptr, nullptr, stream);
}

hipError_t launch_swiglu_quantize(const void *g, const void *u, bool bf16_in,
                                  int64_t nelem, uint8_t *q_codes,
                                  uint8_t *q_scales, uint8_t *r_codes,
                                  uint8_t *r_scales, uint16_t *h_out,
                                  hipStream_t stream) {
  const bool res = r_codes != nullptr;
  const bool nt = nt_stores(nelem, bf16_in ? 4 : 8, res);
  if (bf16_in) {
    if (res)
      return launch_q<true, true, true>(g, u, nelem, nt, q_codes, q_scales, r_codes, r_scales,
                                        h_out, stream);
    return launch_q<true, false, true>(g, u, nelem, nt, q_codes, q_scales, nullptr, nullptr,
                                       h_out, stream);
  }
  if (res)
    return launch_q<false, true, true>(g, u, nelem, nt, q_codes, q_scales, r_codes, r_scales,
                                       h_out, stream);
  return launch_q<false, false, true>(g, u, nelem, nt, q_codes, q_scales, nullptr, nullptr,
                                      h_out, stream);
}

hipError_t launch_dequant(const uint8_t *codes, const uint8_t *scales,
                          int64_t nelem, float *out, hipStream_t stream) {
  const int64_t nchunks = nelem / kChunk;
  const int64_t wgs = (nchunks + kThreads - 1) / kThreads;
  dequant_kernel<<<(unsigned)(wgs < kMaxLoopGrid ? wgs : kMaxLoopGrid), kThreads, 0, stream>>>(
      reinterpret_cast<const uint32_t *>(codes), scales, nchunks,
      reinterpret_cast<float4 *>(out));
  return hipGetLastError();
}

hipError_t launch_fallback_map(const uint8_t *r_codes, const uint8_t *q_scales, int64_t M,
                               int64_t K, int rule, int threshold, uint8_t *phi,
                               hipStream_t stream) {
  const int pcols = (int)((K + 255) / 256);
  const int64_t tiles = ((M + 63) / 64) * pcols;
  fallback_map_kernel<<<(unsigned)(tiles < kMaxLoopGrid ? tiles : kMaxLoopGrid), kThreads, 0,
                        stream>>>(r_codes, q_scales, M, K, rule, threshold, pcols, tiles, phi);
  return hipGetLastError();
}

}  // namespace rfq
