// RFQ product for few activation rows (decode-sized M), in two forms:
//
//   codes in:  Z = (deq q + deq r) deq(w)^T from the quantizer's codes
//              (Eq. 11 with phi = 1; phi = 0 without the residual);
//   streaming: Z from the activations X themselves, each MX block quantized
//              (primary code, Eq. 8; residual of what it lost, quantized
//              again, Eq. 9-10) inside the product's K loop right before the
//              MFMAs that use it - the streaming form of Algorithm 1, in which
//              neither the residual nor any activation code reaches memory.
//
// With few rows the product is bound by streaming W's codes from memory, and
// the large-tile kernels (256 activation rows per tile) would leave most of the
// chip idle.  Here a workgroup owns 16 rows of W (one fragment) and 16
// activation rows, and its four waves split K into four contiguous ranges;
// the four partial 16 x 16 results are summed in a fixed order through LDS.
// The grid is (N/16) x (M/16) workgroups, so W is read once per 16
// activation rows.
//
// Instruction: v_mfma_scale_f32_16x16x128_f8f6f4 with E2M1 operands (format
// 4).  In k-step ks (128 K values, 4 MX blocks) lane l holds row l mod 16 and
// block 4 ks + l/16 (16 code bytes) of its operand and supplies that block's
// scale byte; the weight fragment is the A operand, so the 16 x 16 fp32
// result in lane l holds Z[m = l mod 16][n = 4 (l/16) .. +3].
//
// Loads: a wave walks its K range in groups of 4 k-steps (512 K values) and
// issues the next group's loads before multiplying the current one.  Per
// group a lane loads 4 x 16 code bytes of its W row and the 16 scale bytes of
// the row's group (scale byte of k-step j, lane group g: byte g of word j);
// codes in, the same for q and r.  Rows past M or N are clamped to the last
// row for loading: an activation row only reaches its own output column of
// the MFMA result, and those columns are not stored.
//
// Streaming form: per group, the wave first quantizes the activation blocks
// of its 16-row slice that exist (rows < M), one block per lane and 64 blocks
// per round, with the arithmetic of the standalone quantizer (mx_device.h),
// so the codes are those rfq_quantize_act writes.  The codes and scale bytes
// go to a wave-private LDS area in the operand layout of the codes-in form
// (16-byte chunks XOR-swizzled by row), from which the MFMAs of the group
// read them; the products are therefore bit-identical to the codes-in form.
// Quantizing only existing rows keeps the vector work proportional to M (in
// the MFMA layout every lane would quantize a block, also of rows past M).
// A round's activation loads are issued one round ahead, and the first
// round of the next group before the current group is quantized.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm_common.h"
#include "mx_device.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

constexpr int kSkThreads = 256;     // 4 waves, one K range each
constexpr int kSkRows = 16;         // W rows and activation rows per workgroup
constexpr int kSkGroupK = 512;      // K values per load group (4 k-steps)

struct XGroup { u32x4 q[4], r[4], qs, rs; };
struct WGroup { u32x4 c[4], s; };

// 16 code bytes as the MFMA's 8-register FP4 operand (upper half unused).
__device__ __forceinline__ v8i frag(const u32x4 &d) {
  return v8i{(int)d.x, (int)d.y, (int)d.z, (int)d.w, 0, 0, 0, 0};
}

__device__ __forceinline__ uint32_t scale_of(const u32x4 &s, int j, int g) {
  return (s[j] >> (8 * g)) & 0xFFu;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *p, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ v4f mma16(const u32x4 &wcode, uint32_t wsc, const u32x4 &xcode,
                                     uint32_t xsc, const v4f &acc) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(frag(wcode), frag(xcode), acc, kFmtFp4,
                                                          kFmtFp4, 0, (int)wsc, 0, (int)xsc);
}

// Primary and residual codes and scale bytes of one 32-element block.
template <int E>
__device__ __forceinline__ void quantize_block(const float (&v)[E], u32x4 &qc, uint32_t &qb,
                                               u32x4 &rc, uint32_t &rb, bool res) {
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < E; ++i) amax = fmaxf(amax, fabsf(v[i]));
  qb = scale_byte(amax);
  const float qsc = scale_operand(qb);
  uint32_t c[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float(&p)[8] = *reinterpret_cast<const float(*)[8]>(&v[8 * w]);
    c[w] = encode8(p, qsc);
  }
  qc = u32x4{c[0], c[1], c[2], c[3]};
  if (!res) return;
  float r[E];
  float ramax = 0.0f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float d[8];
    decode8(c[w], qsc, d);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      r[8 * w + i] = v[8 * w + i] - d[i];
      ramax = fmaxf(ramax, fabsf(r[8 * w + i]));
    }
  }
  rb = scale_byte(ramax);
  const float rsc = scale_operand(rb);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float(&p)[8] = *reinterpret_cast<const float(*)[8]>(&r[8 * w]);
    c[w] = encode8(p, rsc);
  }
  rc = u32x4{c[0], c[1], c[2], c[3]};
}

// Fixed-order sum of the four waves' partial 16 x 16 results and the store
// of Z (rows m0 + l mod 16, columns n0 + 4 (l/16) .. +3).
template <bool ZBF16>
__device__ __forceinline__ void reduce_store(v4f (&partial)[kSkThreads / 64][64], const v4f &acc,
                                             int wave, int lane, int64_t m0, int64_t n0,
                                             int64_t M, int64_t N, void *z) {
  partial[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  v4f s = partial[0][lane];
#pragma unroll
  for (int w = 1; w < kSkThreads / 64; ++w) {
    const v4f p = partial[w][lane];
    s = v4f{s[0] + p[0], s[1] + p[1], s[2] + p[2], s[3] + p[3]};
  }
  const int64_t m = m0 + (lane & 15);
  const int64_t n = n0 + 4 * (lane >> 4);
  if (m >= M) return;
  if constexpr (ZBF16) {
    uint16_t *zp = reinterpret_cast<uint16_t *>(z) + m * N + n;
    if (n + 4 <= N && (N % 4) == 0) {
      uint2 v;
      v.x = bf16_rne(s[0]) | (bf16_rne(s[1]) << 16);
      v.y = bf16_rne(s[2]) | (bf16_rne(s[3]) << 16);
      *reinterpret_cast<uint2 *>(zp) = v;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N) zp[e] = (uint16_t)bf16_rne(s[e]);
    }
  } else {
    float *zp = reinterpret_cast<float *>(z) + m * N + n;
    if (n + 4 <= N && (N % 4) == 0) {
      *reinterpret_cast<v4f *>(zp) = s;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N) zp[e] = s[e];
    }
  }
}

template <bool RES, bool ZBF16>
__global__ __launch_bounds__(kSkThreads) void rfq_gemm_skinny_kernel(
    const uint8_t *__restrict__ qc, const uint8_t *__restrict__ qs,
    const uint8_t *__restrict__ rc, const uint8_t *__restrict__ rs,
    const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws, int64_t M, int64_t N,
    int64_t K, void *__restrict__ z) {
  __shared__ v4f partial[kSkThreads / 64][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int row = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * kSkRows, m0 = (int64_t)blockIdx.y * kSkRows;
  const int64_t wn = min(n0 + row, N - 1);
  const int64_t xm = min(m0 + row, M - 1);
  const int64_t kbytes = K / 2, kblocks = K / 32;

  // This wave's groups of 4 k-steps: [gb, ge) of K / 512.
  const int ngroups = (int)(K / kSkGroupK);
  const int gb = (ngroups * wave) / 4, ge = (ngroups * (wave + 1)) / 4;

  const __amdgpu_buffer_rsrc_t rwc = rsrc(wc, N * kbytes), rws = rsrc(ws, N * kblocks);
  const uint32_t w_off = (uint32_t)wn * (uint32_t)kbytes + 16 * g;
  const uint32_t ws_off = (uint32_t)wn * (uint32_t)kblocks;
  auto load_w = [&](WGroup &w, int gi) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w.c[j] = __builtin_amdgcn_raw_buffer_load_b128(rwc, w_off, gi * (kSkGroupK / 2) + 64 * j, 0);
    w.s = __builtin_amdgcn_raw_buffer_load_b128(rws, ws_off, gi * (kSkGroupK / 32), 0);
  };

  const __amdgpu_buffer_rsrc_t rxa = rsrc(qc, M * kbytes), rxb = rsrc(RES ? rc : qc, M * kbytes);
  const __amdgpu_buffer_rsrc_t rxs = rsrc(qs, M * kblocks), rxt = rsrc(RES ? rs : qs, M * kblocks);
  const uint32_t xc_off = (uint32_t)xm * (uint32_t)kbytes + 16 * g;
  const uint32_t xs_off = (uint32_t)xm * (uint32_t)kblocks;
  v4f acc = v4f{0.0f, 0.0f, 0.0f, 0.0f};

  // W and activation codes of a whole group in flight.
  auto load_x = [&](XGroup &xg, int gi) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      xg.q[j] = __builtin_amdgcn_raw_buffer_load_b128(rxa, xc_off, gi * (kSkGroupK / 2) + 64 * j, 0);
      if constexpr (RES)
        xg.r[j] = __builtin_amdgcn_raw_buffer_load_b128(rxb, xc_off, gi * (kSkGroupK / 2) + 64 * j, 0);
    }
    xg.qs = __builtin_amdgcn_raw_buffer_load_b128(rxs, xs_off, gi * (kSkGroupK / 32), 0);
    if constexpr (RES)
      xg.rs = __builtin_amdgcn_raw_buffer_load_b128(rxt, xs_off, gi * (kSkGroupK / 32), 0);
  };
  auto compute = [&](const WGroup &w, const XGroup &xg) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t wsc = scale_of(w.s, j, g);
      acc = mma16(w.c[j], wsc, xg.q[j], scale_of(xg.qs, j, g), acc);
      if constexpr (RES) acc = mma16(w.c[j], wsc, xg.r[j], scale_of(xg.rs, j, g), acc);
    }
  };
  if (gb < ge) {
    WGroup w0, w1;
    XGroup x0, x1;
    load_w(w0, gb);
    load_x(x0, gb);
    int gi = gb;
    for (; gi + 1 < ge; gi += 2) {
      load_w(w1, gi + 1);
      load_x(x1, gi + 1);
      compute(w0, x0);
      if (gi + 2 < ge) {
        load_w(w0, gi + 2);
        load_x(x0, gi + 2);
      }
      compute(w1, x1);
    }
    if (gi < ge) compute(w0, x0);
  }
  reduce_store<ZBF16>(partial, acc, wave, lane, m0, n0, M, N, z);
}

// Wave-private LDS area of the streaming form: the codes of one group (16
// blocks per row) of the slice's 16 rows, in 16-byte chunks (chunk of block b
// of row r at slot b ^ r, so the 16 rows read together by one k-step spread
// over the banks), then the scale bytes [row][block].
constexpr int kGroupBlocks = kSkGroupK / kBlock;
struct alignas(16) StreamArea {
  uint8_t q[kSkRows * kGroupBlocks * 16];
  uint8_t r[kSkRows * kGroupBlocks * 16];
  uint8_t qs[kSkRows * kGroupBlocks];
  uint8_t rs[kSkRows * kGroupBlocks];
};

template <bool RES, bool ZBF16, bool XF32>
__global__ __launch_bounds__(kSkThreads) void rfq_gemm_stream_kernel(
    const void *__restrict__ x, const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws,
    int64_t M, int64_t N, int64_t K, void *__restrict__ z) {
  __shared__ v4f partial[kSkThreads / 64][64];
  __shared__ StreamArea area[kSkThreads / 64];
  constexpr int kElem = XF32 ? 4 : 2;
  constexpr int kPieces = 32 * kElem / 16;        // 16-byte loads per block

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int row = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * kSkRows, m0 = (int64_t)blockIdx.y * kSkRows;
  const int64_t wn = min(n0 + row, N - 1);
  const int64_t kbytes = K / 2, kblocks = K / 32;
  const int ngroups = (int)(K / kSkGroupK);
  const int gb = (ngroups * wave) / 4, ge = (ngroups * (wave + 1)) / 4;

  const __amdgpu_buffer_rsrc_t rwc = rsrc(wc, N * kbytes), rws = rsrc(ws, N * kblocks);
  const uint32_t w_off = (uint32_t)wn * (uint32_t)kbytes + 16 * g;
  const uint32_t ws_off = (uint32_t)wn * (uint32_t)kblocks;
  auto load_w = [&](WGroup &w, int gi) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w.c[j] = __builtin_amdgcn_raw_buffer_load_b128(rwc, w_off, gi * (kSkGroupK / 2) + 64 * j, 0);
    w.s = __builtin_amdgcn_raw_buffer_load_b128(rws, ws_off, gi * (kSkGroupK / 32), 0);
  };

  // Quantization rounds: in round rd lane l takes block t = 64 rd + l of the
  // group, row t / 16 and block t mod 16 of the slice; rows that exist are
  // [0, live).  Lanes past them load nothing (offsets beyond the buffer
  // return zeros without touching memory) and write nothing.
  const int live = (int)min<int64_t>(kSkRows, M - m0);
  const int rounds = (live * kGroupBlocks + 63) / 64;
  const __amdgpu_buffer_rsrc_t rx = rsrc(x, M * K * kElem);
  auto x_off = [&](int rd) {
    const int t = 64 * rd + lane;
    return (t >> 4) < live ? (uint32_t)(((m0 + (t >> 4)) * K + 32 * (t & 15)) * kElem)
                           : 0x80000000u;
  };
  struct XRound { u32x4 v[kPieces]; };
  auto load_round = [&](XRound &xr, int gi, int rd) {
    const uint32_t off = x_off(rd);
#pragma unroll
    for (int p = 0; p < kPieces; ++p)
      xr.v[p] = __builtin_amdgcn_raw_buffer_load_b128(rx, off, gi * kSkGroupK * kElem + 16 * p, 0);
  };
  StreamArea &A = area[wave];
  auto quantize_round = [&](const XRound &xr, int rd) {
    const int t = 64 * rd + lane;
    const int xr_row = t >> 4, xb = t & 15;
    if (xr_row >= live) return;
    float v[32];
    if constexpr (XF32) {
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const u32x4 &u = xr.v[p];
        v[4 * p + 0] = __uint_as_float(u.x); v[4 * p + 1] = __uint_as_float(u.y);
        v[4 * p + 2] = __uint_as_float(u.z); v[4 * p + 3] = __uint_as_float(u.w);
      }
    } else {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const u32x4 &u = xr.v[p];
        v[8 * p + 0] = __uint_as_float(u.x << 16); v[8 * p + 1] = __uint_as_float(u.x & 0xFFFF0000u);
        v[8 * p + 2] = __uint_as_float(u.y << 16); v[8 * p + 3] = __uint_as_float(u.y & 0xFFFF0000u);
        v[8 * p + 4] = __uint_as_float(u.z << 16); v[8 * p + 5] = __uint_as_float(u.z & 0xFFFF0000u);
        v[8 * p + 6] = __uint_as_float(u.w << 16); v[8 * p + 7] = __uint_as_float(u.w & 0xFFFF0000u);
      }
    }
    u32x4 cq, cr;
    uint32_t bq, br = 0;
    quantize_block(v, cq, bq, cr, br, RES);
    const int chunk = 16 * (xr_row * kGroupBlocks + (xb ^ xr_row));
    *reinterpret_cast<u32x4 *>(A.q + chunk) = cq;
    A.qs[xr_row * kGroupBlocks + xb] = (uint8_t)bq;
    if constexpr (RES) {
      *reinterpret_cast<u32x4 *>(A.r + chunk) = cr;
      A.rs[xr_row * kGroupBlocks + xb] = (uint8_t)br;
    }
  };

  v4f acc = v4f{0.0f, 0.0f, 0.0f, 0.0f};
  // One group: quantize its rounds into the LDS area (xn holds round 0 on
  // entry and round 0 of the next group on exit), then multiply it.
  XRound xn, xa, xb;
  auto group = [&](const WGroup &w, int gi) {
    xa = xn;
    if (rounds > 1) load_round(xb, gi, 1);
    if (gi + 1 < ge) load_round(xn, gi + 1, 0);
    quantize_round(xa, 0);
    if (rounds > 1) {
      if (rounds > 2) load_round(xa, gi, 2);
      quantize_round(xb, 1);
      if (rounds > 2) {
        if (rounds > 3) load_round(xb, gi, 3);
        quantize_round(xa, 2);
        if (rounds > 3) quantize_round(xb, 3);
      }
    }
    // The area is private to the wave and LDS serves a wave's accesses in
    // order: the writes above are seen by the reads below, and the reads
    // below precede the next group's writes.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const u32x4 sq = *reinterpret_cast<const u32x4 *>(A.qs + row * kGroupBlocks);
    const u32x4 sr = RES ? *reinterpret_cast<const u32x4 *>(A.rs + row * kGroupBlocks) : sq;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int chunk = 16 * (row * kGroupBlocks + ((4 * j + g) ^ row));
      const uint32_t wsc = scale_of(w.s, j, g);
      acc = mma16(w.c[j], wsc, *reinterpret_cast<const u32x4 *>(A.q + chunk), scale_of(sq, j, g),
                  acc);
      if constexpr (RES)
        acc = mma16(w.c[j], wsc, *reinterpret_cast<const u32x4 *>(A.r + chunk),
                    scale_of(sr, j, g), acc);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  if (gb < ge) {
    WGroup w0, w1;
    load_w(w0, gb);
    load_round(xn, gb, 0);
    int gi = gb;
    for (; gi + 1 < ge; gi += 2) {
      load_w(w1, gi + 1);
      group(w0, gi);
      if (gi + 2 < ge) load_w(w0, gi + 2);
      group(w1, gi + 1);
    }
    if (gi < ge) group(w0, gi);
  }
  reduce_store<ZBF16>(partial, acc, wave, lane, m0, n0, M, N, z);
}

inline dim3 skinny_grid(int64_t M, int64_t N) {
  return dim3((unsigned)((N + kSkRows - 1) / kSkRows), (unsigned)((M + kSkRows - 1) / kSkRows));
}

template <bool RES, bool ZBF16>
hipError_t launch_sk(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc, const uint8_t *rs,
                     const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N, int64_t K,
                     void *z, hipStream_t stream) {
  rfq_gemm_skinny_kernel<RES, ZBF16><<<skinny_grid(M, N), dim3(kSkThreads), 0, stream>>>(
      qc, qs, rc, rs, wc, ws, M, N, K, z);
  return hipGetLastError();
}

template <bool RES, bool ZBF16, bool XF32>
hipError_t launch_st(const void *x, const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N,
                     int64_t K, void *z, hipStream_t stream) {
  rfq_gemm_stream_kernel<RES, ZBF16, XF32><<<skinny_grid(M, N), dim3(kSkThreads), 0, stream>>>(
      x, wc, ws, M, N, K, z);
  return hipGetLastError();
}

}  // namespace

bool gemm_skinny_applies(const uint8_t *q_scales, const uint8_t *r_scales,
                         const uint8_t *w_scales, int64_t M, int64_t N, int64_t K) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(q_scales) |
                      reinterpret_cast<uintptr_t>(r_scales) |
                      reinterpret_cast<uintptr_t>(w_scales);
  const int64_t limit = int64_t(1) << 31;
  return M <= kSkinnyMaxRows && (K % kSkGroupK) == 0 && (a & 15) == 0 &&
         M * (K / 2) < limit && N * (K / 2) < limit;
}

hipError_t launch_gemm_skinny(const uint8_t *q_codes, const uint8_t *q_scales,
                              const uint8_t *r_codes, const uint8_t *r_scales,
                              const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                              int64_t N, int64_t K, void *z, bool z_bf16, hipStream_t stream) {
  if (r_codes) {
    if (z_bf16)
      return launch_sk<true, true>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
    return launch_sk<true, false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
  }
  if (z_bf16)
    return launch_sk<false, true>(q_codes, q_scales, nullptr, nullptr, w_codes, w_scales, M, N, K, z, stream);
  return launch_sk<false, false>(q_codes, q_scales, nullptr, nullptr, w_codes, w_scales, M, N, K, z, stream);
}

hipError_t launch_gemm_stream(const void *x, bool x_bf16, bool residual, const uint8_t *w_codes,
                              const uint8_t *w_scales, int64_t M, int64_t N, int64_t K, void *z,
                              bool z_bf16, hipStream_t stream) {
#define RFQ_ST(R, Z, F) launch_st<R, Z, F>(x, w_codes, w_scales, M, N, K, z, stream)
  if (x_bf16) {
    if (residual) return z_bf16 ? RFQ_ST(true, true, false) : RFQ_ST(true, false, false);
    return z_bf16 ? RFQ_ST(false, true, false) : RFQ_ST(false, false, false);
  }
  if (residual) return z_bf16 ? RFQ_ST(true, true, true) : RFQ_ST(true, false, true);
  return z_bf16 ? RFQ_ST(false, true, true) : RFQ_ST(false, false, true);
#undef RFQ_ST
}

}  // namespace rfq
