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
// chip idle.  Here a workgroup owns 32 rows of W (two fragments; one where
// that gives too few workgroups or for up to 4 activation rows, four where
// 64 rows still give about one workgroup per CU, and one in the streaming
// form) and up to four 16-row activation slices, and its four waves split K
// into four contiguous ranges; the partial 16 x 16 results of the waves are
// summed in a fixed order through LDS.  W is read once per 64 activation
// rows.
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
// codes in, the same for q and r of each slice, one slice ahead.  W rows past
// N are clamped to the last row for loading, activation rows past M to the
// last row or to zeros: an activation row only reaches its own output column
// of the MFMA result, and those columns are not stored.
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

// Store of one 16 x 16 result: Z rows m0 + l mod 16, columns n0 + 4 (l/16) .. +3.
template <bool ZBF16>
__device__ __forceinline__ void store_tile(const v4f &s, int lane, int64_t m0, int64_t n0,
                                           int64_t M, int64_t N, void *z) {
  const int64_t m = m0 + (lane & 15);
  const int64_t n = n0 + 4 * (lane >> 4);
  if (m >= M) return;
  if constexpr (ZBF16) {
    uint16_t *zp = reinterpret_cast<uint16_t *>(z) + m * N + n;
    if (n + 4 <= N && (N % 4) == 0) {
      uint2 v;
      v.x = bf16x2_rne(s[0], s[1]);
      v.y = bf16x2_rne(s[2], s[3]);
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

// Fixed-order sum of the four waves' partial 16 x 16 results and its store.
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
  store_tile<ZBF16>(s, lane, m0, n0, M, N, z);
}

// Codes in: a workgroup owns F fragments of W (16 F rows) and up to S
// activation slices of 16 rows.  Each wave holds a group of W in registers
// while it multiplies every slice against it, so W is read once per launch
// (for M <= 16 S) and the activation codes once per 16 F W rows.  The next
// slice's codes (or the next group's first slice) are loaded while the
// current one is multiplied.  Per output the accumulation order is that of
// a single slice: groups, k-steps, primary then residual, then the
// fixed-order sum over the four waves.
//
// Split K (gridDim.z = parts > 1, fp32 output only): workgroup z covers the
// groups [ngroups z / parts, ngroups (z + 1) / parts) of K / 512, which its
// waves divide as they would the whole K, and writes its partial products to
// the z-th M x N fp32 slab of the output; a second kernel adds the slabs in
// the order z = 0, 1, ...  With one part the ranges and the output are those
// of the unsplit product.
template <int F>
struct WPair { WGroup f[F]; };

template <bool RES, bool ZBF16, int S, int F>
__global__ __launch_bounds__(kSkThreads, F == 1 ? 3 : (F == 2 ? 2 : 1)) void rfq_gemm_skinny_kernel(
    const uint8_t *__restrict__ qc, const uint8_t *__restrict__ qs,
    const uint8_t *__restrict__ rc, const uint8_t *__restrict__ rs,
    const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws, int64_t M, int64_t N,
    int64_t K, void *__restrict__ z) {
  __shared__ v4f partial[kSkThreads / 64][F * S][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int row = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * (F * kSkRows);
  const int64_t m0 = (int64_t)blockIdx.y * (S * kSkRows);
  const int slices = (int)min<int64_t>(S, (M - m0 + kSkRows - 1) / kSkRows);
  const int64_t kbytes = K / 2, kblocks = K / 32;

  // This wave's groups of 4 k-steps: [gb, ge) of K / 512, within this
  // workgroup's part [pb, pe).
  const int ngroups = (int)(K / kSkGroupK);
  const int part = (int)blockIdx.z, parts = (int)gridDim.z;
  const int pb = (ngroups * part) / parts, pe = (ngroups * (part + 1)) / parts;
  const int gb = pb + ((pe - pb) * wave) / 4, ge = pb + ((pe - pb) * (wave + 1)) / 4;

  const __amdgpu_buffer_rsrc_t rwc = rsrc(wc, N * kbytes), rws = rsrc(ws, N * kblocks);
  uint32_t w_off[F], ws_off[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int64_t wn = min(n0 + kSkRows * f + row, N - 1);
    w_off[f] = (uint32_t)wn * (uint32_t)kbytes + 16 * g;
    ws_off[f] = (uint32_t)wn * (uint32_t)kblocks;
  }
  auto load_w = [&](WPair<F> &w, int gi) {
#pragma unroll
    for (int f = 0; f < F; ++f) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w.f[f].c[j] = __builtin_amdgcn_raw_buffer_load_b128(rwc, w_off[f],
                                                            gi * (kSkGroupK / 2) + 64 * j, 0);
      w.f[f].s = __builtin_amdgcn_raw_buffer_load_b128(rws, ws_off[f], gi * (kSkGroupK / 32), 0);
    }
  };

  const __amdgpu_buffer_rsrc_t rxa = rsrc(qc, M * kbytes), rxb = rsrc(RES ? rc : qc, M * kbytes);
  const __amdgpu_buffer_rsrc_t rxs = rsrc(qs, M * kblocks), rxt = rsrc(RES ? rs : qs, M * kblocks);
  // Activation codes of slice sl of group gi (rows past M clamped to the last).
  auto load_x = [&](XGroup &xg, int gi, int sl) {
    const uint32_t xm = (uint32_t)min(m0 + kSkRows * sl + row, M - 1);
    const bool live = sl < slices;
    const uint32_t xc_off = live ? xm * (uint32_t)kbytes + 16 * g : 0x80000000u;
    const uint32_t xs_off = live ? xm * (uint32_t)kblocks : 0x80000000u;
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

  v4f acc[S][F];
#pragma unroll
  for (int sl = 0; sl < S; ++sl)
#pragma unroll
    for (int f = 0; f < F; ++f) acc[sl][f] = v4f{0.0f, 0.0f, 0.0f, 0.0f};

  auto compute = [&](const WPair<F> &w, const XGroup &xg, v4f (&a)[F]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const uint32_t wsc = scale_of(w.f[f].s, j, g);
        a[f] = mma16(w.f[f].c[j], wsc, xg.q[j], scale_of(xg.qs, j, g), a[f]);
        if constexpr (RES) a[f] = mma16(w.f[f].c[j], wsc, xg.r[j], scale_of(xg.rs, j, g), a[f]);
      }
    }
  };
  // One group: every slice against the group's W.  Slice sl of the group is
  // in buffer xa for even sl and xb for odd sl; at each slice the following
  // unit (the next slice, or the next group's first slice) is requested into
  // the other buffer before the current one is waited for.  Slices past M
  // load zeros without touching memory and skip their MFMAs.  With S even
  // the next group again starts in xa; with S = 1 the buffers swap roles.
  auto group = [&](const WPair<F> &w, int gi, XGroup &xa, XGroup &xb) {
#pragma unroll
    for (int sl = 0; sl < S; ++sl) {
      XGroup &cur = (sl & 1) ? xb : xa;
      XGroup &nxt = (sl & 1) ? xa : xb;
      if (sl + 1 < S) load_x(nxt, gi, sl + 1);
      else if (gi + 1 < ge) load_x(nxt, gi + 1, 0);
      if (sl < slices) compute(w, cur, acc[sl]);
    }
  };
  if (gb < ge) {
    WPair<F> w0, w1;
    XGroup xa, xb;
    load_w(w0, gb);
    load_x(xa, gb, 0);
    int gi = gb;
    for (; gi + 1 < ge; gi += 2) {
      load_w(w1, gi + 1);
      group(w0, gi, xa, xb);
      if (gi + 2 < ge) load_w(w0, gi + 2);
      if constexpr (S % 2 == 0) group(w1, gi + 1, xa, xb);
      else group(w1, gi + 1, xb, xa);
    }
    if (gi < ge) group(w0, gi, xa, xb);
  }

  // Fixed-order sum over the four waves; output (fragment f, slice sl) is
  // summed and stored by wave (f S + sl) mod 4.
  void *const zpart = ZBF16 ? z : static_cast<void *>(static_cast<float *>(z) + part * M * N);
#pragma unroll
  for (int f = 0; f < F; ++f)
#pragma unroll
    for (int sl = 0; sl < S; ++sl) partial[wave][f * S + sl][lane] = acc[sl][f];
  __syncthreads();
  for (int p = wave; p < F * S; p += kSkThreads / 64) {
    const int f = p / S, sl = p % S;
    if (sl >= slices) continue;
    v4f s = partial[0][p][lane];
#pragma unroll
    for (int w = 1; w < kSkThreads / 64; ++w) {
      const v4f q = partial[w][p][lane];
      s = v4f{s[0] + q[0], s[1] + q[1], s[2] + q[2], s[3] + q[3]};
    }
    store_tile<ZBF16>(s, lane, m0 + kSkRows * sl, n0 + kSkRows * f, M, N, zpart);
  }
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

// The streaming form holds one W fragment per workgroup (16 rows), or four
// (64 rows) where that still gives about one workgroup per CU: the
// quantization of the activation slice, which every workgroup repeats, is
// then shared by four times the weight rows.  With the quantizer's registers
// a second fragment no longer fits two waves per SIMD, so four take one
// (406-480 registers).
template <int F>
struct StW { WGroup f[F]; };

// (fp32 input: one wave per SIMD; its registers do not fit two without spilling.)
template <bool RES, bool ZBF16, bool XF32, int S, int kStFrags>
__global__ __launch_bounds__(kSkThreads, (XF32 || kStFrags > 1) ? 1 : 2) void rfq_gemm_stream_kernel(
    const void *__restrict__ x, const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws,
    int64_t M, int64_t N, int64_t K, void *__restrict__ z) {
  __shared__ v4f partial[kSkThreads / 64][kStFrags * S][64];
  __shared__ StreamArea area[kSkThreads / 64];
  constexpr int kElem = XF32 ? 4 : 2;
  constexpr int kPieces = 32 * kElem / 16;        // 16-byte loads per block

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int row = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * (kStFrags * kSkRows);
  const int64_t m0 = (int64_t)blockIdx.y * (S * kSkRows);
  const int slices = (int)min<int64_t>(S, (M - m0 + kSkRows - 1) / kSkRows);
  const int64_t kbytes = K / 2, kblocks = K / 32;
  const int ngroups = (int)(K / kSkGroupK);
  const int gb = (ngroups * wave) / 4, ge = (ngroups * (wave + 1)) / 4;

  const __amdgpu_buffer_rsrc_t rwc = rsrc(wc, N * kbytes), rws = rsrc(ws, N * kblocks);
  uint32_t w_off[kStFrags], ws_off[kStFrags];
#pragma unroll
  for (int f = 0; f < kStFrags; ++f) {
    const int64_t wn = min(n0 + kSkRows * f + row, N - 1);
    w_off[f] = (uint32_t)wn * (uint32_t)kbytes + 16 * g;
    ws_off[f] = (uint32_t)wn * (uint32_t)kblocks;
  }
  auto load_w = [&](StW<kStFrags> &w, int gi) {
#pragma unroll
    for (int f = 0; f < kStFrags; ++f) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w.f[f].c[j] = __builtin_amdgcn_raw_buffer_load_b128(rwc, w_off[f],
                                                            gi * (kSkGroupK / 2) + 64 * j, 0);
      w.f[f].s = __builtin_amdgcn_raw_buffer_load_b128(rws, ws_off[f], gi * (kSkGroupK / 32), 0);
    }
  };

  // Quantization rounds of slice sl: in round rd lane l takes block
  // t = 64 rd + l of the group, row t / 16 and block t mod 16 of the slice;
  // the slice's rows that exist are [0, live(sl)).  Lanes past them load
  // nothing (offsets beyond the buffer return zeros without touching
  // memory) and write nothing.
  auto live_rows = [&](int sl) {
    return (int)max<int64_t>(0, min<int64_t>(kSkRows, M - m0 - kSkRows * sl));
  };
  const __amdgpu_buffer_rsrc_t rx = rsrc(x, M * K * kElem);
  struct XRound { u32x4 v[kPieces]; };
  auto load_round = [&](XRound &xr, int gi, int sl, int rd) {
    const int t = 64 * rd + lane;
    const uint32_t off =
        (t >> 4) < live_rows(sl)
            ? (uint32_t)(((m0 + kSkRows * sl + (t >> 4)) * K + 32 * (t & 15)) * kElem)
            : 0x80000000u;
#pragma unroll
    for (int p = 0; p < kPieces; ++p)
      xr.v[p] = __builtin_amdgcn_raw_buffer_load_b128(rx, off, gi * kSkGroupK * kElem + 16 * p, 0);
  };
  StreamArea &A = area[wave];
  auto quantize_round = [&](const XRound &xr, int live, int rd) {
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

  // One unit (group gi, slice sl): quantize the slice's blocks of the group
  // into the LDS area (xn holds the unit's round 0 on entry and the next
  // unit's round 0 on exit), then multiply them with both W fragments.
  // Units run slice by slice, so only one slice's accumulators are live (the
  // slices' passes over the wave's W range re-read it from L2).
  XRound xn, xa, xb;
  auto unit = [&](const StW<kStFrags> &w, int gi, int sl, v4f (&a)[kStFrags]) {
    const int live = live_rows(sl);
    const int rounds = (live * kGroupBlocks + 63) / 64;
    xa = xn;
    if (rounds > 1) load_round(xb, gi, sl, 1);
    if (gi + 1 < ge) load_round(xn, gi + 1, sl, 0);
    else if (sl + 1 < slices) load_round(xn, gb, sl + 1, 0);
    quantize_round(xa, live, 0);
    if (rounds > 1) {
      if (rounds > 2) load_round(xa, gi, sl, 2);
      quantize_round(xb, live, 1);
      if (rounds > 2) {
        if (rounds > 3) load_round(xb, gi, sl, 3);
        quantize_round(xa, live, 2);
        if (rounds > 3) quantize_round(xb, live, 3);
      }
    }
    // The area is private to the wave and LDS serves a wave's accesses in
    // order: the writes above are seen by the reads below, and the reads
    // below precede the next unit's writes.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const u32x4 sq = *reinterpret_cast<const u32x4 *>(A.qs + row * kGroupBlocks);
    const u32x4 sr = RES ? *reinterpret_cast<const u32x4 *>(A.rs + row * kGroupBlocks) : sq;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int chunk = 16 * (row * kGroupBlocks + ((4 * j + g) ^ row));
      const u32x4 cq = *reinterpret_cast<const u32x4 *>(A.q + chunk);
      const u32x4 cr = RES ? *reinterpret_cast<const u32x4 *>(A.r + chunk) : cq;
#pragma unroll
      for (int f = 0; f < kStFrags; ++f) {
        const uint32_t wsc = scale_of(w.f[f].s, j, g);
        a[f] = mma16(w.f[f].c[j], wsc, cq, scale_of(sq, j, g), a[f]);
        if constexpr (RES) a[f] = mma16(w.f[f].c[j], wsc, cr, scale_of(sr, j, g), a[f]);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  if (gb < ge) load_round(xn, gb, 0, 0);
  for (int sl = 0; sl < slices; ++sl) {
    v4f a[kStFrags];
#pragma unroll
    for (int f = 0; f < kStFrags; ++f) a[f] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    if (gb < ge) {
      StW<kStFrags> w0, w1;
      load_w(w0, gb);
      int gi = gb;
      for (; gi + 1 < ge; gi += 2) {
        load_w(w1, gi + 1);
        unit(w0, gi, sl, a);
        if (gi + 2 < ge) load_w(w0, gi + 2);
        unit(w1, gi + 1, sl, a);
      }
      if (gi < ge) unit(w0, gi, sl, a);
    }
#pragma unroll
    for (int f = 0; f < kStFrags; ++f) partial[wave][f * S + sl][lane] = a[f];
  }

  // Fixed-order sum over the four waves, as in the codes-in form.
  __syncthreads();
  for (int p = wave; p < kStFrags * S; p += kSkThreads / 64) {
    const int f = p / S, sl = p % S;
    if (sl >= slices) continue;
    v4f s = partial[0][p][lane];
#pragma unroll
    for (int w = 1; w < kSkThreads / 64; ++w) {
      const v4f q = partial[w][p][lane];
      s = v4f{s[0] + q[0], s[1] + q[1], s[2] + q[2], s[3] + q[3]};
    }
    store_tile<ZBF16>(s, lane, m0 + kSkRows * sl, n0 + kSkRows * f, M, N, z);
  }
}

template <bool RES, bool ZBF16, int S, int F = 2>
hipError_t launch_sk_s(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc, const uint8_t *rs,
                       const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N, int64_t K,
                       void *z, int parts, hipStream_t stream) {
  const dim3 grid((unsigned)((N + F * kSkRows - 1) / (F * kSkRows)),
                  (unsigned)((M + S * kSkRows - 1) / (S * kSkRows)), (unsigned)parts);
  rfq_gemm_skinny_kernel<RES, ZBF16, S, F><<<grid, dim3(kSkThreads), 0, stream>>>(
      qc, qs, rc, rs, wc, ws, M, N, K, z);
  return hipGetLastError();
}

// Slices per workgroup: the fewest of 1, 2 or 4 that cover M's rows, at most
// 4 (more slices per workgroup make the kernel spill, measured slower).
// Weight fragments per workgroup: one (16 rows, twice the workgroups) for up
// to 4 activation rows (whose loads are then negligible) and where two would
// leave CUs without a workgroup; else two (the activation codes are then
// loaded once per 32 weight rows).  Measured on MI355X at 12288 x 4096 and
// 4096 x 12288 weights: 8 - 26% faster where chosen, slower elsewhere.
// Four fragments (64 weight rows, one workgroup per CU at 274-392
// registers) serve 5-64 rows where that gives 176-256 workgroups per row of
// workgroups (11264 <= N < 16384; at 12288 x 4096 weights 16 rows 11.8 ->
// 9.7 us, 32 rows 16.6 -> 12.1, 64 rows 25.4 -> 17.0) and 33-64 rows from
// N = 16384 (64 rows x 24576 x 4096: 37.2 -> 32.8 us); single slices take
// two from N = 16384 at any row count (1 row x 24576 x 4096: 14.5 -> 12.9 us).
constexpr int64_t kFillWorkgroups = 256;    // one per CU on MI355X
int sk_slices(int64_t M) { return M <= kSkRows ? 1 : (M <= 2 * kSkRows ? 2 : 4); }
int sk_fragments(int64_t M, int64_t N) {
  if (skinny_four_fragments(M, N)) return 4;
  const int S = sk_slices(M);
  if (S == 1 && N >= 16384) return 2;
  const int64_t wgs = ((N + 2 * kSkRows - 1) / (2 * kSkRows)) * ((M + S * kSkRows - 1) / (S * kSkRows));
  return (M <= 4 || wgs < kFillWorkgroups) ? 1 : 2;
}
int64_t sk_workgroups(int64_t M, int64_t N) {
  const int64_t S = sk_slices(M), F = sk_fragments(M, N);
  return ((N + F * kSkRows - 1) / (F * kSkRows)) * ((M + S * kSkRows - 1) / (S * kSkRows));
}

template <bool RES, bool ZBF16>
hipError_t launch_sk(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc, const uint8_t *rs,
                     const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N, int64_t K,
                     void *z, hipStream_t stream, int parts = 1) {
#define RFQ_SK(S, F) launch_sk_s<RES, ZBF16, S, F>(qc, qs, rc, rs, wc, ws, M, N, K, z, parts, stream)
  const int S = sk_slices(M), F = sk_fragments(M, N);
  if (S == 1) return F == 4 ? RFQ_SK(1, 4) : (F == 2 ? RFQ_SK(1, 2) : RFQ_SK(1, 1));
  if (S == 2) return F == 4 ? RFQ_SK(2, 4) : (F == 2 ? RFQ_SK(2, 2) : RFQ_SK(2, 1));
  return F == 4 ? RFQ_SK(4, 4) : (F == 2 ? RFQ_SK(4, 2) : RFQ_SK(4, 1));
#undef RFQ_SK
}

template <bool RES, bool ZBF16, bool XF32, int S, int F>
hipError_t launch_st_s(const void *x, const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N,
                       int64_t K, void *z, hipStream_t stream) {
  const dim3 grid((unsigned)((N + F * kSkRows - 1) / (F * kSkRows)),
                  (unsigned)((M + S * kSkRows - 1) / (S * kSkRows)));
  rfq_gemm_stream_kernel<RES, ZBF16, XF32, S, F><<<grid, dim3(kSkThreads), 0, stream>>>(
      x, wc, ws, M, N, K, z);
  return hipGetLastError();
}

// Four fragments from N = 11264 for 5 or more rows (bf16 activations:
// 16 rows x 12288 x 4096 16.6 -> 12.1 us, 64 rows 51.7 -> 41.0 us; 16 rows
// x 24576 x 4096 30.9 -> 23.9 us); one elsewhere (4096 x 12288 weights: 19.1
// against 30.6 us at 16 rows).
template <bool RES, bool ZBF16, bool XF32, int S>
hipError_t launch_st_f(const void *x, const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N,
                       int64_t K, void *z, hipStream_t stream) {
  if (M > 4 && N >= 11264)
    return launch_st_s<RES, ZBF16, XF32, S, 4>(x, wc, ws, M, N, K, z, stream);
  return launch_st_s<RES, ZBF16, XF32, S, 1>(x, wc, ws, M, N, K, z, stream);
}

template <bool RES, bool ZBF16, bool XF32>
hipError_t launch_st(const void *x, const uint8_t *wc, const uint8_t *ws, int64_t M, int64_t N,
                     int64_t K, void *z, hipStream_t stream) {
  if (M <= kSkRows) return launch_st_f<RES, ZBF16, XF32, 1>(x, wc, ws, M, N, K, z, stream);
  if (M <= 2 * kSkRows) return launch_st_f<RES, ZBF16, XF32, 2>(x, wc, ws, M, N, K, z, stream);
  return launch_st_f<RES, ZBF16, XF32, 4>(x, wc, ws, M, N, K, z, stream);
}

}  // namespace

bool skinny_grid_uneven(int64_t M, int64_t N) {
  const int64_t wgs = sk_workgroups(M, N);
  return wgs > kFillWorkgroups && wgs < 2 * kFillWorkgroups;
}

// Where the grid's last round of workgroups is at most a quarter full (257
// to 320 workgroups: one weight fragment per workgroup at 4096 < N <= 5120),
// the CUs that run two finish last; three parts of K even that out, at the
// cost of the sum.  Each part keeps at least 8 groups of 512 (two per wave).
// Measured at 5120 x 13824 weights, bf16 Z, sum included: 1 row 15.0 -> 12.8
// us, 8 rows 17.9 -> 15.2, 16 rows 23.7 -> 19.3; at 6144 x 12288 (384
// workgroups) 1 row 13.1 -> 14.6 and 8 rows 17.7 -> 17.5; at 4096 x 12288
// (256 workgroups) and N >= 12288 every split was slower (1 row x 4096 x
// 12288: 8.2 -> 9.5 us).
int skinny_split_parts(int64_t M, int64_t N, int64_t K) {
  constexpr int kParts = 3;
  if (M > kSkRows || K / kSkGroupK < 8 * kParts) return 1;
  const int64_t wgs = sk_workgroups(M, N);
  return (wgs > kFillWorkgroups && 4 * wgs <= 5 * kFillWorkgroups) ? kParts : 1;
}

bool skinny_four_fragments(int64_t M, int64_t N) {
  if (M <= 4 || M > 4 * kSkRows) return false;
  if (N >= 11264 && N < 16384) return true;
  return N >= 16384 && M > 2 * kSkRows;
}

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

hipError_t launch_gemm_skinny_split(const uint8_t *q_codes, const uint8_t *q_scales,
                                    const uint8_t *r_codes, const uint8_t *r_scales,
                                    const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                                    int64_t N, int64_t K, void *z, bool z_bf16, int parts,
                                    float *work, hipStream_t stream) {
  const hipError_t e =
      r_codes ? launch_sk<true, false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M,
                                       N, K, work, stream, parts)
              : launch_sk<false, false>(q_codes, q_scales, nullptr, nullptr, w_codes, w_scales, M,
                                        N, K, work, stream, parts);
  if (e != hipSuccess) return e;
  return launch_splitk_sum(work, parts, M * N, z, z_bf16, stream);
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
