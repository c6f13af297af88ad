// HiF4 form of the RFQ path on gfx950 (Sec. 3.3, Eq. 5-6, with the RFQ
// steps of Sec. 4.3, Eq. 8-11): the quantizer (primary HiF4 code and, for
// activations, the HiF4 code of the residual it leaves), dequantization and
// the RFQ product.
//
// Format.  A block is 64 consecutive elements of a row along K.  Per block
// one 32-bit metadata word: bits 0-7 the E6M2 macro scale byte (E << 2 | M,
// S = 2^(E-48) (1 + M/4), Eq. 5), bits 8-15 the 1-bit micro-exponents of the
// eight 8-element groups (E1_8, bit g for elements 8g..8g+7), bits 16-31
// those of the sixteen 4-element groups (E1_16, bit j for elements 4j..4j+3).
// Per element a 4-bit S1P2 code, sign << 3 | k with magnitude k/4, two per
// byte, element 2j in the low nibble of byte j.  Value (Eq. 6):
//     V_i = S 2^(E1_8[i/8] + E1_16[i/4]) (-1)^sign k/4.
// With c = 4 + M this is V_i = +-k c 2^(E - 52 + e_i): at most 6 significant
// bits with exponents in [-52, 19], so every value is exact in bf16 and every
// product of two values is exact in fp32.
//
// Encoder.  The paper fixes the decode but not the encoder; this library
// takes these choices (dequantization and the product are exact for any
// metadata and codes):
//   - S is the smallest E6M2 value with 7 S >= amax (7 = 1.75 * 2^2, the
//     largest factor an element can carry), so no element saturates unless
//     amax exceeds 7 times the largest E6M2 value (then byte 255);
//   - the 4-element group j needs the smallest e_j in {0, 1, 2} with
//     1.75 * 2^e_j * S >= its largest magnitude; the 8-element group g takes
//     E1_8[g] = 1 when one of its two 4-element groups needs 2, and then
//     E1_16[j] = max(e_j - E1_8[g], 0);
//   - k is |x| / (S 2^e / 4) rounded to nearest, ties to even, at most 7; the
//     sign is kept, also for a zero.
// The rounding is k = rne(|x| / u) with the grid unit u = c 2^(E - 52 + e),
// c = 4 + M.  A quotient from the reciprocal of u, refined once with the
// exact remainder fma(-y, u, |x|), is the correctly rounded |x|/u wherever
// the integer rounding depends on it: an exact tie j + 1/2 is representable
// and comes out exactly, and any other |x|/u lies at least ulp(|x|)/(c 2^p)
// > ulp(y)/2 away from j + 1/2 (2^p the power of two in u), more than the
// refined quotient's error.  Where k could be nonzero, |x| >= u/2 >= 2^-51,
// so the remainder stays far above the fp32 subnormal range.  The residual
// x - V is exact in fp32 (V is the grid value nearest x, so the difference is
// a multiple of the finer of ulp(x) and the grid's last bit and smaller than
// a grid unit); it is formed as fma(-k, +-u, x), whose exact result rounds to
// itself, with +0 for x = V, so the second encode sees exactly the residual.
//
// Quantizer work decomposition: a lane owns 8 consecutive elements (one
// 8-element group, 16 bytes of bf16 or 32 of fp32 input); the 8 lanes of a
// block combine their maxima and metadata bits with DPP; a wave covers 32
// blocks in 4 steps, each load instruction reading 1 KB (bf16) of contiguous
// input and each code store writing 256 contiguous bytes.
//
// Product.  gfx950 has no matrix-core format for HiF4, so the product
// decodes codes to bf16 and runs v_mfma_f32_32x32x16_bf16, whose products are
// exact; accumulation is fp32.  A workgroup computes a 128 x 256 tile of Z
// with waves in two roles: producer waves load the codes and metadata of one
// K block (64 values) of the tile's 128 activation rows (and 128 residual
// rows) and 256 weight rows, decode them and write bf16 rows into one of two
// LDS buffers, while four consumer waves (2 x 2, each a 64 x 128 sub-tile)
// multiply the other buffer; one workgroup barrier per K block hands the
// buffers over.  Every SIMD runs one consumer and (with the residual) two
// producers, so decoding (VALU) and multiplication (matrix core) overlap and
// the decode has two instruction streams to issue from.  16-byte chunks of
// an LDS row are XOR-swizzled by row so that fragment reads and row writes
// are free of bank conflicts.  Rows past M or N are clamped to the last row
// for loading; their results are not stored.
#include <hip/hip_runtime.h>
#include <algorithm>
#include <stdint.h>

#include <atomic>

#include "gemm_common.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kH = 64;                 // elements per HiF4 block
constexpr int kQThreads = 256;
constexpr int kQSteps = 4;             // 8-element units per lane (large tensors)
// Below this many 8-element units a lane takes one unit, so that small
// (decode-sized) tensors spread over four times as many waves.
constexpr int64_t kQSmallUnits = int64_t(1) << 18;
constexpr int kLoopGrid = 1 << 16;     // dequantization grid cap (loops over the rest)

// Every lane of these permutations has a source, so the old value never
// shows; passing v as it lets the compiler fold the move into the operation.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xF, 0xF, true);
}

// Maximum and bitwise OR over aligned groups of 8 lanes (quad_perm 1,0,3,2,
// quad_perm 2,3,0,1, then row_half_mirror, which pairs lane i with 7 - i).
__device__ __forceinline__ float max8(float v) {
  v = fmaxf(v, __uint_as_float(dpp_u<0xB1>(__float_as_uint(v))));
  v = fmaxf(v, __uint_as_float(dpp_u<0x4E>(__float_as_uint(v))));
  return fmaxf(v, __uint_as_float(dpp_u<0x141>(__float_as_uint(v))));
}
__device__ __forceinline__ uint32_t or8(uint32_t v) {
  v |= dpp_u<0xB1>(v);
  v |= dpp_u<0x4E>(v);
  return v | dpp_u<0x141>(v);
}

// E6M2 value of byte b: (4 + (b & 3)) 2^((b >> 2) - 50), whose fp32 pattern
// is (b + 316) << 21.
__device__ __forceinline__ float macro_value(uint32_t b) {
  return __uint_as_float((b + 316u) << 21);
}

// Smallest byte with 7 S >= amax.  The candidate rounds amax / 7 up to two
// mantissa bits; it is off by at most one step, which the exact tests (7 S
// has at most 6 significant bits) correct.
__device__ __forceinline__ uint32_t macro_byte(float amax) {
  const uint32_t u = __float_as_uint(amax * (1.0f / 7.0f));
  int b = (int)(u >> 21) - 316 + ((u & 0x1FFFFFu) != 0 ? 1 : 0);
  b = min(max(b, 0), 255);
  if (b < 255 && 7.0f * macro_value((uint32_t)b) < amax) ++b;
  if (b > 0 && 7.0f * macro_value((uint32_t)b - 1u) >= amax) --b;
  return (uint32_t)b;
}

// 2^p for p in the normal range.
__device__ __forceinline__ float pow2(int p) { return __uint_as_float((uint32_t)(p + 127) << 23); }

// Encodes the 8 elements of this lane (8-element group g of its block): the
// lane's 32 code bits, the block's metadata word (same in all 8 lanes) and,
// with WANT_R, the residuals x - V (exact: x - V is representable and the
// fma rounds it once).
template <bool WANT_R>
__device__ __forceinline__ uint32_t encode8(const float (&x)[8], int g, uint32_t &meta,
                                            float (&res)[8]) {
  float ga = fabsf(x[0]), gb = fabsf(x[4]);
#pragma unroll
  for (int i = 1; i < 4; ++i) {
    ga = fmaxf(ga, fabsf(x[i]));
    gb = fmaxf(gb, fabsf(x[4 + i]));
  }
  const uint32_t byte = macro_byte(max8(fmaxf(ga, gb)));
  const float t0 = 1.75f * macro_value(byte);                // exact
  const int na = (ga > t0) + (ga > 2.0f * t0), nb = (gb > t0) + (gb > 2.0f * t0);
  const int e8 = (na == 2) | (nb == 2);
  const int ea = max(na - e8, 0), eb = max(nb - e8, 0);
  meta = byte | or8(((uint32_t)e8 << (8 + g)) | ((uint32_t)ea << (16 + 2 * g)) |
                    ((uint32_t)eb << (17 + 2 * g)));
  const int E = (int)(byte >> 2);
  const float c = (float)(4 + (byte & 3));
  const float rc = __builtin_amdgcn_rcpf(c);
  // Per 4-element group: the grid unit c 2^(E-52+e) and its reciprocal
  // (2^(52-E-e) / c, both powers of two exact scalings).
  const float unit_a = c * pow2(E - 52 + e8 + ea), unit_b = c * pow2(E - 52 + e8 + eb);
  const float ru_a = rc * pow2(52 - E - e8 - ea), ru_b = rc * pow2(52 - E - e8 - eb);
  uint32_t code = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float unit = i < 4 ? unit_a : unit_b, ru = i < 4 ? ru_a : ru_b;
    const float a = fabsf(x[i]);
    const float y = a * ru;
    const float yq = fmaf(fmaf(-y, unit, a), ru, y);
    const float kf = fminf(__builtin_rintf(yq), 7.0f);
    code |= (((__float_as_uint(x[i]) >> 28) & 8u) | (uint32_t)kf) << (4 * i);
    if constexpr (WANT_R) res[i] = fmaf(-kf, copysignf(unit, x[i]), x[i]);
  }
  return code;
}

template <bool BF16_IN>
__device__ __forceinline__ void unpack8(const u32x4 (&w)[BF16_IN ? 1 : 2], float (&v)[8]) {
  if constexpr (BF16_IN) {
    const u32x4 a = w[0];
    v[0] = __uint_as_float(a.x << 16); v[1] = __uint_as_float(a.x & 0xFFFF0000u);
    v[2] = __uint_as_float(a.y << 16); v[3] = __uint_as_float(a.y & 0xFFFF0000u);
    v[4] = __uint_as_float(a.z << 16); v[5] = __uint_as_float(a.z & 0xFFFF0000u);
    v[6] = __uint_as_float(a.w << 16); v[7] = __uint_as_float(a.w & 0xFFFF0000u);
  } else {
    v[0] = __uint_as_float(w[0].x); v[1] = __uint_as_float(w[0].y);
    v[2] = __uint_as_float(w[0].z); v[3] = __uint_as_float(w[0].w);
    v[4] = __uint_as_float(w[1].x); v[5] = __uint_as_float(w[1].y);
    v[6] = __uint_as_float(w[1].z); v[7] = __uint_as_float(w[1].w);
  }
}

// nunits = elements / 8.  Lanes past the end load the last unit (never out
// of bounds) and store nothing; a block is wholly inside or past the end.
template <bool BF16_IN, bool RES, int STEPS>
__global__ __launch_bounds__(kQThreads) void hif4_quantize_kernel(
    const void *__restrict__ x, int64_t nunits, uint8_t *__restrict__ qc,
    uint32_t *__restrict__ qm, uint8_t *__restrict__ rc, uint32_t *__restrict__ rm) {
  constexpr int kLoads = BF16_IN ? 1 : 2;
  const int lane = threadIdx.x & 63, g = lane & 7;
  const int64_t u0 =
      ((int64_t)blockIdx.x * (kQThreads / 64) + (threadIdx.x >> 6)) * (64 * STEPS);
  const u32x4 *xin = reinterpret_cast<const u32x4 *>(x);
  u32x4 in[STEPS][kLoads];
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    int64_t u = u0 + 64 * s + lane;
    u = u < nunits ? u : nunits - 1;
#pragma unroll
    for (int l = 0; l < kLoads; ++l) in[s][l] = __builtin_nontemporal_load(xin + kLoads * u + l);
  }
#pragma unroll
  for (int s = 0; s < STEPS; ++s) {
    const int64_t u = u0 + 64 * s + lane;
    float v[8], r[8];
    unpack8<BF16_IN>(in[s], v);
    uint32_t meta;
    const uint32_t code = encode8<RES>(v, g, meta, r);
    if (u < nunits) {
      reinterpret_cast<uint32_t *>(qc)[u] = code;
      if (g == 0) qm[u >> 3] = meta;
    }
    if constexpr (RES) {
      float unused[8];
      uint32_t rmeta;
      const uint32_t rcode = encode8<false>(r, g, rmeta, unused);
      if (u < nunits) {
        reinterpret_cast<uint32_t *>(rc)[u] = rcode;
        if (g == 0) rm[u >> 3] = rmeta;
      }
    }
  }
}

// Unit (value of k = 1) of the two 4-element groups of 8-element group g:
// c 2^(E - 52 + e).
__device__ __forceinline__ void group_units(uint32_t meta, int g, float &ua, float &ub) {
  const float base = (float)(4 + (meta & 3)) * pow2((int)((meta >> 2) & 63) - 52);
  const uint32_t e8 = (meta >> (8 + g)) & 1u;
  const uint32_t ea = e8 + ((meta >> (16 + 2 * g)) & 1u);
  const uint32_t eb = e8 + ((meta >> (17 + 2 * g)) & 1u);
  ua = __uint_as_float(__float_as_uint(base) + (ea << 23));
  ub = __uint_as_float(__float_as_uint(base) + (eb << 23));
}

// One dequantization thread: 8 elements (one code word) to fp32 or to bf16
// (exact either way).
template <bool BF16_OUT>
__global__ __launch_bounds__(256) void hif4_dequant_kernel(
    const uint32_t *__restrict__ codes, const uint32_t *__restrict__ meta, int64_t nunits,
    void *__restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x; u < nunits; u += stride) {
    const uint32_t w = codes[u];
    float ua, ub;
    group_units(meta[u >> 3], (int)(u & 7), ua, ub);
    float d[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t nib = (w >> (4 * i)) & 15u;
      const float mag = (float)(nib & 7u) * (i < 4 ? ua : ub);
      d[i] = (nib & 8u) ? -mag : mag;
    }
    if constexpr (BF16_OUT) {
      reinterpret_cast<u32x4 *>(out)[u] =
          u32x4{(__float_as_uint(d[0]) >> 16) | (__float_as_uint(d[1]) & 0xFFFF0000u),
                (__float_as_uint(d[2]) >> 16) | (__float_as_uint(d[3]) & 0xFFFF0000u),
                (__float_as_uint(d[4]) >> 16) | (__float_as_uint(d[5]) & 0xFFFF0000u),
                (__float_as_uint(d[6]) >> 16) | (__float_as_uint(d[7]) & 0xFFFF0000u)};
    } else {
      float4 *o = reinterpret_cast<float4 *>(out);
      o[2 * u] = make_float4(d[0], d[1], d[2], d[3]);
      o[2 * u + 1] = make_float4(d[4], d[5], d[6], d[7]);
    }
  }
}

// ---------------------------------------------------------------- product

constexpr int kBM = 128;                       // tile: activation rows x BN weight rows
constexpr int kRowBytes = kH * 2;              // one decoded bf16 row of a K block
constexpr int kTM = 64;                        // consumer sub-tile: 64 x BN/2
constexpr int kFM = kTM / 32;

// BN = 256 weight rows per tile, or 128 where 256-row tiles would leave CUs
// idle (fewer activation rows).
template <bool RES, int BN>
struct HSmem {
  static constexpr int kWRow0 = (RES ? 2 : 1) * kBM;    // q rows, r rows, then w rows
  static constexpr int kRows = kWRow0 + BN;
  static constexpr int kBufBytes = kRows * kRowBytes;
  static constexpr int kBytes = 2 * kBufBytes;
  // Producer waves: each lane decodes two half-block rows per step (8 waves,
  // two per SIMD, with the residual and BN = 256).
  static constexpr int kProducers = kRows / 64;
  static constexpr int kThreads = (kProducers + 4) * 64;
  static constexpr int kTN = BN / 2, kFN = kTN / 32;
};

// LDS serves a 16-byte access of 16 lanes at a time across 256 bytes of
// banks (two 128-byte rows): with the XOR by (row >> 1) & 7 the 16
// consecutive rows of a fragment read, and the producers' stores (8 rows x
// two chunk halves per 16 lanes), land in 16 distinct slots (row & 7 let
// rows r and r + 8 collide).
__device__ __forceinline__ int hswz(int row, int chunk) {
  return row * kRowBytes + 16 * (chunk ^ ((row >> 1) & 7));
}

// a & m, opaque to the optimizer, so that the byte conversions below stay
// single v_cvt_f32_ubyte{0..3} instructions instead of a bit-field extract
// per element followed by a conversion.
__device__ __forceinline__ uint32_t and_opaque(uint32_t a, uint32_t m) {
  uint32_t r;
  asm("v_and_b32 %0, %1, %2" : "=v"(r) : "s"(m), "v"(a));
  return r;
}

// bf16 pairs of the 8 elements of code word w (8-element group g of a block
// with metadata meta): element 2p in the low half of pair p.
__device__ __forceinline__ u32x4 decode8_bf16(uint32_t w, uint32_t meta, int g) {
  float ua, ub;
  group_units(meta, g, ua, ub);
  const uint32_t lo = and_opaque(w, 0x07070707u), hi = and_opaque(w >> 4, 0x07070707u);
  const uint32_t w4 = w << 4;
  uint32_t p[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float u = q < 2 ? ua : ub;
    const float f0 = (float)((lo >> (8 * q)) & 0xFFu) * u;   // element 2q (exact)
    const float f1 = (float)((hi >> (8 * q)) & 0xFFu) * u;   // element 2q + 1
    const uint32_t pair = __builtin_amdgcn_perm(__float_as_uint(f1), __float_as_uint(f0),
                                                0x07060302u);
    // Sign bits: bit 7 of byte q of w4 (element 2q) to bit 15, bit 7 of
    // byte q of w (element 2q + 1) to bit 31.
    const uint32_t sgn = __builtin_amdgcn_perm(w, w4, 0x000C000Cu | (q << 8) | ((4 + q) << 24));
    p[q] = pair | (sgn & 0x80008000u);
  }
  return u32x4{p[0], p[1], p[2], p[3]};
}

// WBF16: the weights come as bf16 values wv[N][K] (for example HiF4 weights
// decoded once) and are copied into LDS as they are; only the activation
// codes are decoded.
// SPLIT: the grid holds ceil(K / ksplit) copies of the tile grid, copy s
// multiplying K columns [s ksplit, (s + 1) ksplit) (ksplit a multiple of 64)
// and writing its fp32 partial product to z + s M N.
template <bool RES, bool ZBF16, bool WBF16, int BN, bool SPLIT = false>
__global__ __launch_bounds__((HSmem<RES, BN>::kThreads)) void hif4_gemm_kernel(
    const uint8_t *__restrict__ qc, const uint32_t *__restrict__ qm,
    const uint8_t *__restrict__ rc, const uint32_t *__restrict__ rm,
    const uint8_t *__restrict__ wc, const uint32_t *__restrict__ wm,
    const uint16_t *__restrict__ wv, int64_t M, int64_t N, int64_t K, void *__restrict__ z,
    int64_t ksplit) {
  static_assert(!SPLIT || !ZBF16, "split partials are fp32");
  using S = HSmem<RES, BN>;
  constexpr int kTN = S::kTN, kFN = S::kFN;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  const int ntm = (int)((M + kBM - 1) / kBM), ntn = (int)((N + BN - 1) / BN);
  int bid = blockIdx.x, split = 0;
  if constexpr (SPLIT) {
    split = bid / (ntm * ntn);
    bid -= split * ntm * ntn;
    z = reinterpret_cast<float *>(z) + (int64_t)split * M * N;
  }
  int tm, tn;
  tile_coords<8>(bid, ntm, ntn, tm, tn);
  const int64_t m0 = (int64_t)tm * kBM, n0 = (int64_t)tn * BN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // This workgroup's K blocks: [kb0, kb0 + nsteps).
  const int64_t kb0 = SPLIT ? (int64_t)split * (ksplit / kH) : 0;
  const int nsteps = (int)((SPLIT ? min(ksplit, K - kb0 * kH) : K) / kH);
  const int64_t kbytes = K / 2, kblocks = K / kH;

  if (wave < S::kProducers) {
    // ---- producer: (row, half) items; a half is 32 elements, 16 code bytes.
    constexpr int kPT = S::kProducers * 64;
    constexpr int kItems = S::kRows * 2 / kPT;
    static_assert(kItems * kPT == S::kRows * 2, "item split");
    const int pt = tid;
    const uint8_t *src[kItems];
    const uint32_t *msrc[kItems];
    const u32x4 *vsrc[kItems];
    int lrow[kItems];
    bool is_w[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int r = pt / 2 + (kPT / 2) * i;
      lrow[i] = r;
      is_w[i] = r >= S::kWRow0;
      vsrc[i] = nullptr;
      int64_t grow;
      if (r >= S::kWRow0) {
        grow = min(n0 + (r - S::kWRow0), N - 1);
        if constexpr (WBF16) {
          vsrc[i] = reinterpret_cast<const u32x4 *>(wv + grow * K + kb0 * kH + 32 * (pt & 1));
          src[i] = nullptr;
          msrc[i] = nullptr;
        } else {
          src[i] = wc + grow * kbytes + kb0 * (kH / 2) + 16 * (pt & 1);
          msrc[i] = wm + grow * kblocks + kb0;
        }
      } else {
        const bool is_r = RES && r >= kBM;
        grow = min(m0 + (is_r ? r - kBM : r), M - 1);
        src[i] = (is_r ? rc : qc) + grow * kbytes + kb0 * (kH / 2) + 16 * (pt & 1);
        msrc[i] = (is_r ? rm : qm) + grow * kblocks + kb0;
      }
    }
    const int h = pt & 1;
    // Codes (or bf16 weight values: four 16-byte pieces per item) of step
    // s + 1 are loaded while step s is decoded.  Whether an item is a weight
    // row is uniform over a wave.
    constexpr int kV = WBF16 ? 4 : 1;
    u32x4 cw[kItems][kV], nw[kItems][kV];
    uint32_t mw[kItems], nm[kItems];
    auto load = [&](int s, u32x4 (&c)[kItems][kV], uint32_t (&m)[kItems]) {
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
        if (WBF16 && is_w[i]) {
#pragma unroll
          for (int v = 0; v < kV; ++v) c[i][v] = vsrc[i][(int64_t)s * 8 + v];
        } else {
          c[i][0] = *reinterpret_cast<const u32x4 *>(src[i] + (int64_t)s * 32);
          m[i] = msrc[i][s];
        }
      }
    };
    load(0, cw, mw);
    for (int s = 0; s < nsteps; ++s) {
      if (s + 1 < nsteps) load(s + 1, nw, nm);
      uint8_t *buf = smem + (s & 1) * S::kBufBytes;
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
        if (WBF16 && is_w[i]) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<u32x4 *>(buf + hswz(lrow[i], 4 * h + q)) = cw[i][q % kV];
        } else {
          const uint32_t d[4] = {cw[i][0].x, cw[i][0].y, cw[i][0].z, cw[i][0].w};
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<u32x4 *>(buf + hswz(lrow[i], 4 * h + q)) =
                decode8_bf16(d[q], mw[i], 4 * h + q);
        }
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
#pragma unroll
        for (int v = 0; v < kV; ++v) cw[i][v] = nw[i][v];
        mw[i] = nm[i];
      }
    }
    return;
  }

  // ---- consumer: 2 x 2 waves, each 64 activation rows x 128 weight rows.
  const int cw_ = wave - S::kProducers, wmi = cw_ >> 1, wni = cw_ & 1;
  const int frow = lane & 31, half = lane >> 5;
  v16f acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j) acc[i][j] = v16f{};

  auto frag = [&](const uint8_t *buf, int row, int kk) {
    return *reinterpret_cast<const v8bf *>(buf + hswz(row, 2 * kk + half));
  };
  for (int s = 0; s < nsteps; ++s) {
    __syncthreads();
    const uint8_t *buf = smem + (s & 1) * S::kBufBytes;
#pragma unroll
    for (int kk = 0; kk < kH / 16; ++kk) {
      v8bf wf[kFN], xf[kFM], rf[RES ? kFM : 1];
#pragma unroll
      for (int j = 0; j < kFN; ++j) wf[j] = frag(buf, S::kWRow0 + wni * kTN + 32 * j + frow, kk);
#pragma unroll
      for (int i = 0; i < kFM; ++i) {
        xf[i] = frag(buf, wmi * kTM + 32 * i + frow, kk);
        if constexpr (RES) rf[i] = frag(buf, kBM + wmi * kTM + 32 * i + frow, kk);
      }
#pragma unroll
      for (int i = 0; i < kFM; ++i)
#pragma unroll
        for (int j = 0; j < kFN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[j], xf[i], acc[i][j], 0, 0, 0);
      if constexpr (RES) {
#pragma unroll
        for (int i = 0; i < kFM; ++i)
#pragma unroll
          for (int j = 0; j < kFN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[j], rf[i], acc[i][j], 0, 0, 0);
      }
    }
  }

  // ---- epilogue: lane holds Z[m][n .. n+3] for n = 8a + 4 half (a = 0..3)
  // of each fragment (weights are the first MFMA operand).  The lane's row
  // and column origins are formed here from the thread index rather than
  // kept from before the loop (that value is otherwise held across the
  // loop at the register limit).
  const bool vec_ok = (N & 3) == 0;
  const int elane = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int64_t erow0 = m0 + wmi * kTM + (elane & 31);
  const int64_t ecol0 = n0 + wni * kTN + 4 * (elane >> 5);
#pragma unroll
  for (int i = 0; i < kFM; ++i) {
    const int64_t m = erow0 + 32 * i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int64_t n = ecol0 + 32 * j + 8 * a;
        const v16f &c = acc[i][j];
        if constexpr (ZBF16) {
          uint16_t *zp = reinterpret_cast<uint16_t *>(z) + m * N + n;
          if (vec_ok && n + 3 < N) {
            uint2 w;
            w.x = bf16x2_rne(c[4 * a], c[4 * a + 1]);
            w.y = bf16x2_rne(c[4 * a + 2], c[4 * a + 3]);
            *reinterpret_cast<uint2 *>(zp) = w;
          } else {
#pragma unroll
            for (int b = 0; b < 4; ++b)
              if (n + b < N) zp[b] = (uint16_t)bf16_rne(c[4 * a + b]);
          }
        } else {
          float *zp = reinterpret_cast<float *>(z) + m * N + n;
          if (vec_ok && n + 3 < N) {
            *reinterpret_cast<float4 *>(zp) =
                make_float4(c[4 * a], c[4 * a + 1], c[4 * a + 2], c[4 * a + 3]);
          } else {
#pragma unroll
            for (int b = 0; b < 4; ++b)
              if (n + b < N) zp[b] = c[4 * a + b];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------- few rows
//
// Product for at most 64 activation rows (decode, short prefill): one
// workgroup per 16, 32 or 64 weight rows (F = 1, 2 or 4 fragments of 16) and
// up to MAXM activation rows, or S slices of 16; its WAVES waves take
// interleaved chunks of 128 K values (wave w:
// chunks w, w + WAVES, ...) and run v_mfma_f32_16x16x32_bf16 with the
// weights as the first operand; the partial sums are added in wave order at
// the end.
//
// Weights go straight from memory into operand registers: lane l (row
// l mod 16 of a fragment, quarter g = l / 16) loads the 16 code bytes of
// elements 32 g .. 32 g + 31 of its row's chunk (half g mod 2 of block
// 2 c + g / 2, one metadata word) and decodes them into four 8-element
// operand pieces; MFMA jj of the chunk takes piece jj from every lane, so
// it contracts elements 32 g + 8 jj + (0..7) over the four quarters - a
// fixed permutation of the chunk's K values inside the instruction, which
// the activation operand follows.  The activation rows below M (primary and
// residual) are decoded, one code word per work item, into a wave-private
// LDS area in the same order (16-byte pieces XOR-swizzled by row), from
// which lane l reads row l mod 16; rows at or above M are never written and
// only feed result columns m >= M, which are not stored.  Loads use buffer
// descriptors based at the workgroup's first weight row (32-bit offsets);
// K values past K (a final half chunk) load as zeros, without memory access.
constexpr int kFewRows = 16;
constexpr int kFewMaxRows = 64;             // four slices of 16 activation rows
constexpr int kFewChunk = 128;              // K values per chunk
constexpr uint32_t kFewSkip = 0x80000000u;  // load offset past every buffer: zeros
// Per wave: 16 primary and 16 residual activation rows of one chunk, bf16.
constexpr int kFewXRow = kFewChunk * 2;     // bytes of one decoded row chunk

__device__ __forceinline__ int few_xoff(int row, int piece) {
  return row * kFewXRow + 16 * (piece ^ (row & 15));
}

// The largest K the few-row kernel takes: its buffer ranges and offsets,
// for 32 weight rows of bf16 values (2^30 bytes) or 64 of codes (2^29),
// stay below the skip offset.
constexpr int64_t kFewMaxK = int64_t(1) << 24;

// S > 1: the activation rows come in slices of 16 (MAXM = 16), each
// decoded into the wave's LDS area in turn and multiplied with the weight
// pieces of the chunk, which are decoded once for all slices.
//
// Split K (gridDim.y = parts > 1, fp32 output only): workgroup row y takes
// the chunks [C y / parts, C (y + 1) / parts) of the C chunks, which its
// waves interleave as they would all of them, and writes its partial
// products to the y-th M x N fp32 slab of the output; a second kernel adds
// the slabs in order.  With one part this is the unsplit product.
template <bool RES, bool ZBF16, bool WBF16, int NR, int MAXM, int WAVES, int S = 1>
__global__ __launch_bounds__(WAVES * 64) void hif4_gemm_few_kernel(
    const uint8_t *__restrict__ qc, const uint32_t *__restrict__ qm,
    const uint8_t *__restrict__ rc, const uint32_t *__restrict__ rm,
    const uint8_t *__restrict__ wc, const uint32_t *__restrict__ wm,
    const uint16_t *__restrict__ wv, int64_t M, int64_t N, int64_t K, void *__restrict__ z) {
  static_assert(NR == 16 || NR == 32 || NR == 64, "weight rows per workgroup");
  static_assert(S == 1 || MAXM == kFewRows, "slices of 16 activation rows");
  constexpr int F = NR / 16, kFewWaves = WAVES;
  static_assert(F * S <= 8, "partial sums of at most 8 output tiles per wave");
  __shared__ __attribute__((aligned(16))) uint8_t xarea[kFewWaves][2 * kFewRows * kFewXRow];
  __shared__ v4f part[kFewWaves][F * S][64];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, g = lane >> 4;
  const int64_t n0 = (int64_t)blockIdx.x * NR;
  const int64_t kbytes = K / 2, kblocks = K / kH;
  const int nchunks = (int)((K + kFewChunk - 1) / kFewChunk);
  const int kpart = (int)blockIdx.y, kparts = (int)gridDim.y;
  const int cb = (nchunks * kpart) / kparts, ce = (nchunks * (kpart + 1)) / kparts;
  const int slices = S == 1 ? 1 : (int)min<int64_t>(S, (M + kFewRows - 1) / kFewRows);
  // Rows of this workgroup's buffers: NR weight rows from n0 (clamped to N).
  const int64_t nrows = min<int64_t>(NR, N - n0);
  auto rsrc = [](const void *p, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes,
                                             0x00020000);
  };
  const __amdgpu_buffer_rsrc_t bw =
      WBF16 ? rsrc(wv + n0 * K, nrows * K * 2) : rsrc(wc + n0 * kbytes, nrows * kbytes);
  const __amdgpu_buffer_rsrc_t bwm = rsrc(WBF16 ? nullptr : wm + n0 * kblocks, nrows * kblocks * 4);
  uint32_t w_off[F], wm_off[F];
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int64_t lr = min<int64_t>(16 * f + r, nrows - 1);
    w_off[f] = WBF16 ? (uint32_t)(lr * K * 2 + 64 * g) : (uint32_t)(lr * kbytes + 16 * g);
    wm_off[f] = (uint32_t)(lr * kblocks + (g >> 1)) * 4u;
  }

  // Activation work items (one slice): code word w (0..15) of row j of the
  // chunk, j < M primary rows then M residual rows (M <= MAXM); lane l
  // takes items l + 64 i.
  constexpr int kXI = (RES ? 2 : 1) * MAXM * 16 / 64;
  const __amdgpu_buffer_rsrc_t bq = rsrc(qc, M * kbytes), br = rsrc(RES ? rc : qc, M * kbytes);
  const __amdgpu_buffer_rsrc_t bqm = rsrc(qm, M * kblocks * 4),
                               brm = rsrc(RES ? rm : qm, M * kblocks * 4);
  // Item i of this lane: residual or primary, its activation row and word.
  struct XItem {
    bool res;
    int row, w;
  };
  auto xitem = [&](int i, int ms) {
    const int t = lane + 64 * i, j = t >> 4;
    const bool is_r = RES && j >= ms;
    return XItem{is_r, is_r ? j - ms : j, t & 15};
  };

  struct WChunk {
    u32x4 w[F][WBF16 ? 4 : 1];
    uint32_t m[F];
  };
  struct XChunk {
    uint32_t c[kXI], m[kXI];
  };
  auto load_w = [&](int c, WChunk &o) {
    // Quarter g of chunk c exists when 128 c + 32 g < K (K is a multiple of 64).
    const bool live = (int64_t)kFewChunk * c + 32 * g < K;
#pragma unroll
    for (int f = 0; f < F; ++f) {
      if constexpr (WBF16) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          o.w[f][jj] = __builtin_amdgcn_raw_buffer_load_b128(
              bw, live ? w_off[f] + 16 * jj : kFewSkip, kFewChunk * 2 * c, 0);
      } else {
        o.w[f][0] = __builtin_amdgcn_raw_buffer_load_b128(bw, live ? w_off[f] : kFewSkip,
                                                          (kFewChunk / 2) * c, 0);
        o.m[f] = __builtin_amdgcn_raw_buffer_load_b32(bwm, live ? wm_off[f] : kFewSkip, 8 * c, 0);
      }
    }
  };
  auto load_x = [&](int c, int s, XChunk &o) {
    if constexpr (S == 1) {
      const int ms = (int)M;
#pragma unroll
      for (int i = 0; i < kXI; ++i) {
        if (lane + 64 * i < (RES ? 2 : 1) * ms * 16) {
          const XItem it = xitem(i, ms);
          const bool xl = (int64_t)kFewChunk * c + 8 * it.w < K;
          const uint32_t off = (uint32_t)it.row * (uint32_t)kbytes + 4 * it.w;
          const uint32_t moff = ((uint32_t)it.row * (uint32_t)kblocks + (it.w >> 3)) * 4u;
          o.c[i] = __builtin_amdgcn_raw_buffer_load_b32(it.res ? br : bq, xl ? off : kFewSkip,
                                                        (kFewChunk / 2) * c, 0);
          o.m[i] = __builtin_amdgcn_raw_buffer_load_b32(it.res ? brm : bqm, xl ? moff : kFewSkip,
                                                        8 * c, 0);
        }
      }
    } else {
      // Whole 16-row slices: item i is word t mod 16 of row (t / 16) mod 16
      // of the slice, residual for t >= 256 (t = lane + 64 i); rows at or
      // past M load zeros without memory access.  The slice's row offset
      // goes into the scalar offset, so the per-item offsets are the same
      // for every slice.
      const uint32_t sc = (uint32_t)(kFewRows * s) * (uint32_t)kbytes + (kFewChunk / 2) * c;
      const uint32_t sm = (uint32_t)(kFewRows * s) * (uint32_t)kblocks * 4u + 8 * c;
#pragma unroll
      for (int i = 0; i < kXI; ++i) {
        const int t = lane + 64 * i, row = (t >> 4) & 15, w = t & 15;
        const bool res = RES && t >= 256;
        const bool xl = kFewRows * s + row < M && (int64_t)kFewChunk * c + 8 * w < K;
        const uint32_t off = (uint32_t)row * (uint32_t)kbytes + 4 * w;
        const uint32_t moff = ((uint32_t)row * (uint32_t)kblocks + (w >> 3)) * 4u;
        o.c[i] = __builtin_amdgcn_raw_buffer_load_b32(res ? br : bq, xl ? off : kFewSkip, sc, 0);
        o.m[i] = __builtin_amdgcn_raw_buffer_load_b32(res ? brm : bqm, xl ? moff : kFewSkip, sm, 0);
      }
    }
  };

  uint8_t *X = xarea[wave];
  v4f acc[S][F];
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int f = 0; f < F; ++f) acc[s][f] = v4f{0.f, 0.f, 0.f, 0.f};
  WChunk wcur, wnxt;
  XChunk xcur, xnxt;
  if (cb + wave < ce) {
    load_w(cb + wave, wcur);
    load_x(cb + wave, 0, xcur);
  }
  // The next unit's activation codes (the next slice, or the next chunk's
  // first) are requested before a unit is decoded.
  auto load_next_x = [&](int c, int s) {
    if (s + 1 < slices) load_x(c, s + 1, xnxt);
    else if (c + kFewWaves < ce) load_x(c + kFewWaves, 0, xnxt);
  };
  for (int c = cb + wave; c < ce; c += kFewWaves) {
    if (c + kFewWaves < ce) load_w(c + kFewWaves, wnxt);
    u32x4 wp[F][4];
#pragma unroll
    for (int s = 0; s < S; ++s) {
      if (s < slices) {
        load_next_x(c, s);
        // Activation rows of the slice into the wave's LDS area.
        if constexpr (S == 1) {
          const int ms = (int)M;
#pragma unroll
          for (int i = 0; i < kXI; ++i) {
            if (lane + 64 * i < (RES ? 2 : 1) * ms * 16) {
              const XItem it = xitem(i, ms);
              *reinterpret_cast<u32x4 *>(X + few_xoff(it.res ? kFewRows + it.row : it.row, it.w)) =
                  decode8_bf16(xcur.c[i], xcur.m[i], it.w & 7);
            }
          }
        } else {
#pragma unroll
          for (int i = 0; i < kXI; ++i) {
            const int t = lane + 64 * i, row = (t >> 4) & 15, w = t & 15;
            const bool res = RES && t >= 256;
            *reinterpret_cast<u32x4 *>(X + few_xoff(res ? kFewRows + row : row, w)) =
                decode8_bf16(xcur.c[i], xcur.m[i], w & 7);
          }
        }
        // Weight pieces in registers, once per chunk for all its slices.
        if (s == 0) {
#pragma unroll
          for (int f = 0; f < F; ++f) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              if constexpr (WBF16) {
                wp[f][jj] = wcur.w[f][jj];
              } else {
                const uint32_t words[4] = {wcur.w[f][0].x, wcur.w[f][0].y, wcur.w[f][0].z,
                                           wcur.w[f][0].w};
                wp[f][jj] = decode8_bf16(words[jj], wcur.m[f], 4 * (g & 1) + jj);
              }
            }
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const v8bf xq = *reinterpret_cast<const v8bf *>(X + few_xoff(r, 4 * g + jj));
          v8bf xr = xq;
          if constexpr (RES)
            xr = *reinterpret_cast<const v8bf *>(X + few_xoff(kFewRows + r, 4 * g + jj));
#pragma unroll
          for (int f = 0; f < F; ++f) {
            const v8bf wf = __builtin_bit_cast(v8bf, wp[f][jj]);
            acc[s][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, xq, acc[s][f], 0, 0, 0);
            if constexpr (RES)
              acc[s][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, xr, acc[s][f], 0, 0, 0);
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        xcur = xnxt;
      }
    }
    wcur = wnxt;
  }
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int f = 0; f < F; ++f) part[wave][f * S + s][lane] = acc[s][f];
  __syncthreads();
  // Output tile p (weight fragment p / S, slice p mod S), summed in wave
  // order and stored by wave p mod WAVES.
  const bool vec_ok = (N & 3) == 0;
  for (int p = wave; p < F * S; p += kFewWaves) {
    const int f = p / S, s = p % S;
    const int64_t m = (int64_t)kFewRows * s + r;
    if (s >= slices || m >= M) continue;
    v4f t = part[0][p][lane];
#pragma unroll
    for (int w = 1; w < kFewWaves; ++w) t += part[w][p][lane];
    const int64_t n = n0 + 16 * f + 4 * g;
    if constexpr (ZBF16) {
      uint16_t *zp = reinterpret_cast<uint16_t *>(z) + m * N + n;
      if (vec_ok && n + 3 < N) {
        uint2 o;
        o.x = bf16x2_rne(t[0], t[1]);
        o.y = bf16x2_rne(t[2], t[3]);
        *reinterpret_cast<uint2 *>(zp) = o;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < N) zp[e] = (uint16_t)bf16_rne(t[e]);
      }
    } else {
      float *zp = reinterpret_cast<float *>(z) + kpart * M * N + m * N + n;
      if (vec_ok && n + 3 < N) {
        *reinterpret_cast<float4 *>(zp) = make_float4(t[0], t[1], t[2], t[3]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < N) zp[e] = t[e];
      }
    }
  }
}

template <bool RES, bool ZBF16, bool WBF16, int BN, bool SPLIT = false>
hipError_t launch_tiles(const uint8_t *qc, const uint32_t *qm, const uint8_t *rc,
                        const uint32_t *rm, const uint8_t *wc, const uint32_t *wm,
                        const uint16_t *wv, int64_t M, int64_t N, int64_t K, void *z,
                        hipStream_t stream, int parts = 1, int64_t ksplit = 0) {
  using S = HSmem<RES, BN>;
  auto kern = hif4_gemm_kernel<RES, ZBF16, WBF16, BN, SPLIT>;
  static std::atomic<bool> attr_done[kMaxDevices];
  const hipError_t e = set_lds_limit(attr_done, reinterpret_cast<const void *>(kern), S::kBytes);
  if (e != hipSuccess) return e;
  const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + BN - 1) / BN);
  kern<<<dim3((unsigned)(tiles * parts)), dim3(S::kThreads), S::kBytes, stream>>>(
      qc, qm, rc, rm, wc, wm, wv, M, N, K, z, SPLIT ? ksplit : K);
  return hipGetLastError();
}

// Workgroups that fill the chip once (256 CUs on MI355X).
constexpr int64_t kFillTiles = 256;

// The few-row kernel's sizes (K and its grid) and row counts: up to 64 rows,
// and 65-128 rows at N <= 4096, there as two launches on 64-row halves (the
// tile kernel has at most 32 tiles there, each with the whole reduction:
// 96 rows x 4096 x 12288 314 -> 175 us; every row's result is the few-row
// kernel's for that row).
bool few_fits(int64_t N, int64_t K) {
  return K <= kFewMaxK && (N + 15) / 16 <= int64_t(UINT32_MAX / 1024);
}
bool few_halves(int64_t M, int64_t N, int64_t K) {
  return few_fits(N, K) && M > kFewMaxRows && M <= 2 * kFewMaxRows && N <= 4096;
}
bool few_rows_product(int64_t M, int64_t N, int64_t K) {
  return (M <= kFewMaxRows && few_fits(N, K)) || few_halves(M, N, K);
}

// Workgroup shape of the few-row kernel for M activation rows against N
// weight rows: weight rows per workgroup, activation rows per slice, waves,
// slices.  Eight waves per workgroup (sixteen up to 8 rows where N <= 4096:
// the grid then holds at most 256 workgroups, and K splits further: 1 row
// x 4096 x 12288 20.9 -> 17.3 us, 8 rows 29.6 -> 25.1 us), the same in both
// weight forms, so that both add every output's partial sums in the same
// order.  Weight rows per workgroup: 16 up to 4 activation rows.  Above,
// every workgroup decodes all activation rows again, so more weight rows per
// workgroup spread that decode, as long as the grid keeps about one
// workgroup per CU (one fits per CU at these register counts): 64 from N =
// 11264 (176 or more workgroups; 32 for the bf16-weight form, whose 64-row
// variant spills), 32 above N = 4096, 16 up to it (256 workgroups at most).
// Measured at 16 rows: 12288 x 4096 weights 35.4 -> 27.5 us against 32 rows
// and four waves, 4096 x 12288 52.2 -> 43.9 us against 32 rows.
struct FewShape {
  int nr, maxm, waves, slices;
};
FewShape few_shape(int64_t M, int64_t N, bool wbf16) {
  const bool wide = !wbf16 && N >= 11264, narrow = N <= 4096;
  const int nr = narrow ? 16 : (wide ? 64 : 32);
  if (M <= 4) return FewShape{16, 4, narrow ? 16 : 8, 1};
  if (M <= 8) return FewShape{nr, 8, narrow ? 16 : 8, 1};
  if (M <= kFewRows) return FewShape{nr, 16, 8, 1};
  if (M <= 2 * kFewRows) return FewShape{nr, 16, 8, 2};
  return FewShape{narrow ? 16 : 32, 16, 8, 4};
}

// Parts of K for the few-row kernel given a workspace (1: unsplit; never
// with the two launches on row halves).  The grid's g workgroups run in
// rounds of 256 (one per CU); where the last round is partly empty, p parts
// (g p workgroups, each a p-th of K) fill it better.  Parts are taken where
// they raise the filled fraction of the last round, (g p / 256) /
// ceil(g p / 256), by at least 0.2 (the sum kernel and the shorter K loops
// cost the rest: a gain of 0.15 at 1 row x 9216 x 4096 measured 16.2 ->
// 17.0 us), every wave keeps at least two chunks of 128, and the workgroups
// have 8 waves (the 16-wave shapes up to 8 rows at N <= 4096 already split
// K finely: 1 row x 3072 x 16384 20.0 -> 21.7 us with 4 parts).  Measured
// (bf16 Z, sum included): 5120 x 13824 weights (160 workgroups; 320 up to 4
// rows), 1 row 29.7 -> 23.2 us (4 parts), 8 rows 39.4 -> 29.2, 16 rows
// 52.3 -> 40.4, 64 rows 114.0 -> 80.3 (3 parts); 64 rows x 12288 x 4096 (384
// workgroups) 71.9 -> 61.1 (2 parts); where the grid fills its rounds (4096
// x 12288: 256 workgroups) or a wave would keep one chunk (12288 x 4096 up
// to 32 rows), every split was slower.
int few_split_parts(int64_t M, int64_t N, int64_t K) {
  if (M > kFewMaxRows || !few_fits(N, K)) return 1;
  const FewShape f = few_shape(M, N, false);
  if (f.waves != 8) return 1;
  const int64_t g = (N + f.nr - 1) / f.nr;
  const int64_t nchunks = (K + kFewChunk - 1) / kFewChunk;
  auto filled = [&](int64_t p) {
    const int64_t wgs = g * p, rounds = (wgs + kFillTiles - 1) / kFillTiles;
    return double(wgs) / double(rounds * kFillTiles);
  };
  int best = 1;
  double fb = filled(1);
  for (int p = 2; p <= 4; ++p) {
    if (nchunks < int64_t(2) * p * f.waves) break;
    const double fp = filled(p);
    if (fp >= filled(1) + 0.2 && fp > fb) {
      best = p;
      fb = fp;
    }
  }
  return best;
}

template <bool RES, bool ZBF16, bool WBF16>
hipError_t launch_hg(const uint8_t *qc, const uint32_t *qm, const uint8_t *rc,
                     const uint32_t *rm, const uint8_t *wc, const uint32_t *wm,
                     const uint16_t *wv, int64_t M, int64_t N, int64_t K, void *z,
                     hipStream_t stream, int parts = 1) {
  if (few_halves(M, N, K)) {
    const int64_t kb = K / 2, km = K / kH;
    hipError_t e = launch_hg<RES, ZBF16, WBF16>(qc, qm, rc, rm, wc, wm, wv, kFewMaxRows, N, K, z,
                                                stream);
    if (e != hipSuccess) return e;
    const int64_t r0 = kFewMaxRows;
    return launch_hg<RES, ZBF16, WBF16>(qc + r0 * kb, qm + r0 * km, RES ? rc + r0 * kb : rc,
                                        RES ? rm + r0 * km : rm, wc, wm, wv, M - r0, N, K,
                                        static_cast<uint8_t *>(z) + r0 * N * (ZBF16 ? 2 : 4),
                                        stream);
  }
  if (M <= kFewMaxRows && few_fits(N, K)) {
#define RFQ_FEW_S(NR, MAXM, W, S)                                                              \
  if (f.nr == NR && f.maxm == MAXM && f.waves == W && f.slices == S) {                         \
    hif4_gemm_few_kernel<RES, ZBF16, WBF16, NR, MAXM, W, S>                                    \
        <<<dim3((unsigned)((N + NR - 1) / NR), (unsigned)parts), dim3(W * 64), 0, stream>>>(    \
            qc, qm, rc, rm, wc, wm, wv, M, N, K, z);                                           \
    return hipGetLastError();                                                                  \
  }
    const FewShape f = few_shape(M, N, WBF16);
    RFQ_FEW_S(16, 4, 16, 1) RFQ_FEW_S(16, 4, 8, 1)
    RFQ_FEW_S(16, 8, 16, 1) RFQ_FEW_S(32, 8, 8, 1)
    RFQ_FEW_S(16, 16, 8, 1) RFQ_FEW_S(32, 16, 8, 1)
    RFQ_FEW_S(16, 16, 8, 2) RFQ_FEW_S(32, 16, 8, 2)
    RFQ_FEW_S(16, 16, 8, 4) RFQ_FEW_S(32, 16, 8, 4)
    if constexpr (!WBF16) {
      RFQ_FEW_S(64, 8, 8, 1) RFQ_FEW_S(64, 16, 8, 1) RFQ_FEW_S(64, 16, 8, 2)
    }
#undef RFQ_FEW_S
    return hipErrorInvalidValue;
  }
  if (((M + kBM - 1) / kBM) * ((N + 255) / 256) < kFillTiles)
    return launch_tiles<RES, ZBF16, WBF16, 128>(qc, qm, rc, rm, wc, wm, wv, M, N, K, z, stream);
  return launch_tiles<RES, ZBF16, WBF16, 256>(qc, qm, rc, rm, wc, wm, wv, M, N, K, z, stream);
}


template <int STEPS>
hipError_t launch_hq(const void *x, bool bf16_in, int64_t nunits, uint8_t *qc, uint32_t *qm,
                     uint8_t *rc, uint32_t *rm, hipStream_t stream) {
  const int64_t per_wg = (kQThreads / 64) * 64 * STEPS;
  const dim3 grid((unsigned)((nunits + per_wg - 1) / per_wg)), block(kQThreads);
  if (bf16_in) {
    if (rc)
      hif4_quantize_kernel<true, true, STEPS><<<grid, block, 0, stream>>>(x, nunits, qc, qm, rc, rm);
    else
      hif4_quantize_kernel<true, false, STEPS><<<grid, block, 0, stream>>>(x, nunits, qc, qm,
                                                                          nullptr, nullptr);
  } else {
    if (rc)
      hif4_quantize_kernel<false, true, STEPS><<<grid, block, 0, stream>>>(x, nunits, qc, qm, rc,
                                                                          rm);
    else
      hif4_quantize_kernel<false, false, STEPS><<<grid, block, 0, stream>>>(x, nunits, qc, qm,
                                                                           nullptr, nullptr);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_hif4_quantize(const void *x, bool bf16_in, int64_t nelem, uint8_t *q_codes,
                                uint32_t *q_meta, uint8_t *r_codes, uint32_t *r_meta,
                                hipStream_t stream) {
  const int64_t nunits = nelem / 8;
  if (nunits < kQSmallUnits)
    return launch_hq<1>(x, bf16_in, nunits, q_codes, q_meta, r_codes, r_meta, stream);
  return launch_hq<kQSteps>(x, bf16_in, nunits, q_codes, q_meta, r_codes, r_meta, stream);
}

hipError_t launch_hif4_dequant(const uint8_t *codes, const uint32_t *meta, int64_t nelem,
                               void *out, bool bf16_out, hipStream_t stream) {
  const int64_t nunits = nelem / 8;
  const int64_t wgs = (nunits + 255) / 256;
  const unsigned grid = (unsigned)(wgs < kLoopGrid ? wgs : kLoopGrid);
  const uint32_t *c = reinterpret_cast<const uint32_t *>(codes);
  if (bf16_out)
    hif4_dequant_kernel<true><<<grid, 256, 0, stream>>>(c, meta, nunits, out);
  else
    hif4_dequant_kernel<false><<<grid, 256, 0, stream>>>(c, meta, nunits, out);
  return hipGetLastError();
}

hipError_t launch_hif4_gemm(const uint8_t *q_codes, const uint32_t *q_meta,
                            const uint8_t *r_codes, const uint32_t *r_meta,
                            const uint8_t *w_codes, const uint32_t *w_meta,
                            const uint16_t *w_bf16, int64_t M, int64_t N, int64_t K, void *z,
                            bool z_bf16, hipStream_t stream) {
  const bool res = r_codes != nullptr, wb = w_bf16 != nullptr;
#define RFQ_HG(R, Z, W) \
  if (res == R && z_bf16 == Z && wb == W) \
    return launch_hg<R, Z, W>(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta, w_bf16, M, N, \
                              K, z, stream);
  RFQ_HG(true, true, false) RFQ_HG(true, false, false) RFQ_HG(false, true, false)
  RFQ_HG(false, false, false) RFQ_HG(true, true, true) RFQ_HG(true, false, true)
  RFQ_HG(false, true, true) RFQ_HG(false, false, true)
#undef RFQ_HG
  return hipErrorInvalidValue;
}

// Split of K over 128-wide tiles: where those number at most 128 (a few
// hundred activation rows against a narrow weight, the down projection of an
// MLP), 256 / tiles parts (at most 8) of at least 4 blocks each, so that
// parts x tiles workgroups fill the 256 CUs about once; the partials take
// parts x M x N x 4 <= 16 MiB.
static SplitPlan tile_split_plan(int64_t M, int64_t N, int64_t K) {
  SplitPlan p{1, K, 0};
  if (((M + kBM - 1) / kBM) * ((N + 255) / 256) >= kFillTiles) return p;
  const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + 127) / 128);
  if (tiles > 128) return p;
  constexpr int64_t kMinBlocks = 4;
  const int64_t blocks = K / kH;
  const int64_t want = std::min<int64_t>(std::min<int64_t>(8, 256 / tiles), blocks / kMinBlocks);
  if (want < 2) return p;
  const int64_t per = (blocks + want - 1) / want;
  p.parts = (int)((blocks + per - 1) / per);
  if (p.parts < 2) return SplitPlan{1, K, 0};
  p.ksplit = per * kH;
  p.work_bytes = (int64_t)p.parts * M * N * 4;
  return p;
}

// With a workspace the tile split also replaces the few-row kernel where it
// splits, from 49 activation rows; where N <= 4096, from 24 rows with K >=
// 12288 and from 40 below.  Measured (bf16 Z, the few-row kernel split or
// not by its own rule): 64 rows x 4096 x 12288 91.2 -> 47.7 us, 128 rows
// (two launches on halves) 183.4 -> 54.2, 24 rows 50.5 -> 45.3, 16 rows
// 40.6 against 44.6; 64 rows x 5120 x 13824 80.1 -> 65.1, 48 rows 64.2
// against 63.9; 64 rows x 13824 x 5120 88.5 -> 72.9; 64 rows x 12288 x 4096
// 61.6 -> 59.6, 48 rows 50.4 against 58.0; 4096 x 4096 weights 48 rows 25.9
// -> 22.4, 96 rows 50.8 -> 26.9, 32 rows 18.7 against 21.1.
static bool split_on_tiles(int64_t M, int64_t N, int64_t K, const SplitPlan &tiles) {
  if (!few_rows_product(M, N, K)) return true;
  if (tiles.parts < 2) return false;
  const int64_t from = N <= 4096 ? (K >= 12288 ? 24 : 40) : 49;
  return M >= from;
}

// Without a split, from this many rows the weights are decoded to bf16 once
// into the workspace and the bf16-weight product runs on them (the same bits
// as the codes form, whose tile rows each decode all of W again).  Measured
// (bf16 Z, decode included): 4096 rows x 4096 x 12288 832 -> 740 us, 4096 x
// 12288 x 4096 847 -> 754-780, 4096 x 13824 x 5120 1218 -> 1084-1100, 1024
// rows x 12288 x 4096 268 -> 249; at 512 rows no gain (220 against 228).
constexpr int64_t kDecodeMinRows = 1024;
constexpr int64_t kDecodeMaxBytes = int64_t(1) << 30;

SplitPlan hif4_split_plan(int64_t M, int64_t N, int64_t K) {
  SplitPlan p{1, K, 0};
  if (M <= 0 || N <= 0 || K < kH || K % kH) return p;
  const SplitPlan tiles = tile_split_plan(M, N, K);
  if (tiles.parts < 2 && !few_rows_product(M, N, K) && M >= kDecodeMinRows &&
      N * K * 2 <= kDecodeMaxBytes) {
    p.decode_w = true;
    p.work_bytes = N * K * 2;
    return p;
  }
  if (split_on_tiles(M, N, K, tiles)) return tiles;
  p.few_rows = true;
  p.parts = few_split_parts(M, N, K);
  if (p.parts > 1) p.work_bytes = (int64_t)p.parts * M * N * 4;
  return p;
}

hipError_t launch_hif4_gemm_split(const uint8_t *q_codes, const uint32_t *q_meta,
                                  const uint8_t *r_codes, const uint32_t *r_meta,
                                  const uint8_t *w_codes, const uint32_t *w_meta, int64_t M,
                                  int64_t N, int64_t K, void *z, bool z_bf16, float *work,
                                  int64_t work_bytes, hipStream_t stream) {
  const SplitPlan p = hif4_split_plan(M, N, K);
  if (p.decode_w && work != nullptr && work_bytes >= p.work_bytes) {
    uint16_t *wv = reinterpret_cast<uint16_t *>(work);
    const hipError_t e = launch_hif4_dequant(w_codes, w_meta, N * K, wv, true, stream);
    if (e != hipSuccess) return e;
    return launch_hif4_gemm(q_codes, q_meta, r_codes, r_meta, nullptr, nullptr, wv, M, N, K, z,
                            z_bf16, stream);
  }
  if (p.parts < 2 || work == nullptr || work_bytes < p.work_bytes)
    return launch_hif4_gemm(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta, nullptr, M, N, K,
                            z, z_bf16, stream);
  if (p.few_rows) {
    const hipError_t e =
        r_codes ? launch_hg<true, false, false>(q_codes, q_meta, r_codes, r_meta, w_codes, w_meta,
                                                nullptr, M, N, K, work, stream, p.parts)
                : launch_hg<false, false, false>(q_codes, q_meta, nullptr, nullptr, w_codes,
                                                 w_meta, nullptr, M, N, K, work, stream, p.parts);
    if (e != hipSuccess) return e;
    return launch_splitk_sum(work, p.parts, M * N, z, z_bf16, stream);
  }
  const hipError_t e =
      r_codes ? launch_tiles<true, false, false, 128, true>(q_codes, q_meta, r_codes, r_meta,
                                                             w_codes, w_meta, nullptr, M, N, K,
                                                             work, stream, p.parts, p.ksplit)
              : launch_tiles<false, false, false, 128, true>(q_codes, q_meta, nullptr, nullptr,
                                                              w_codes, w_meta, nullptr, M, N, K,
                                                              work, stream, p.parts, p.ksplit);
  if (e != hipSuccess) return e;
  return launch_splitk_sum(work, p.parts, M * N, z, z_bf16, stream);
}

}  // namespace rfq
