// RFQ product, large-tile kernel for K a multiple of 512 (Eq. 11, Algorithm 1
// with phi = 1; phi = 0 without the residual operand).
//
// Output tile 256 x 256 per workgroup of 8 waves (4 x 2, each wave 64 x 128
// = 2 x 4 fragments of 32 x 32), one workgroup per CU and two waves per SIMD:
// while one wave waits on LDS or global loads the other issues MFMAs.
// (Measured on 4096 x 4096 x 12288, bit-identical outputs: 4 waves of
// 128 x 128 with one wave per SIMD idled the matrix core on every wait; two
// 4-wave 128 x 256 workgroups per CU were 5-6% faster than that; this layout,
// which loads a quarter fewer operand bytes per output than the two
// workgroups, is another 4% faster.  The cost of the global loads lies in the
// load instructions themselves: pointing them at always-cached data does not
// change the time.)  Where the 256 x 256 tiles would leave CUs idle, the same
// code runs 128 x 128 tiles (4 waves of 64 x 64, up to three workgroups per
// CU); each output is accumulated in the same order in both shapes, so they
// give the same bits.
//
// Instruction: v_mfma_scale_f32_32x32x64_f8f6f4 with E2M1 operands: lane l
// of an operand holds row (l mod 32) and 32 consecutive K values (one MX
// block) and supplies that block's scale byte; the 32 x 32 fp32 result gives
// lane l the rows 8a + 4(l/32) + 0..3 (a = 0..3) of column (l mod 32).  With
// weights as the first operand those are runs of four consecutive outputs
// of one row of Z.  (On gfx950 this form sustains about 7.6 PFLOP/s of FP4
// against about 6.1 for the 16x16x128 form in register-only loops.)
//
// One stage is 128 K values = 4 MX blocks = two k-steps: lane half h takes
// blocks 2h (k-step 0) and 2h+1 (k-step 1) - the contraction order inside an
// instruction is free as long as both operands use the same assignment - so
// a fragment is one 16-byte chunk per k-step and one 16-bit scale pair per
// stage (op_sel picks the byte).  Every weight fragment feeds the primary and
// the residual MFMA, which is the residual contraction sharing the weight
// tile.
//
// Pipeline per stage st (two LDS stage buffers of 52 KiB, one barrier per stage): the
// fragments of stage st are read from buffer st mod 2 and multiplied while
// stage st+1, held in registers, is written to the other buffer (its previous
// contents were last read before the barrier that ended stage st-1); then
// stage st+2 is fetched into the registers.  Loads go through buffer
// descriptors (scalar base and size, a 32-bit offset per load).  Scale bytes
// arrive 16 per row every four stages (a 4-byte fetch per row and stage costs
// a whole L2 request for 4 useful bytes).  Inside LDS the 16-byte chunks of a
// row are XOR-swizzled by row, so the 16 rows served together by one 16-byte
// read hit distinct banks.
//
// Epilogue: each wave stages its results through LDS (padded rows) and
// writes Z with 16-byte stores covering whole row segments.  The SwiGLU
// epilogue instead takes the product of interleaved gate/up weights (32-row
// groups: gate rows 32g.., then up rows 32g..), so that columns 64g..64g+31
// of Z are g and 64g+32..64g+63 are u for the same 32 hidden units: it rounds
// both to bf16 as a bf16 Z would be, forms h = bf16(silu(g) u) and quantizes
// each 32-wide block of h (primary and residual, Eq. 8-10) from registers,
// with the same arithmetic as the standalone SwiGLU quantizer.
//
// Rows past M or N are clamped to the last row for loading (their results
// are never stored), so no load leaves its tensor.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "gemm_common.h"
#include "mx_device.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

// Workgroup tile: WM x WN waves, each 64 rows x 32 FN columns (2 x FN
// fragments of 32 x 32).
template <int WM, int WN, int FN>
struct Tile {
  static constexpr int kThreads = 64 * WM * WN;
  static constexpr int kFM = 2, kFN = FN;
  static constexpr int kTM = 32 * kFM, kTN = 32 * FN;   // wave sub-tile
  static constexpr int kBM = kTM * WM, kBN = kTN * WN;  // workgroup tile
  static constexpr int kWaveRows = WM;                  // waves along M
  static constexpr int kWaveCols = WN;
  static constexpr int kRPL = kThreads / 4;             // buffer rows per load step (4 chunks a row)
};
// 256 x 256, 8 waves of 64 x 128, one workgroup per CU, two waves per SIMD.
using Big = Tile<4, 2, 4>;
// 128 x 128, 4 waves of 64 x 64, for products whose 256 x 256 tiles would
// leave CUs idle; up to three workgroups per CU.
using Mid = Tile<2, 2, 2>;

constexpr int kStageK = 128;
constexpr int kRowBytes = kStageK / 2;
constexpr int kGroup = 4;

// LDS stage buffer: rows [0, kBM) q, (RES) [kBM, 2 kBM) r, then kBN weight
// rows, 64 code bytes each; then one 4-byte scale word per row.
template <class C, bool RES>
struct Layout {
  static constexpr int kARows = RES ? 2 * C::kBM : C::kBM;   // q rows, then r rows
  static constexpr int kRows = kARows + C::kBN;
  static constexpr int kWRow = kARows;
  static constexpr int kDataBytes = kRows * kRowBytes;
  static constexpr int kScaleBytes = kRows * 4;
  static constexpr int kStageBytes = kDataBytes + kScaleBytes;
  static constexpr int kBytes = 2 * kStageBytes;
  static constexpr int kLoads = kRows * 4 / C::kThreads;
  static constexpr int kScaleLoads = (kRows + C::kThreads - 1) / C::kThreads;
  static_assert(kRows * 4 % C::kThreads == 0, "whole load steps");
};

// Byte offset of 16-byte chunk c of buffer row r.  LDS serves a 16-byte
// access of 16 lanes at a time across 256 bytes of banks, so the 16
// consecutive rows that one fragment read touches (same chunk) must land in
// 16 distinct 16-byte slots: a row is 4 slots wide, and the XOR with
// (r >> 2) & 3 separates the four rows that share a slot column (with
// (r >> 1) & 3, rows r and r + 8 collided: 2-way conflicts measured as a
// third of the LDS's active cycles).  The stores (4 rows x 4 chunks per 16
// lanes) stay conflict-free.
__device__ __forceinline__ int chunk_off(int r, int c) {
  return r * kRowBytes + 16 * (c ^ ((r >> 2) & 3));
}

__device__ __forceinline__ v8i as_v8i(const u32x4 &d) {
  return v8i{(int)d.x, (int)d.y, (int)d.z, (int)d.w, 0, 0, 0, 0};
}

// Epilogue staging: a wave writes 32 rows x 64 columns of fp32 or bf16 per
// pass; rows are padded by 16 bytes so the 32 rows written together spread
// over the banks.
template <bool ZBF16>
struct Epi {
  static constexpr int kElem = ZBF16 ? 2 : 4;
  static constexpr int kRowStride = 64 * kElem + 16;
  static constexpr int kWaveBytes = 32 * kRowStride;
  static constexpr int kChunksPerRow = 64 * kElem / 16;
};

// Outputs of the SwiGLU epilogue: codes and scales of h [M][nh] (residual
// pair optional) and, when h is not null, h itself in bf16.
struct SwigluOut {
  uint8_t *qc, *qs, *rc, *rs;
  uint16_t *h;
  int64_t nh;
};

// Scale pairs of one stage (both k-steps) for the wave's fragments.
template <class C, bool RES>
struct Scales {
  int w[C::kFN], q[C::kFM], r[RES ? C::kFM : 1];
};

// Instruction classes of the scheduling masks.
constexpr int kMfma = 0x008, kVmemRead = 0x020, kDsRead = 0x100, kDsWrite = 0x200;

// NM MFMAs with NA instructions of class MA and NB of class MB spread evenly
// between them (each MFMA is followed by its share).
template <int NM, int NA, int MA, int NB = 0, int MB = kVmemRead, int I = 0>
__device__ __forceinline__ void spread() {
  if constexpr (I < NM) {
    constexpr int na = (NA * (I + 1)) / NM - (NA * I) / NM;
    constexpr int nb = (NB * (I + 1)) / NM - (NB * I) / NM;
    __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
    if constexpr (na > 0) __builtin_amdgcn_sched_group_barrier(MA, na, 0);
    if constexpr (nb > 0) __builtin_amdgcn_sched_group_barrier(MB, nb, 0);
    spread<NM, NA, MA, NB, MB, I + 1>();
  }
}

// N LDS reads, issued before anything that follows in the region.
template <int N>
__device__ __forceinline__ void reads_first() {
  if constexpr (N > 0) __builtin_amdgcn_sched_group_barrier(kDsRead, N, 0);
}

// SwiGLU epilogue of one wave.  Fragment pair p of fragment row i holds g
// (fragment 2p) and u (fragment 2p+1) of h block (n_base + 64 p) / 64 for
// row m_base + 32 i.  Lane l has 16 of the block's 32 values, positions
// 8a + 4(l/32) + v for accumulator element 4a + v; the other 16 are in lane
// l ^ 32.  The block maximum and the 16-bit code pieces are exchanged with
// that lane; the lower lane stores the primary codes, the upper the residual.
template <class C, bool HRES>
__device__ __forceinline__ void swiglu_epilogue(const v16f (&acc)[C::kFM][C::kFN],
                                                const SwigluOut so, int64_t M, int64_t m_base,
                                                int64_t n_base, int h) {
  const int64_t nblk = so.nh / 32;
#pragma unroll
  for (int i = 0; i < C::kFM; ++i) {
#pragma unroll
    for (int p = 0; p < C::kFN / 2; ++p) {
      const v16f &ag = acc[i][2 * p], &au = acc[i][2 * p + 1];
      const int64_t m = m_base + 32 * i;
      const int64_t blk = (n_base + 64 * p) / 64;
      // g, u and h rounded to bf16 in pairs by the hardware conversion (the
      // bits of the integer rounding the standalone SwiGLU quantizer uses).
      float hv[16];
      uint32_t hpair[8];
      float am = 0.0f;
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const uint32_t gp = bf16x2_rne(ag[e], ag[e + 1]), up = bf16x2_rne(au[e], au[e + 1]);
        hpair[e / 2] = bf16x2_rne(
            swiglu_f32(__uint_as_float(gp << 16), __uint_as_float(up << 16)),
            swiglu_f32(__uint_as_float(gp & 0xFFFF0000u), __uint_as_float(up & 0xFFFF0000u)));
        hv[e] = __uint_as_float(hpair[e / 2] << 16);
        hv[e + 1] = __uint_as_float(hpair[e / 2] & 0xFFFF0000u);
        am = fmaxf(am, fmaxf(fabsf(hv[e]), fabsf(hv[e + 1])));
      }
      am = fmaxf(am, __shfl_xor(am, 32));
      const uint32_t qb = scale_byte(am);
      const float qsc = scale_operand(qb);
      uint32_t qp[4], rp[4] = {0, 0, 0, 0}, rb = 0;
#pragma unroll
      for (int a = 0; a < 4; ++a)
        qp[a] = encode4(hv[4 * a], hv[4 * a + 1], hv[4 * a + 2], hv[4 * a + 3], qsc);
      if constexpr (HRES) {
        float r[16], ram = 0.0f;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          float d[4];
          decode4(qp[a], qsc, d);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            r[4 * a + v] = hv[4 * a + v] - d[v];
            ram = fmaxf(ram, fabsf(r[4 * a + v]));
          }
        }
        ram = fmaxf(ram, __shfl_xor(ram, 32));
        rb = scale_byte(ram);
        const float rsc = scale_operand(rb);
#pragma unroll
        for (int a = 0; a < 4; ++a)
          rp[a] = encode4(r[4 * a], r[4 * a + 1], r[4 * a + 2], r[4 * a + 3], rsc);
      }
      // Bytes 4a, 4a+1 of the block come from the lower lane, 4a+2, 4a+3
      // from the upper: each lane sends the pieces its partner stores.
      const uint32_t s01 = h ? (qp[0] | qp[1] << 16) : (rp[0] | rp[1] << 16);
      const uint32_t s23 = h ? (qp[2] | qp[3] << 16) : (rp[2] | rp[3] << 16);
      const uint32_t g01 = __shfl_xor(s01, 32), g23 = __shfl_xor(s23, 32);
      if (m < M && blk < nblk) {
        const int64_t off = m * (so.nh / 2) + 16 * blk;
        if (h == 0) {
          const u32x4 w = {qp[0] | (g01 << 16), qp[1] | (g01 & 0xFFFF0000u),
                           qp[2] | (g23 << 16), qp[3] | (g23 & 0xFFFF0000u)};
          *reinterpret_cast<u32x4 *>(so.qc + off) = w;
          so.qs[m * nblk + blk] = (uint8_t)qb;
        } else if constexpr (HRES) {
          const u32x4 w = {(g01 & 0xFFFFu) | (rp[0] << 16), (g01 >> 16) | (rp[1] << 16),
                           (g23 & 0xFFFFu) | (rp[2] << 16), (g23 >> 16) | (rp[3] << 16)};
          *reinterpret_cast<u32x4 *>(so.rc + off) = w;
          so.rs[m * nblk + blk] = (uint8_t)rb;
        }
        if (so.h) {
          uint16_t *hp = so.h + m * so.nh + 32 * blk + 4 * h;
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            uint2 w;
            w.x = hpair[2 * a];
            w.y = hpair[2 * a + 1];
            *reinterpret_cast<uint2 *>(hp + 8 * a) = w;
          }
        }
      }
    }
  }
}

// Fallback-indicator map: one byte per tile of kPhiRows activation rows by
// kPhiK reduction columns (a wave's rows by two stages); 256 x 256 tiles only.
constexpr int kPhiRows = 64, kPhiK = 256;
// LDS reserved for the map rows of a workgroup (K up to 2^20).
constexpr int kPhiMapMaxBytes = Big::kWaveRows * ((1 << 20) / kPhiK);

// The product of one workgroup tile (both tile shapes; the kernels below
// fix the shape and the occupancy).  SPLIT: the grid holds ceil(K / ksplit)
// copies of the tile grid, copy s multiplying K columns [s ksplit, (s + 1)
// ksplit) (ksplit a multiple of 512) and writing its fp32 partial product to
// z + s M N.
template <class C, bool RES, bool ZBF16, bool SWIGLU, bool HRES, bool PHI, bool SPLIT = false>
__device__ __forceinline__ void gemm_tile(
    const uint8_t *__restrict__ qc, const uint8_t *__restrict__ qs,
    const uint8_t *__restrict__ rc, const uint8_t *__restrict__ rs,
    const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws,
    int64_t M, int64_t N, int64_t K, void *__restrict__ z, const SwigluOut so,
    const uint8_t *__restrict__ phi, int64_t ksplit) {
  static_assert(!PHI || std::is_same<C, Big>::value, "fallback-indicator maps use 256 x 256 tiles");
  static_assert(!SPLIT || (!ZBF16 && !SWIGLU && !PHI), "split partials are fp32 products");
  using L = Layout<C, RES>;
  constexpr int kBM = C::kBM, kBN = C::kBN, kTM = C::kTM, kTN = C::kTN;
  constexpr int kFM = C::kFM, kFN = C::kFN, kRPL = C::kRPL, kThreads = C::kThreads;
  constexpr int kWaveRows = C::kWaveRows;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

  const int ntm = (int)((M + kBM - 1) / kBM), ntn = (int)((N + kBN - 1) / kBN);
  int bid = blockIdx.x, split = 0;
  if constexpr (SPLIT) {
    split = bid / (ntm * ntn);
    bid -= split * ntm * ntn;
    z = reinterpret_cast<float *>(z) + (int64_t)split * M * N;
  }
  int tm, tn;
  tile_coords<1024 / kBM>(bid, ntm, ntn, tm, tn);
  const int64_t m0 = (int64_t)tm * kBM, n0 = (int64_t)tn * kBN;
  // First K column of this workgroup's range, as code and scale byte offsets.
  const int64_t kb = SPLIT ? (int64_t)split * ksplit : 0;
  const int kb_code = (int)(kb / 2), kb_scale = (int)(kb / 32);

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::kWaveCols, wn = wave % C::kWaveCols;
  const int64_t kbytes = K / 2, kblocks = K / 32;
  const int nstages = (int)((SPLIT ? min(ksplit, K - kb) : K) / kStageK);

  const int trow = tid / 4, tcol = 16 * (tid & 3);
  auto rsrc = [](const uint8_t *p, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(p), (short)0, (int)bytes,
                                             0x00020000);
  };
  const __amdgpu_buffer_rsrc_t cq = rsrc(qc, M * kbytes), cr = rsrc(RES ? rc : qc, M * kbytes),
                               cw = rsrc(wc, N * kbytes);
  const __amdgpu_buffer_rsrc_t sq = rsrc(qs, M * kblocks), sr = rsrc(RES ? rs : qs, M * kblocks),
                               sw = rsrc(ws, N * kblocks);
  // Chunk u of this thread: buffer row trow + kRPL u, chunk tid mod 4.
  // Operand of buffer row block u (kRPL rows): 0 q, 1 r, 2 w.
  auto op_of = [](int u) { return u * kRPL < kBM ? 0 : (RES && u * kRPL < 2 * kBM ? 1 : 2); };
  uint32_t a_off[kBM / kRPL], w_off[kBN / kRPL];
#pragma unroll
  for (int u = 0; u < kBM / kRPL; ++u)
    a_off[u] = (uint32_t)min(m0 + trow + kRPL * u, M - 1) * (uint32_t)kbytes + tcol;
#pragma unroll
  for (int u = 0; u < kBN / kRPL; ++u)
    w_off[u] = (uint32_t)min(n0 + trow + kRPL * u, N - 1) * (uint32_t)kbytes + tcol;

  // Scale rows: buffer row min(tid + 256 v, kRows - 1); within a wave all
  // rows belong to one operand.
  auto sbr = [&](int v) { return min(tid + kThreads * v, L::kRows - 1); };
  auto sop = [&](int br) { return br < kBM ? 0 : (RES && br < 2 * kBM ? 1 : 2); };
  int s_op[L::kScaleLoads];
  uint32_t s_off[L::kScaleLoads];
#pragma unroll
  for (int v = 0; v < L::kScaleLoads; ++v) {
    const int br = sbr(v);
    s_op[v] = __builtin_amdgcn_readfirstlane(sop(br));
    const int o = sop(br);
    s_off[v] = o == 2 ? (uint32_t)min(n0 + br - L::kWRow, N - 1) * (uint32_t)kblocks
                      : (uint32_t)min(m0 + br - (o == 1 ? kBM : 0), M - 1) * (uint32_t)kblocks;
  }

  // pf: the stage in flight (registers); grp: 16 scale bytes (kGroup
  // stages) of this thread's scale rows.
  u32x4 pf[L::kLoads];
  u32x4 grp[L::kScaleLoads];
  // Offset of a skipped load: at or past the end of any operand below
  // 2 GiB of codes (for larger operands it may land inside the buffer,
  // which only costs the fetch: the data is never read).
  constexpr uint32_t kSkipOffset = 0x80000000u;
  // Residual row block b of a stage is fetched only where bit b of rmask
  // is set (fallback-indicator path); otherwise its load gets an offset
  // past the end of the buffer, which the buffer range check turns into
  // zeros without a memory access (the block's LDS rows are then never
  // read).
  auto load_stage = [&](int st, int rmask) {
#pragma unroll
    for (int u = 0; u < L::kLoads; ++u) {
      const int o = op_of(u);
      uint32_t off = o == 2 ? w_off[u - L::kWRow / kRPL] : a_off[u % (kBM / kRPL)];
      if constexpr (PHI && RES)
        if (o == 1) off = ((rmask >> (u - kBM / kRPL)) & 1) ? off : kSkipOffset;
      pf[u] = __builtin_amdgcn_raw_buffer_load_b128(o == 0 ? cq : (o == 1 ? cr : cw), off,
                                                    kb_code + st * kRowBytes, 0);
    }
  };
  auto load_group = [&](int gi) {
#pragma unroll
    for (int v = 0; v < L::kScaleLoads; ++v)
      grp[v] = __builtin_amdgcn_raw_buffer_load_b128(s_op[v] == 0 ? sq : (s_op[v] == 1 ? sr : sw),
                                                     s_off[v], kb_scale + 16 * gi, 0);
  };
  // Writes the register stage and word `word` of the scale group to LDS.
  auto store_stage = [&](int buf, auto word_tag) {
    constexpr int W = decltype(word_tag)::value;
    uint8_t *b = smem + buf * L::kStageBytes;
#pragma unroll
    for (int u = 0; u < L::kLoads; ++u)
      *reinterpret_cast<u32x4 *>(b + chunk_off(trow + kRPL * u, tid & 3)) = pf[u];
#pragma unroll
    for (int v = 0; v < L::kScaleLoads; ++v)
      *reinterpret_cast<uint32_t *>(b + L::kDataBytes + 4 * sbr(v)) = grp[v][W];
  };

  const int frow = lane & 31, h = lane >> 5;
  auto wrow = [&](int j) { return L::kWRow + wn * kTN + 32 * j + frow; };
  auto qrow = [&](int i) { return wm * kTM + 32 * i + frow; };
  auto lds = [&](int buf) { return smem + buf * L::kStageBytes; };

  struct WFrag { u32x4 w[kFN]; };
  struct AFrag { u32x4 q, r; };
  auto read_w = [&](int buf, int s, WFrag &f) {
#pragma unroll
    for (int j = 0; j < kFN; ++j)
      f.w[j] = *reinterpret_cast<const u32x4 *>(lds(buf) + chunk_off(wrow(j), 2 * h + s));
  };
  auto read_q = [&](int buf, int s, int i, AFrag &f) {
    f.q = *reinterpret_cast<const u32x4 *>(lds(buf) + chunk_off(qrow(i), 2 * h + s));
  };
  auto read_r = [&](int buf, int s, int i, AFrag &f) {
    if constexpr (RES)
      f.r = *reinterpret_cast<const u32x4 *>(lds(buf) + chunk_off(kBM + qrow(i), 2 * h + s));
  };
  auto read_a = [&](int buf, int s, int i, AFrag &f) {
    read_q(buf, s, i, f);
    read_r(buf, s, i, f);
  };
  auto read_scales = [&](int buf, Scales<C, RES> &sc) {
    const uint8_t *b = lds(buf) + L::kDataBytes + 2 * h;
#pragma unroll
    for (int j = 0; j < kFN; ++j) sc.w[j] = *reinterpret_cast<const uint16_t *>(b + 4 * wrow(j));
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      sc.q[i] = *reinterpret_cast<const uint16_t *>(b + 4 * qrow(i));
      if constexpr (RES) sc.r[i] = *reinterpret_cast<const uint16_t *>(b + 4 * (kBM + qrow(i)));
    }
  };

  v16f acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j) acc[i][j] = v16f{};

  auto mma_row = [&](const WFrag &w, const AFrag &a, const Scales<C, RES> &sc, int i, auto s_tag) {
    constexpr int S = decltype(s_tag)::value;
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
          as_v8i(w.w[j]), as_v8i(a.q), acc[i][j], kFmtFp4, kFmtFp4, S, sc.w[j], S, sc.q[i]);
      if constexpr (RES)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            as_v8i(w.w[j]), as_v8i(a.r), acc[i][j], kFmtFp4, kFmtFp4, S, sc.w[j], S, sc.r[i]);
    }
  };
  // The primary (R false) or the residual (R true) MFMAs of fragment row i,
  // for the fallback-indicator path, which issues them in two groups.
  auto mma_part = [&](const WFrag &w, const AFrag &a, const Scales<C, RES> &sc, int i, auto s_tag,
                      auto r_tag) {
    constexpr int S = decltype(s_tag)::value;
    constexpr bool R = decltype(r_tag)::value;
#pragma unroll
    for (int j = 0; j < kFN; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
          as_v8i(w.w[j]), as_v8i(R ? a.r : a.q), acc[i][j], kFmtFp4, kFmtFp4, S, sc.w[j], S,
          R ? sc.r[i] : sc.q[i]);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using W0 = std::integral_constant<int, 0>;
  using W1 = std::integral_constant<int, 1>;
  using W2 = std::integral_constant<int, 2>;
  using W3 = std::integral_constant<int, 3>;
  using HO = std::integral_constant<bool, true>;
  using NoHO = std::integral_constant<bool, false>;
  using Rl = std::integral_constant<bool, true>;
  using NoRl = std::integral_constant<bool, false>;

  // The fallback-indicator bytes of this workgroup's four wave rows, copied
  // to LDS behind the stage buffers, four per reduction tile (one 32-bit
  // word per tile; the prologue's barrier publishes them).
  const int pcols = (int)((K + kPhiK - 1) / kPhiK);
  uint8_t *phi_lds = smem + L::kBytes;
  if constexpr (PHI) {
    const int64_t prow0 = m0 / kPhiRows, prows = (M + kPhiRows - 1) / kPhiRows;
    for (int i = tid; i < kWaveRows * pcols; i += kThreads) {
      const int64_t pr = prow0 + i % kWaveRows;
      phi_lds[i] = pr < prows ? phi[pr * pcols + i / kWaveRows] : (uint8_t)0;
    }
  }
  const int wm_u = __builtin_amdgcn_readfirstlane(wm);
  // This thread's residual row blocks (u = kBM / kRPL + b) belong to wave
  // rows lw and lw + 2, b = 0, 1: rows 16 wave + 128 b of the residual tile.
  const int lw = __builtin_amdgcn_readfirstlane(wave >> 2);
  auto phi_word = [&](int st) -> uint32_t {
    return __builtin_amdgcn_readfirstlane(
        *reinterpret_cast<const uint32_t *>(phi_lds + kWaveRows * (st / 2)));
  };
  // Bit b: the residual row block b of stage st is needed.
  auto res_mask = [&](int st) -> int {
    const uint32_t w = phi_word(st);
    return (((w >> (8 * lw)) & 0xFFu) ? 1 : 0) | (((w >> (8 * (lw + 2))) & 0xFFu) ? 2 : 0);
  };
  // ---- prologue: stage 0 into buffer 0, stage 1 in registers.
  if constexpr (PHI) __syncthreads();   // the indicator words
  load_group(0);
  load_stage(0, PHI ? res_mask(0) : 3);
  store_stage(0, W0{});
  __builtin_amdgcn_sched_barrier(0);
  load_stage(min(1, nstages - 1), PHI ? res_mask(min(1, nstages - 1)) : 3);
  asm volatile("" ::: "memory");
  __syncthreads();

  auto region_end = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  };
  constexpr int kRowMfma = RES ? 2 * kFN : kFN;
  constexpr int kAR = RES ? 2 : 1;
  constexpr int kSR = kFN + kFM * (RES ? 2 : 1);
  using Prim = std::integral_constant<bool, false>;
  using Resi = std::integral_constant<bool, true>;
  // Stage st: multiply buffer st mod 2; write stage st+1 (in registers) to
  // the other buffer, whose previous contents were last read before the
  // barrier that ended stage st-1; then fetch stage st+2.  With a
  // fallback-indicator map, each k-step issues the primary MFMAs of both
  // rows (the writes and loads spread between them) and then, where the
  // wave's indicator `on` is set, the residual MFMAs; residual row blocks
  // that no wave row of the workgroup needs are not fetched.
  auto stage = [&](int st, auto handover_tag, auto word_tag, auto reload_tag) {
    constexpr bool HANDOVER = decltype(handover_tag)::value;
    constexpr bool RELOAD = decltype(reload_tag)::value;
    const int buf = st & 1, nbuf = buf ^ 1;
    constexpr int kW = HANDOVER ? L::kLoads + L::kScaleLoads : 0;
    constexpr int kV = (HANDOVER ? L::kLoads : 0) + (RELOAD ? L::kScaleLoads : 0);
    int on = 1, lmask = 3;
    if constexpr (PHI) {
      on = (phi_word(st) >> (8 * wm_u)) & 0xFFu;
      if constexpr (HANDOVER) lmask = res_mask(min(st + 2, nstages - 1));
    }
    WFrag w;
    AFrag a0, a1;
    Scales<C, RES> sc;
    read_w(buf, 0, w);
    read_scales(buf, sc);
    read_a(buf, 0, 0, a0);
    read_a(buf, 0, 1, a1);
    if constexpr (HANDOVER) store_stage(nbuf, word_tag);
    if constexpr (PHI) {
      mma_part(w, a0, sc, 0, S0{}, Prim{});
      mma_part(w, a1, sc, 1, S0{}, Prim{});
      reads_first<kFN + kSR + 2 * kAR>();
      spread<2 * kFN, kW, kDsWrite>();
      region_end();
      if (on) {
        mma_part(w, a0, sc, 0, S0{}, Resi{});
        mma_part(w, a1, sc, 1, S0{}, Resi{});
      }
    } else {
      mma_row(w, a0, sc, 0, S0{});
      mma_row(w, a1, sc, 1, S0{});
      reads_first<kFN + kSR + 2 * kAR>();
      spread<2 * kRowMfma, kW, kDsWrite>();
    }
    region_end();

    if constexpr (RELOAD) load_group((st + 2) / kGroup);
    if constexpr (HANDOVER) load_stage(min(st + 2, nstages - 1), lmask);
    WFrag w1;
    AFrag b0, b1;
    read_w(buf, 1, w1);
    read_a(buf, 1, 0, b0);
    read_a(buf, 1, 1, b1);
    if constexpr (PHI) {
      mma_part(w1, b0, sc, 0, S1{}, Prim{});
      mma_part(w1, b1, sc, 1, S1{}, Prim{});
      reads_first<kFN + 2 * kAR>();
      spread<2 * kFN, kV, kVmemRead>();
      region_end();
      if (on) {
        mma_part(w1, b0, sc, 0, S1{}, Resi{});
        mma_part(w1, b1, sc, 1, S1{}, Resi{});
      }
    } else {
      mma_row(w1, b0, sc, 0, S1{});
      mma_row(w1, b1, sc, 1, S1{});
      reads_first<kFN + 2 * kAR>();
      spread<2 * kRowMfma, kV, kVmemRead>();
    }
    region_end();
    __syncthreads();
  };

  // nstages is a multiple of kGroup; stage st writes scale word
  // (st+1) mod kGroup, so unrolling by kGroup keeps it static.  The scale
  // group is refetched after its last word is written.  (The last group's
  // stages are written as conditional: unconditional straight-line copies
  // make the register allocator spill.)
  int st = 0;
  for (; st < nstages - kGroup; st += kGroup) {
    stage(st + 0, HO{}, W1{}, NoRl{});
    stage(st + 1, HO{}, W2{}, NoRl{});
    stage(st + 2, HO{}, W3{}, Rl{});
    stage(st + 3, HO{}, W0{}, NoRl{});
  }
  if (st + 0 < nstages - 1) stage(st + 0, HO{}, W1{}, NoRl{});
  if (st + 1 < nstages - 1) stage(st + 1, HO{}, W2{}, NoRl{});
  if (st + 2 < nstages - 1) stage(st + 2, HO{}, W3{}, NoRl{});
  stage(nstages - 1, NoHO{}, W0{}, NoRl{});

  if constexpr (SWIGLU) {
    swiglu_epilogue<C, HRES>(acc, so, M, m0 + wm * kTM + frow, n0 + wn * kTN, h);
    return;
  }

  // ---- epilogue: per pass (i, jp) a wave owns 32 rows x 64 columns.
  using E = Epi<ZBF16>;
  uint8_t *ep = smem + wave * E::kWaveBytes;
  const bool vec_ok = ZBF16 ? (N % 8) == 0 : (N % 4) == 0;
  constexpr int kPer = 16 / E::kElem;
#pragma unroll
  for (int i = 0; i < kFM; ++i) {
#pragma unroll
    for (int jp = 0; jp < kFN / 2; ++jp) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const v16f &a = acc[i][2 * jp + jj];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint8_t *p = ep + frow * E::kRowStride + (32 * jj + 8 * g + 4 * h) * E::kElem;
          if constexpr (ZBF16) {
            uint2 w;
            w.x = bf16x2_rne(a[4 * g], a[4 * g + 1]);
            w.y = bf16x2_rne(a[4 * g + 2], a[4 * g + 3]);
            *reinterpret_cast<uint2 *>(p) = w;
          } else {
            *reinterpret_cast<float4 *>(p) = make_float4(a[4 * g], a[4 * g + 1], a[4 * g + 2],
                                                         a[4 * g + 3]);
          }
        }
      }
      const int64_t mrow0 = m0 + wm * kTM + 32 * i;
      const int64_t ncol0 = n0 + wn * kTN + 64 * jp;
#pragma unroll
      for (int k = 0; k < 32 * E::kChunksPerRow / 64; ++k) {
        const int idx = 64 * k + lane;
        const int row = idx / E::kChunksPerRow, cc = idx % E::kChunksPerRow;
        const uint4 d = *reinterpret_cast<const uint4 *>(ep + row * E::kRowStride + 16 * cc);
        const int64_t m = mrow0 + row;
        const int64_t n = ncol0 + kPer * cc;
        if (m >= M) continue;
        if (vec_ok && n + kPer <= N) {
          uint8_t *zp = reinterpret_cast<uint8_t *>(z) + (m * N + n) * E::kElem;
          *reinterpret_cast<uint4 *>(zp) = d;
        } else {
          const uint32_t w4[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
          for (int e = 0; e < kPer; ++e) {
            if (n + e < N) {
              if constexpr (ZBF16)
                reinterpret_cast<uint16_t *>(z)[m * N + n + e] =
                    (uint16_t)(w4[e / 2] >> (16 * (e & 1)));
              else
                reinterpret_cast<uint32_t *>(z)[m * N + n + e] = w4[e];
            }
          }
        }
      }
    }
  }
}

#define RFQ_TILE_ARGS                                                                      \
  const uint8_t *__restrict__ qc, const uint8_t *__restrict__ qs,                          \
      const uint8_t *__restrict__ rc, const uint8_t *__restrict__ rs,                      \
      const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws, int64_t M, int64_t N, \
      int64_t K, void *__restrict__ z, SwigluOut so, const uint8_t *__restrict__ phi,      \
      int64_t ksplit

template <bool RES, bool ZBF16, bool SWIGLU = false, bool HRES = false, bool PHI = false>
__global__ __launch_bounds__(Big::kThreads, 2) void rfq_gemm_large_kernel(RFQ_TILE_ARGS) {
  gemm_tile<Big, RES, ZBF16, SWIGLU, HRES, PHI>(qc, qs, rc, rs, wc, ws, M, N, K, z, so, phi,
                                                ksplit);
}

template <bool RES, bool ZBF16, bool SWIGLU = false, bool HRES = false>
__global__ __launch_bounds__(Mid::kThreads, 3) void rfq_gemm_mid_kernel(RFQ_TILE_ARGS) {
  gemm_tile<Mid, RES, ZBF16, SWIGLU, HRES, false>(qc, qs, rc, rs, wc, ws, M, N, K, z, so, phi,
                                                  ksplit);
}

// K split over several workgroups per 128 x 128 tile: fp32 partial products.
template <bool RES>
__global__ __launch_bounds__(Mid::kThreads, 3) void rfq_gemm_split_kernel(RFQ_TILE_ARGS) {
  gemm_tile<Mid, RES, false, false, false, false, true>(qc, qs, rc, rs, wc, ws, M, N, K, z, so,
                                                        phi, ksplit);
}
#undef RFQ_TILE_ARGS

// Z = sum of the S partial products p[s][M N], added in the order s = 0, 1,
// ...; four outputs per work item (V4: M N a multiple of 4), fp32 or bf16.
template <bool ZBF16, bool V4>
__global__ __launch_bounds__(256) void splitk_sum_kernel(const float *__restrict__ p, int S,
                                                         int64_t mn, void *__restrict__ z) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  if constexpr (V4) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < mn / 4; i += stride) {
      float4 a = reinterpret_cast<const float4 *>(p)[i];
      for (int s = 1; s < S; ++s) {
        const float4 b = reinterpret_cast<const float4 *>(p + s * mn)[i];
        a.x += b.x;
        a.y += b.y;
        a.z += b.z;
        a.w += b.w;
      }
      if constexpr (ZBF16)
        reinterpret_cast<uint2 *>(z)[i] = uint2{bf16x2_rne(a.x, a.y), bf16x2_rne(a.z, a.w)};
      else
        reinterpret_cast<float4 *>(z)[i] = a;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < mn; i += stride) {
      float a = p[i];
      for (int s = 1; s < S; ++s) a += p[s * mn + i];
      if constexpr (ZBF16)
        reinterpret_cast<uint16_t *>(z)[i] = (uint16_t)bf16_rne(a);
      else
        reinterpret_cast<float *>(z)[i] = a;
    }
  }
}

template <class C, bool RES, bool ZBF16, bool SWIGLU = false, bool HRES = false, bool PHI = false>
hipError_t launch(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc,
                  const uint8_t *rs, const uint8_t *wc, const uint8_t *ws,
                  int64_t M, int64_t N, int64_t K, void *z, hipStream_t stream,
                  const SwigluOut &so = SwigluOut{}, const uint8_t *phi = nullptr) {
  using L = Layout<C, RES>;
  static_assert((C::kThreads / 64) * Epi<ZBF16>::kWaveBytes <= L::kBytes, "epilogue staging fits");
  void (*kern)(const uint8_t *, const uint8_t *, const uint8_t *, const uint8_t *,
               const uint8_t *, const uint8_t *, int64_t, int64_t, int64_t, void *, SwigluOut,
               const uint8_t *, int64_t);
  if constexpr (std::is_same<C, Big>::value)
    kern = rfq_gemm_large_kernel<RES, ZBF16, SWIGLU, HRES, PHI>;
  else
    kern = rfq_gemm_mid_kernel<RES, ZBF16, SWIGLU, HRES>;
  // LDS: the two stage buffers, then (PHI) the rows of the indicator map.
  constexpr int kMaxBytes = L::kBytes + (PHI ? kPhiMapMaxBytes : 0);
  const int phi_bytes =
      PHI ? (int)(((C::kWaveRows * ((K + kPhiK - 1) / kPhiK)) + 15) / 16 * 16) : 0;
  static std::atomic<bool> attr_done[kMaxDevices];
  const hipError_t e = set_lds_limit(attr_done, reinterpret_cast<const void *>(kern), kMaxBytes);
  if (e != hipSuccess) return e;
  const int64_t ntiles = ((M + C::kBM - 1) / C::kBM) * ((N + C::kBN - 1) / C::kBN);
  kern<<<dim3((unsigned)ntiles), dim3(C::kThreads), L::kBytes + phi_bytes, stream>>>(
      qc, qs, rc, rs, wc, ws, M, N, K, z, so, phi, K);
  return hipGetLastError();
}

// K split into `parts` ranges of ksplit columns (a multiple of 512): the
// partial products go to work[parts][M][N] (fp32), then one pass adds them.
template <bool RES>
hipError_t launch_split(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc,
                        const uint8_t *rs, const uint8_t *wc, const uint8_t *ws, int64_t M,
                        int64_t N, int64_t K, void *z, bool z_bf16, float *work, int parts,
                        int64_t ksplit, hipStream_t stream) {
  using L = Layout<Mid, RES>;
  auto kern = rfq_gemm_split_kernel<RES>;
  static std::atomic<bool> attr_done[kMaxDevices];
  hipError_t e = set_lds_limit(attr_done, reinterpret_cast<const void *>(kern), L::kBytes);
  if (e != hipSuccess) return e;
  const int64_t ntiles = ((M + Mid::kBM - 1) / Mid::kBM) * ((N + Mid::kBN - 1) / Mid::kBN);
  kern<<<dim3((unsigned)(ntiles * parts)), dim3(Mid::kThreads), L::kBytes, stream>>>(
      qc, qs, rc, rs, wc, ws, M, N, K, work, SwigluOut{}, nullptr, ksplit);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_splitk_sum(work, parts, M * N, z, z_bf16, stream);
}

// Parts of K for the split product (1: no split), so that the parts x tiles
// workgroups fill the 256 CUs about once: 256 / tiles parts (at most 8) up to
// 128 tiles of 128 x 128, and for K >= 8192 512 / tiles (at most 4) up to
// 192 tiles; parts x tiles <= 512, so the partials take at most 32 MiB.
// Measured against the unsplit 128-wide tiles (random codes, bf16 Z): 64
// rows x 4096 x 12288 64.7 -> 18.5 us (8 parts); 129 rows 60.3 -> 23.9 (4);
// 256 rows 61.9 -> 28.5 (4); 512 rows 63.2 -> 44.3 (2); 64 rows x 5120 x
// 13824 80.9 -> 24.6 (6); 512 rows 72.5 -> 57.5 (3); 128 rows x 12288 x
// 4096 25.7 -> 22.1 (2).  With K = 4096 and 192 tiles (129 rows x 12288)
// two parts cost more than they save (21.3 -> 25.5 us).
int splitk_default_parts(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((M + Mid::kBM - 1) / Mid::kBM) * ((N + Mid::kBN - 1) / Mid::kBN);
  if (tiles <= 128) return (int)std::min<int64_t>(8, 256 / tiles);
  if (tiles <= 192 && K >= 8192) return (int)std::min<int64_t>(4, 512 / tiles);
  return 1;
}

// 128 x 128 tiles while they number fewer than two per CU of the 256 (up to
// three run on a CU at once).  Measured, same outputs either way: 0.53-0.58
// of the 256 x 256 time where those tiles fill at most a quarter of the CUs
// (129-256 rows x 12288 x 4096: 22-25 us against 40-43 us; 129-768 rows x
// 4096 x 12288: 60-67 us against 108-117 us), 0.8-0.96 at 384-480 tiles,
// 1.06-1.23 at 512-576.
bool use_mid_tiles(int64_t M, int64_t N) {
  const int64_t mid = ((M + Mid::kBM - 1) / Mid::kBM) * ((N + Mid::kBN - 1) / Mid::kBN);
  return mid < 2 * 256;
}

}  // namespace

hipError_t launch_splitk_sum(const float *work, int parts, int64_t mn, void *z, bool z_bf16,
                             hipStream_t stream) {
  const bool v4 = (mn % 4) == 0;
  const int64_t items = v4 ? mn / 4 : mn;
  const unsigned blocks = (unsigned)std::min<int64_t>((items + 255) / 256, 4096);
  if (z_bf16) {
    if (v4) splitk_sum_kernel<true, true><<<blocks, 256, 0, stream>>>(work, parts, mn, z);
    else splitk_sum_kernel<true, false><<<blocks, 256, 0, stream>>>(work, parts, mn, z);
  } else {
    if (v4) splitk_sum_kernel<false, true><<<blocks, 256, 0, stream>>>(work, parts, mn, z);
    else splitk_sum_kernel<false, false><<<blocks, 256, 0, stream>>>(work, parts, mn, z);
  }
  return hipGetLastError();
}

SplitPlan splitk_plan(int64_t M, int64_t N, int64_t K, int parts_wanted) {
  SplitPlan p{1, K, 0};
  const int64_t units = K / (kStageK * kGroup);
  if (!use_mid_tiles(M, N) || units < 2) return p;
  int want = parts_wanted;
  if (want <= 0) want = splitk_default_parts(M, N, K);
  if (want < 2) return p;
  const int64_t per = (units + want - 1) / want;
  p.parts = (int)((units + per - 1) / per);
  if (p.parts < 2) return SplitPlan{1, K, 0};
  p.ksplit = per * kStageK * kGroup;
  p.work_bytes = (int64_t)p.parts * M * N * 4;
  return p;
}

hipError_t launch_gemm_large_split(const uint8_t *q_codes, const uint8_t *q_scales,
                                   const uint8_t *r_codes, const uint8_t *r_scales,
                                   const uint8_t *w_codes, const uint8_t *w_scales, int64_t M,
                                   int64_t N, int64_t K, void *z, bool z_bf16,
                                   const SplitPlan &plan, float *work, hipStream_t stream) {
  if (plan.parts < 2)
    return launch_gemm_large(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K,
                             z, z_bf16, stream);
  if (r_codes)
    return launch_split<true>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K,
                              z, z_bf16, work, plan.parts, plan.ksplit, stream);
  return launch_split<false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z,
                             z_bf16, work, plan.parts, plan.ksplit, stream);
}

bool large_tiles_beat_few_rows(int64_t M, int64_t N) {
  return M > 64 && (N + Mid::kBN - 1) / Mid::kBN >= 96;
}

bool gemm_large_applies(const uint8_t *q_scales, const uint8_t *r_scales,
                        const uint8_t *w_scales, int64_t M, int64_t N, int64_t K) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(q_scales) |
                      reinterpret_cast<uintptr_t>(r_scales) |
                      reinterpret_cast<uintptr_t>(w_scales);
  // Byte offsets inside an operand are 32-bit.
  const int64_t limit = int64_t(1) << 32;
  return (K % (kStageK * kGroup)) == 0 && (a & 15) == 0 && M * (K / 2) < limit &&
         N * (K / 2) < limit;
}

// 256-row tile rows that run 256 x 256 tiles where those do not fill their
// last round of 256 well: a last round of at most 64 tiles would run at a
// quarter of the chip for a whole tile time, so the tile rows of that round
// run 128 x 128 tiles in a second launch instead (1536 rows x 12288 x 4096:
// 101 -> 85 us; 4096 rows x 5120 x 13824: 330 -> 308 us).  Returns the
// number of tile rows of the 256 x 256 launch (all of them where nothing is
// peeled).
static int64_t big_tile_rows(int64_t M, int64_t N) {
  const int64_t ntm = (M + Big::kBM - 1) / Big::kBM, ntn = (N + Big::kBN - 1) / Big::kBN;
  const int64_t tiles = ntm * ntn, tail = tiles % 256;
  if (tail == 0 || tail > 64) return ntm;
  const int64_t rows = (tiles - tail) / ntn;
  return rows > 0 ? rows : ntm;
}

hipError_t launch_gemm_large(const uint8_t *q_codes, const uint8_t *q_scales,
                             const uint8_t *r_codes, const uint8_t *r_scales,
                             const uint8_t *w_codes, const uint8_t *w_scales,
                             int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                             hipStream_t stream) {
  auto go = [&](auto tile, int64_t row0, int64_t rows) {
    using C = decltype(tile);
    // Activation rows [row0, row0 + rows) and the same rows of Z.
    const uint8_t *qc = q_codes + row0 * (K / 2), *qs = q_scales + row0 * (K / 32);
    const uint8_t *rc = r_codes ? r_codes + row0 * (K / 2) : nullptr;
    const uint8_t *rs = r_codes ? r_scales + row0 * (K / 32) : nullptr;
    void *zr = static_cast<uint8_t *>(z) + row0 * N * (z_bf16 ? 2 : 4);
    if (r_codes) {
      if (z_bf16)
        return launch<C, true, true>(qc, qs, rc, rs, w_codes, w_scales, rows, N, K, zr, stream);
      return launch<C, true, false>(qc, qs, rc, rs, w_codes, w_scales, rows, N, K, zr, stream);
    }
    if (z_bf16)
      return launch<C, false, true>(qc, qs, rc, rs, w_codes, w_scales, rows, N, K, zr, stream);
    return launch<C, false, false>(qc, qs, rc, rs, w_codes, w_scales, rows, N, K, zr, stream);
  };
  if (use_mid_tiles(M, N)) return go(Mid{}, 0, M);
  const int64_t big_rows = std::min<int64_t>(big_tile_rows(M, N) * Big::kBM, M);
  const hipError_t e = go(Big{}, 0, big_rows);
  if (e != hipSuccess || big_rows == M) return e;
  // Both tile shapes accumulate every output in the same order, so the
  // peeled rows carry the bits the 256 x 256 tiles would give them.
  return go(Mid{}, big_rows, M - big_rows);
}

hipError_t launch_gemm_large_phi(const uint8_t *q_codes, const uint8_t *q_scales,
                                 const uint8_t *r_codes, const uint8_t *r_scales,
                                 const uint8_t *w_codes, const uint8_t *w_scales,
                                 const uint8_t *phi, int64_t M, int64_t N, int64_t K, void *z,
                                 bool z_bf16, hipStream_t stream) {
  if (z_bf16)
    return launch<Big, true, true, false, false, true>(q_codes, q_scales, r_codes, r_scales,
                                                       w_codes, w_scales, M, N, K, z, stream,
                                                       SwigluOut{}, phi);
  return launch<Big, true, false, false, false, true>(q_codes, q_scales, r_codes, r_scales,
                                                      w_codes, w_scales, M, N, K, z, stream,
                                                      SwigluOut{}, phi);
}

hipError_t launch_gemm_swiglu(const uint8_t *q_codes, const uint8_t *q_scales,
                              const uint8_t *r_codes, const uint8_t *r_scales,
                              const uint8_t *wgu_codes, const uint8_t *wgu_scales,
                              int64_t M, int64_t Nh, int64_t K, uint8_t *hq_codes,
                              uint8_t *hq_scales, uint8_t *hr_codes, uint8_t *hr_scales,
                              uint16_t *h_out, hipStream_t stream) {
  const SwigluOut so{hq_codes, hq_scales, hr_codes, hr_scales, h_out, Nh};
  const int64_t N = 2 * Nh;
  auto go = [&](auto tile) {
    using C = decltype(tile);
    if (r_codes) {
      if (hr_codes)
        return launch<C, true, true, true, true>(q_codes, q_scales, r_codes, r_scales, wgu_codes,
                                                 wgu_scales, M, N, K, nullptr, stream, so);
      return launch<C, true, true, true, false>(q_codes, q_scales, r_codes, r_scales, wgu_codes,
                                                wgu_scales, M, N, K, nullptr, stream, so);
    }
    if (hr_codes)
      return launch<C, false, true, true, true>(q_codes, q_scales, r_codes, r_scales, wgu_codes,
                                                wgu_scales, M, N, K, nullptr, stream, so);
    return launch<C, false, true, true, false>(q_codes, q_scales, r_codes, r_scales, wgu_codes,
                                               wgu_scales, M, N, K, nullptr, stream, so);
  };
  return use_mid_tiles(M, N) ? go(Mid{}) : go(Big{});
}

}  // namespace rfq
