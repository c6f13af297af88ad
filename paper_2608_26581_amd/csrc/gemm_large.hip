// RFQ product, large-tile kernel for K a multiple of 128 (Eq. 11, Algorithm 1
// with phi = 1; phi = 0 without the residual operand).
//
// Output tile 256 x 256 per workgroup of 4 waves (2 x 2, each wave 128 x 128 =
// 4 x 4 fragments of 32 x 32, one wave per SIMD with its accumulators in the
// AGPR file).  Instruction: v_mfma_scale_f32_32x32x64_f8f6f4 with E2M1
// operands: lane l of an operand holds row (l mod 32) and 32 consecutive K
// values (one MX block) and supplies that block's scale byte; the 32 x 32
// fp32 result gives lane l the rows 8a + 4(l/32) + 0..3 (a = 0..3) of column
// (l mod 32).  With weights as the first operand those are four runs of four
// consecutive outputs of one row of Z.  (On gfx950 this instruction sustains
// about 7.6 PFLOP/s of FP4 against about 6.1 for the 16x16x128 form, measured
// with register-only loops.)
//
// One stage is 128 K values = 4 MX blocks = two k-steps: lane half h takes
// blocks 2h (k-step 0) and 2h+1 (k-step 1) - the contraction order inside an
// instruction is free as long as both operands use the same assignment - so
// a fragment is one 16-byte chunk per k-step and one 16-bit scale pair per
// stage (op_sel picks the byte).  Per k-step a wave reads 4 w, 4 q and 4 r
// chunks and issues 32 MFMAs; every weight fragment feeds the primary and the
// residual MFMA, which is the residual contraction sharing the weight tile.
//
// Software pipeline (one wave per SIMD, so the wave hides its own latencies):
// the global loads of stage s+1 are issued at the start of stage s into
// registers; while the MFMAs of k-step 0 run, the chunks of k-step 1 are read
// from LDS; while those of k-step 1 run, the prefetched stage is written to
// the other LDS buffer, the workgroup synchronizes once, and the chunks and
// scales of the next stage's k-step 0 are read.  Plain global loads are used
// (on this access pattern they sustain 17-22 TB/s where global_load_lds tops
// out near 7 TB/s).  Inside LDS the 16-byte chunks of a row are XOR-swizzled
// by row, so the 8 rows served together by one 16-byte read hit distinct banks.
//
// Epilogue: each wave stages its results through LDS (padded rows) and
// writes Z with 16-byte stores covering whole row segments.
//
// Rows past M or N are clamped to the last row for loading (their results
// are never stored), so no load leaves its tensor.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "gemm_common.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

constexpr int kBM = 256, kBN = 256;
constexpr int kThreads = 256;                // 4 waves
constexpr int kTM = 128, kTN = 128;          // wave sub-tile
constexpr int kFM = kTM / 32, kFN = kTN / 32;   // 32x32 fragments
constexpr int kStageK = 128;
constexpr int kRowBytes = kStageK / 2;       // 64 code bytes per row per stage
constexpr int kPF = 2;                       // stages of global loads in flight

template <bool RES>
struct Layout {
  static constexpr int kOps = RES ? 3 : 2;                 // q, (r), w
  static constexpr int kRows = kOps * 256;
  static constexpr int kDataBytes = kRows * kRowBytes;
  static constexpr int kScaleBytes = kRows * 4;
  static constexpr int kStageBytes = kDataBytes + kScaleBytes;
  static constexpr int kBytes = 3 * kStageBytes;
  static constexpr int kWRow = (kOps - 1) * 256;           // first weight row
  static constexpr int kLoads = kRows * 4 / kThreads;      // 16-byte chunks per thread
  static constexpr int kScaleLoads = kRows / kThreads;     // one row of scales each
};

// Scale bytes are fetched 16 per row (kGroup stages) at a time: a 4-byte
// fetch per row and stage would cost a whole L2 request for 4 useful bytes.
constexpr int kGroup = 4;

// Byte offset of 16-byte chunk c of buffer row r.
__device__ __forceinline__ int chunk_off(int r, int c) {
  return r * kRowBytes + 16 * (c ^ ((r >> 1) & 3));
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

// Fragments of one k-step: w, q and (RES) r chunks of the wave's rows (the
// FP4 operand occupies the low four registers of the MFMA source).
template <bool RES>
struct Frags {
  u32x4 w[kFN], q[kFM], r[RES ? kFM : 1];
};
// Scale pairs of one stage (both k-steps).
template <bool RES>
struct Scales {
  int w[kFN], q[kFM], r[RES ? kFM : 1];
};

// Scheduling pattern for one region: NM MFMAs with ND LDS instructions and
// NV global loads spread evenly between them.
template <int NM, int ND, int NV, int I = 0>
__device__ __forceinline__ void interleave() {
  if constexpr (I < NM) {
    constexpr int nd = (ND * (I + 1)) / NM - (ND * I) / NM;
    constexpr int nv = (NV * (I + 1)) / NM - (NV * I) / NM;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);          // one MFMA
    if constexpr (nd > 0) __builtin_amdgcn_sched_group_barrier(0x080, nd, 0);   // LDS
    if constexpr (nv > 0) __builtin_amdgcn_sched_group_barrier(0x020, nv, 0);   // loads
    interleave<NM, ND, NV, I + 1>();
  }
}

template <bool RES, bool ZBF16>
__global__ __launch_bounds__(kThreads) void rfq_gemm_large_kernel(
    const uint8_t *__restrict__ qc, const uint8_t *__restrict__ qs,
    const uint8_t *__restrict__ rc, const uint8_t *__restrict__ rs,
    const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws,
    int64_t M, int64_t N, int64_t K, void *__restrict__ z) {
  using L = Layout<RES>;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];

  int tm, tn;
  tile_coords<4>(blockIdx.x, (int)((M + kBM - 1) / kBM), (int)((N + kBN - 1) / kBN), tm, tn);
  const int64_t m0 = (int64_t)tm * kBM, n0 = (int64_t)tn * kBN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t kbytes = K / 2, kblocks = K / 32;
  const int nstages = (int)(K / kStageK);

  // ---- staged chunks.  Chunk u of this thread is chunk tid + 256 u of the
  // stage tile: buffer row (tid / 4 + 64 u), chunk (tid mod 4); rows
  // [256 o, 256 o + 256) belong to operand o (q, r, w), so u / 4 is the
  // operand.  Loads go through buffer descriptors (base and size in scalar
  // registers, a 32-bit offset per load; the caller guarantees every code and
  // scale tensor is below 4 GiB).  Source rows are clamped to the tensor.
  const int trow = tid / 4, tcol = 16 * (tid & 3);
  auto rsrc = [](const uint8_t *p, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(p), (short)0, (int)bytes,
                                             0x00020000);
  };
  const __amdgpu_buffer_rsrc_t c_rsrc[3] = {
      rsrc(qc, M * kbytes), rsrc(RES ? rc : qc, M * kbytes), rsrc(wc, N * kbytes)};
  const __amdgpu_buffer_rsrc_t s_rsrc[3] = {
      rsrc(qs, M * kblocks), rsrc(RES ? rs : qs, M * kblocks), rsrc(ws, N * kblocks)};
  auto crsrc = [&](int o) { return c_rsrc[o == L::kOps - 1 ? 2 : o]; };
  auto srsrc = [&](int o) { return s_rsrc[o == L::kOps - 1 ? 2 : o]; };
  // Row byte offsets of this thread's chunks (activation rows serve q and r).
  uint32_t a_off[4], w_off[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    a_off[u] = (uint32_t)min(m0 + trow + 64 * u, M - 1) * (uint32_t)kbytes + tcol;
    w_off[u] = (uint32_t)min(n0 + trow + 64 * u, N - 1) * (uint32_t)kbytes + tcol;
  }
  const uint32_t as_off = (uint32_t)min(m0 + tid, M - 1) * (uint32_t)kblocks;
  const uint32_t ws_off = (uint32_t)min(n0 + tid, N - 1) * (uint32_t)kblocks;

  // Register prefetch sets: stage s lives in set s mod kPF until it is
  // written to LDS; kPF stages of loads are in flight behind the one being
  // multiplied.  The scale bytes of kGroup stages (16 per row, this thread's
  // row of each operand) live in `grp`.
  struct Stage {
    u32x4 d[L::kLoads];
  };
  Stage pf[kPF];
  u32x4 grp[L::kScaleLoads];
  auto load_stage = [&](Stage &g, int st) {
#pragma unroll
    for (int u = 0; u < L::kLoads; ++u) {
      const int o = u / 4;
      const uint32_t off = (o == L::kOps - 1 ? w_off : a_off)[u % 4];
      g.d[u] = __builtin_amdgcn_raw_buffer_load_b128(crsrc(o), off, st * kRowBytes, 0);
    }
  };
  auto load_group = [&](int gi) {
#pragma unroll
    for (int v = 0; v < L::kScaleLoads; ++v)
      grp[v] = __builtin_amdgcn_raw_buffer_load_b128(
          srsrc(v), v == L::kOps - 1 ? ws_off : as_off, 16 * gi, 0);
  };
  // Writes a register stage and word `word` of the scale group to LDS.
  auto store_stage = [&](const Stage &g, int buf, auto word_tag) {
    constexpr int W = decltype(word_tag)::value;
    uint8_t *b = smem + buf * L::kStageBytes;
#pragma unroll
    for (int u = 0; u < L::kLoads; ++u)
      *reinterpret_cast<u32x4 *>(b + chunk_off(trow + 64 * u, tid & 3)) = g.d[u];
#pragma unroll
    for (int v = 0; v < L::kScaleLoads; ++v)
      *reinterpret_cast<uint32_t *>(b + L::kDataBytes + 4 * (tid + kThreads * v)) = grp[v][W];
  };

  const int frow = lane & 31, h = lane >> 5;
  // Buffer rows of this wave's fragments.
  auto wrow = [&](int j) { return L::kWRow + wn * kTN + 32 * j + frow; };
  auto qrow = [&](int i) { return wm * kTM + 32 * i + frow; };
  auto lds = [&](int buf) { return smem + buf * L::kStageBytes; };

  // Weight chunks of one k-step, and the q / r chunks of one fragment row.
  struct WFrag { u32x4 w[kFN]; };
  struct AFrag { u32x4 q, r; };
  auto read_w = [&](int buf, int s, WFrag &f) {
#pragma unroll
    for (int j = 0; j < kFN; ++j)
      f.w[j] = *reinterpret_cast<const u32x4 *>(lds(buf) + chunk_off(wrow(j), 2 * h + s));
  };
  auto read_a = [&](int buf, int s, int i, AFrag &f) {
    f.q = *reinterpret_cast<const u32x4 *>(lds(buf) + chunk_off(qrow(i), 2 * h + s));
    if constexpr (RES)
      f.r = *reinterpret_cast<const u32x4 *>(lds(buf) + chunk_off(256 + qrow(i), 2 * h + s));
  };
  auto read_scales = [&](int buf, Scales<RES> &sc) {
    const uint8_t *b = lds(buf) + L::kDataBytes + 2 * h;
#pragma unroll
    for (int j = 0; j < kFN; ++j) sc.w[j] = *reinterpret_cast<const uint16_t *>(b + 4 * wrow(j));
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      sc.q[i] = *reinterpret_cast<const uint16_t *>(b + 4 * qrow(i));
      if constexpr (RES) sc.r[i] = *reinterpret_cast<const uint16_t *>(b + 4 * (256 + qrow(i)));
    }
  };

  v16f acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j) acc[i][j] = v16f{};

  // MFMAs of fragment row i of one k-step.
  auto mma_row = [&](const WFrag &w, const AFrag &a, const Scales<RES> &sc, int i, auto s_tag) {
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
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;

  using W0 = std::integral_constant<int, 0>;
  // ---- prologue: stage 0 into LDS buffer 0, stages 1 .. kPF in flight.
  load_group(0);
  load_stage(pf[0], 0);
  store_stage(pf[0], 0, W0{});
  // Issued stage by stage, in order, so that the wait before each LDS write
  // of the loop can leave the later stages in flight.
#pragma unroll
  for (int p = 1; p <= kPF; ++p) {
    load_stage(pf[p % kPF], min(p, nstages - 1));
    __builtin_amdgcn_sched_barrier(0);
  }
  asm volatile("" ::: "memory");
  __syncthreads();
  WFrag w0, w1;
  AFrag a0, a1;
  Scales<RES> sc;
  read_w(0, 0, w0);
  read_scales(0, sc);
  read_a(0, 0, 0, a0);

  // One stage = 4 fragment rows x 2 k-steps of MFMAs.  LDS buffers rotate
  // over 3 so that the buffer written during stage st (for st+1) was last
  // read before the barrier of stage st-1.  Every other instruction of the
  // stage is spread between the MFMAs so that no burst of memory
  // instructions stalls the single wave of the SIMD:
  //   k0 row 0-1 : LDS writes of stage st+1      | read A(k0, 1), A(k0, 2)
  //   k0 row 2-3 : global loads of st+1+kPF       | read A(k0, 3), W(k1), A(k1, 0)
  //   k1 row 0-1 :                                | read A(k1, 1), A(k1, 2)
  //   barrier (every wave's LDS writes of stage st+1 are done)
  //   k1 row 2-3 :                                | read A(k1, 3), next W(k0),
  //                                                 scales and A(k0, 0)
  // Rolling A fragments: row i+1 is read while row i is multiplied.
  constexpr int kRowMfma = RES ? 8 : 4;
  auto region_end = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  };
  // Stage st writes stage st+1 (scale word (st+1) mod kGroup) to LDS; when
  // that is the last word of its group, the next group is fetched before
  // the stage's data loads, so that waiting for it never waits for them.
  auto stage = [&](int st, Stage &next_set, auto handover_tag, auto word_tag,
                   auto reload_tag) {
    constexpr bool HANDOVER = decltype(handover_tag)::value;
    constexpr bool RELOAD = decltype(reload_tag)::value;
    const int buf = st % 3, nbuf = (st + 1) % 3;
    constexpr int kW = HANDOVER ? L::kLoads + L::kScaleLoads : 0;   // LDS writes
    constexpr int kV = (HANDOVER ? L::kLoads : 0) + (RELOAD ? L::kScaleLoads : 0);   // loads
    constexpr int kAR = RES ? 2 : 1;                                 // reads per A row

    if constexpr (HANDOVER) store_stage(next_set, nbuf, word_tag);
    read_a(buf, 0, 1, a1);
    mma_row(w0, a0, sc, 0, S0{});
    read_a(buf, 0, 2, a0);
    mma_row(w0, a1, sc, 1, S0{});
    interleave<2 * kRowMfma, kW + 2 * kAR, 0>();
    region_end();

    if constexpr (RELOAD) load_group((st + 2) / kGroup);
    if constexpr (HANDOVER) load_stage(next_set, min(st + 1 + kPF, nstages - 1));
    read_a(buf, 0, 3, a1);
    read_w(buf, 1, w1);
    mma_row(w0, a0, sc, 2, S0{});
    read_a(buf, 1, 0, a0);
    mma_row(w0, a1, sc, 3, S0{});
    interleave<2 * kRowMfma, 2 * kAR + kFN, kV>();
    region_end();

    read_a(buf, 1, 1, a1);
    mma_row(w1, a0, sc, 0, S1{});
    read_a(buf, 1, 2, a0);
    mma_row(w1, a1, sc, 1, S1{});
    interleave<2 * kRowMfma, 2 * kAR, 0>();
    region_end();
    __syncthreads();

    read_a(buf, 1, 3, a1);
    Scales<RES> scn = sc;
    if constexpr (HANDOVER) {
      read_w(nbuf, 0, w0);
      read_scales(nbuf, scn);
    }
    mma_row(w1, a0, sc, 2, S1{});
    if constexpr (HANDOVER) read_a(nbuf, 0, 0, a0);
    mma_row(w1, a1, sc, 3, S1{});
    interleave<2 * kRowMfma, HANDOVER ? 2 * kAR + kFN + kFM * (RES ? 2 : 1) + kFN : kAR, 0>();
    region_end();
    sc = scn;
  };
  using HO = std::integral_constant<bool, true>;
  using NoHO = std::integral_constant<bool, false>;
  using Rl = std::integral_constant<bool, true>;
  using NoRl = std::integral_constant<bool, false>;
  using W1 = std::integral_constant<int, 1>;
  using W2 = std::integral_constant<int, 2>;
  using W3 = std::integral_constant<int, 3>;
  static_assert(kGroup == 4 && kPF == 2, "the unrolled loop below assumes these");

  // nstages is a multiple of kGroup.  Stage st writes set (st+1) mod kPF and
  // scale word (st+1) mod kGroup, so unrolling by kGroup keeps both static.
  int st = 0;
  for (; st < nstages - kGroup; st += kGroup) {
    stage(st + 0, pf[1], HO{}, W1{}, NoRl{});
    stage(st + 1, pf[0], HO{}, W2{}, NoRl{});
    stage(st + 2, pf[1], HO{}, W3{}, Rl{});
    stage(st + 3, pf[0], HO{}, W0{}, NoRl{});
  }
  // The last group.  (Its stages are written as conditional: unconditional
  // straight-line copies make the register allocator spill.)
  if (st + 0 < nstages - 1) stage(st + 0, pf[1], HO{}, W1{}, NoRl{});
  if (st + 1 < nstages - 1) stage(st + 1, pf[0], HO{}, W2{}, NoRl{});
  if (st + 2 < nstages - 1) stage(st + 2, pf[1], HO{}, W3{}, NoRl{});
  stage(nstages - 1, pf[0], NoHO{}, W0{}, NoRl{});
  __syncthreads();

  // ---- epilogue: per pass (i, jp) a wave owns 32 rows x 64 columns.
  using E = Epi<ZBF16>;
  uint8_t *ep = smem + wave * E::kWaveBytes;
  const bool vec_ok = ZBF16 ? (N % 8) == 0 : (N % 4) == 0;
  constexpr int kPer = 16 / E::kElem;          // elements per 16-byte piece
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
            w.x = bf16_rne(a[4 * g]) | (bf16_rne(a[4 * g + 1]) << 16);
            w.y = bf16_rne(a[4 * g + 2]) | (bf16_rne(a[4 * g + 3]) << 16);
            *reinterpret_cast<uint2 *>(p) = w;
          } else {
            *reinterpret_cast<float4 *>(p) = make_float4(a[4 * g], a[4 * g + 1], a[4 * g + 2],
                                                         a[4 * g + 3]);
          }
        }
      }
      // Read back whole 16-byte pieces of rows and store them.
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

template <bool RES, bool ZBF16>
hipError_t launch(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc,
                  const uint8_t *rs, const uint8_t *wc, const uint8_t *ws,
                  int64_t M, int64_t N, int64_t K, void *z, hipStream_t stream) {
  using L = Layout<RES>;
  static_assert(4 * Epi<ZBF16>::kWaveBytes <= L::kBytes, "epilogue staging fits");
  auto kern = rfq_gemm_large_kernel<RES, ZBF16>;
  static std::atomic<bool> attr_done{false};
  if (!attr_done.load(std::memory_order_acquire)) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
    if (e != hipSuccess) return e;
    attr_done.store(true, std::memory_order_release);
  }
  const int64_t ntiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
  kern<<<dim3((unsigned)ntiles), dim3(kThreads), L::kBytes, stream>>>(qc, qs, rc, rs, wc, ws,
                                                                       M, N, K, z);
  return hipGetLastError();
}

}  // namespace

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

hipError_t launch_gemm_large(const uint8_t *q_codes, const uint8_t *q_scales,
                             const uint8_t *r_codes, const uint8_t *r_scales,
                             const uint8_t *w_codes, const uint8_t *w_scales,
                             int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                             hipStream_t stream) {
  if (r_codes) {
    if (z_bf16)
      return launch<true, true>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
    return launch<true, false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
  }
  if (z_bf16)
    return launch<false, true>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
  return launch<false, false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
}

}  // namespace rfq
