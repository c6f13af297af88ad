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

template <bool RES>
struct Layout {
  static constexpr int kOps = RES ? 3 : 2;                 // q, (r), w
  static constexpr int kRows = kOps * 256;
  static constexpr int kDataBytes = kRows * kRowBytes;
  static constexpr int kScaleBytes = kRows * 4;
  static constexpr int kStageBytes = kDataBytes + kScaleBytes;
  static constexpr int kBytes = 2 * kStageBytes;
  static constexpr int kWRow = (kOps - 1) * 256;           // first weight row
  static constexpr int kLoads = kRows * 4 / kThreads;      // 16-byte chunks per thread
  static constexpr int kScaleLoads = kRows / kThreads;     // one row of scales each
};

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

  // ---- fixed per-thread sources of the staged chunks, as 32-bit byte
  // offsets from the operand base (the caller guarantees every code and scale
  // tensor is smaller than 4 GiB).  Chunk u of this thread is chunk
  // tid + 256 u of the stage tile: buffer row (tid / 4 + 64 u), chunk
  // (tid mod 4); rows [256 o, 256 o + 256) belong to operand o (q, r, w), so
  // u / 4 is the operand.
  uint32_t src[L::kLoads];
#pragma unroll
  for (int u = 0; u < L::kLoads; ++u) {
    const bool is_w = u / 4 == L::kOps - 1;
    const int rl = tid / 4 + 64 * (u % 4);
    const int64_t grow = min((is_w ? n0 : m0) + rl, (is_w ? N : M) - 1);
    src[u] = (uint32_t)(grow * kbytes + 16 * (tid & 3));
  }
  // Scale row tid + 256 v of the stage tile (operand v), 4 bytes per stage.
  uint32_t ssrc[L::kScaleLoads];
#pragma unroll
  for (int v = 0; v < L::kScaleLoads; ++v) {
    const bool is_w = v == L::kOps - 1;
    const int64_t grow = min((is_w ? n0 : m0) + tid, (is_w ? N : M) - 1);
    ssrc[v] = (uint32_t)(grow * kblocks);
  }
  auto codes_of = [&](int o) { return o == L::kOps - 1 ? wc : (o == 0 ? qc : rc); };
  auto scales_of = [&](int o) { return o == L::kOps - 1 ? ws : (o == 0 ? qs : rs); };

  u32x4 pref[L::kLoads];
  uint32_t spref[L::kScaleLoads];
  auto load_stage = [&](int st) {
#pragma unroll
    for (int u = 0; u < L::kLoads; ++u)
      pref[u] = *reinterpret_cast<const u32x4 *>(codes_of(u / 4) + src[u] +
                                                 (uint32_t)st * kRowBytes);
#pragma unroll
    for (int v = 0; v < L::kScaleLoads; ++v)
      spref[v] = *reinterpret_cast<const uint32_t *>(scales_of(v) + ssrc[v] + 4u * st);
  };
  auto store_stage = [&](int buf) {
    uint8_t *b = smem + buf * L::kStageBytes;
#pragma unroll
    for (int u = 0; u < L::kLoads; ++u)
      *reinterpret_cast<u32x4 *>(b + chunk_off(tid / 4 + 64 * u, tid & 3)) = pref[u];
#pragma unroll
    for (int v = 0; v < L::kScaleLoads; ++v)
      *reinterpret_cast<uint32_t *>(b + L::kDataBytes + 4 * (tid + kThreads * v)) = spref[v];
  };

  const int frow = lane & 31, h = lane >> 5;
  // Buffer rows of this wave's fragments.
  auto wrow = [&](int j) { return L::kWRow + wn * kTN + 32 * j + frow; };
  auto qrow = [&](int i) { return wm * kTM + 32 * i + frow; };

  auto read_frags = [&](int buf, int s, Frags<RES> &f) {
    const uint8_t *b = smem + buf * L::kStageBytes;
#pragma unroll
    for (int j = 0; j < kFN; ++j)
      f.w[j] = *reinterpret_cast<const u32x4 *>(b + chunk_off(wrow(j), 2 * h + s));
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      f.q[i] = *reinterpret_cast<const u32x4 *>(b + chunk_off(qrow(i), 2 * h + s));
      if constexpr (RES)
        f.r[i] = *reinterpret_cast<const u32x4 *>(b + chunk_off(256 + qrow(i), 2 * h + s));
    }
  };
  auto read_scales = [&](int buf, Scales<RES> &sc) {
    const uint8_t *b = smem + buf * L::kStageBytes + L::kDataBytes + 2 * h;
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

  // MFMAs of one k-step, rows i in [i0, i1).
  auto mma = [&](const Frags<RES> &f, const Scales<RES> &sc, auto s_tag, int i0, int i1) {
    constexpr int S = decltype(s_tag)::value;
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      if (i < i0 || i >= i1) continue;
#pragma unroll
      for (int j = 0; j < kFN; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            as_v8i(f.w[j]), as_v8i(f.q[i]), acc[i][j], kFmtFp4, kFmtFp4, S, sc.w[j], S, sc.q[i]);
        if constexpr (RES)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              as_v8i(f.w[j]), as_v8i(f.r[i]), acc[i][j], kFmtFp4, kFmtFp4, S, sc.w[j], S, sc.r[i]);
      }
    }
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;

  Frags<RES> f0, f1;
  Scales<RES> sc;

  load_stage(0);
  store_stage(0);
  __syncthreads();
  read_frags(0, 0, f0);
  read_scales(0, sc);

  // The memory clobbers pin the global loads, LDS writes and LDS reads to
  // their places in the pipeline (the compiler would otherwise sink the
  // global loads next to their LDS writes); the MFMAs are free to move
  // within the regions delimited by the scheduling barriers.
  for (int st = 0; st + 1 < nstages; ++st) {
    const int buf = st & 1;
    load_stage(st + 1);
    asm volatile("" ::: "memory");
    // k-step 0 on f0 while k-step 1 is read into f1.
    read_frags(buf, 1, f1);
    mma(f0, sc, S0{}, 0, kFM);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
    // k-step 1 on f1; it overlaps the hand-over of the next stage: LDS write
    // of the prefetched stage, one barrier, reads of the next k-step 0.
    mma(f1, sc, S1{}, 0, kFM / 2);
    store_stage(buf ^ 1);
    __syncthreads();
    read_frags(buf ^ 1, 0, f0);
    Scales<RES> scn;
    read_scales(buf ^ 1, scn);
    mma(f1, sc, S1{}, kFM / 2, kFM);
    sc = scn;
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  }
  {
    const int buf = (nstages - 1) & 1;
    read_frags(buf, 1, f1);
    mma(f0, sc, S0{}, 0, kFM);
    mma(f1, sc, S1{}, 0, kFM);
  }
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
  return (K % kStageK) == 0 && (a & 3) == 0 && M * (K / 2) < limit && N * (K / 2) < limit;
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
