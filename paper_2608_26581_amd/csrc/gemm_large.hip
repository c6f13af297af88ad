// RFQ product, large-tile kernel for K a multiple of 128 (Eq. 11, Algorithm 1
// with phi = 1; phi = 0 without the residual operand).
//
// Output tile 256 x 256 per workgroup of 8 waves (4 along M x 2 along N, each
// wave 64 x 128 = 4 x 8 fragments of 16 x 16).  One stage is 128 K values =
// one v_mfma_scale_f32_16x16x128_f8f6f4 depth: lane group g (lanes 16g ..
// 16g+15) takes MX block g of the stage, so each lane reads one 16-byte chunk
// and one scale byte per fragment.  Per stage a wave issues 8 fragment reads
// of w, 4 of q, 4 of r and 64 MFMAs; every weight fragment feeds two MFMAs
// (primary and residual), which is the residual contraction sharing the
// weight tile.
//
// Operand tiles move from global memory straight into LDS with
// global_load_lds_dwordx4 (no VGPR staging): one wave instruction fills 1 KB
// of LDS, lane s writing bytes [16 s, 16 s + 16).  Choosing which global chunk
// each lane fetches lays the tile out with its 16-byte chunks XOR-swizzled by
// row, so the 16 rows one fragment read touches fall in distinct banks.  Three
// stage buffers (156 KB of the 160 KB LDS) let a single barrier per stage
// separate the loads of stage s+2 from the reads of stage s.
//
// Rows past M or N are clamped to the last row for loading (their results
// are never stored), so no load leaves its tensor.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "gemm_common.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

constexpr int kBM = 256, kBN = 256;
constexpr int kThreads = 512;                // 8 waves
constexpr int kTM = 64, kTN = 128;           // wave sub-tile
constexpr int kFM = kTM / 16, kFN = kTN / 16;
constexpr int kStageK = 128;
constexpr int kRowBytes = kStageK / 2;       // 64 code bytes per row per stage
constexpr int kNumBuf = 3;

template <bool RES>
struct Layout {
  static constexpr int kOps = RES ? 3 : 2;                 // q, (r), w
  static constexpr int kDataBytes = kOps * 256 * kRowBytes;
  static constexpr int kScaleBytes = 4 * 256 * 4;          // q, r, w, spare
  static constexpr int kStageBytes = kDataBytes + kScaleBytes;
  static constexpr int kBytes = kNumBuf * kStageBytes;
  static constexpr int kWRow = (kOps - 1) * 256;           // first weight row
  // Loads per thread per stage: data (2 per operand) + scales.
  static constexpr int kScaleInstr = RES ? 2 : 1;
  static constexpr int kLoads = 2 * kOps + kScaleInstr;
};

// Byte offset of 16-byte chunk c of buffer row r.
__device__ __forceinline__ int chunk_off(int r, int c) {
  return r * kRowBytes + 16 * (c ^ ((r >> 1) & 3));
}

// Global -> LDS copies.  Written as inline assembly so that the compiler
// neither reorders them across the explicit waits below nor guards every LDS
// read with a wait for all outstanding copies (it cannot tell which buffer a
// copy targets); m0 carries the wave-uniform LDS destination, lane s writes
// bytes [size*s, size*s + size) from there.  Completion is tracked by hand
// with s_waitcnt vmcnt, and the only vector-memory loads in the main loop are
// these copies.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(lds) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void *g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off"
               :: "v"(g), "s"(lds) : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)((__attribute__((address_space(3))) const uint8_t *)p);
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

  // ---- per-lane source rows of this wave's DMA instructions (fixed over K)
  // Data: operand o, sub-block t in {0,1} covers tile rows 32*wave + 16*t ..
  // + 15; lane s fills slot s: row 32*wave + 16*t + s/4, slot s%4.
  const uint8_t *dsrc[L::kOps][2];
  int dlds[L::kOps][2];
#pragma unroll
  for (int o = 0; o < L::kOps; ++o) {
    const uint8_t *codes = (o == L::kOps - 1) ? wc : (o == 0 ? qc : rc);
    const int64_t row0 = (o == L::kOps - 1) ? n0 : m0;
    const int64_t limit = (o == L::kOps - 1) ? N : M;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int rl = 32 * wave + 16 * t + (lane >> 2);          // row in tile
      const int rb = o * 256 + rl;                              // row in buffer
      const int c = (lane & 3) ^ ((rb >> 1) & 3);               // chunk it holds
      const int64_t grow = min(row0 + rl, limit - 1);
      dsrc[o][t] = codes + grow * kbytes + 16 * c;
      dlds[o][t] = (o * 256 + 32 * wave + 16 * t) * kRowBytes;  // wave-uniform
    }
  }
  // Scales: instruction J covers 64 rows of operand J/4 (J/4 == 3: spare
  // region, refilled with weight scales); lane s loads one row's 4 bytes.
  const uint8_t *ssrc[L::kScaleInstr];
  int slds[L::kScaleInstr];
#pragma unroll
  for (int i = 0; i < L::kScaleInstr; ++i) {
    const int J = L::kScaleInstr * wave + i;
    const int op = J >> 2;
    const bool is_w = RES ? (op >= 2) : (op == 1);
    const uint8_t *scales = is_w ? ws : (op == 0 ? qs : rs);
    const int64_t row0 = is_w ? n0 : m0;
    const int64_t limit = is_w ? N : M;
    const int rl = 64 * (J & 3) + lane;
    const int64_t grow = min(row0 + rl, limit - 1);
    ssrc[i] = scales + grow * kblocks;
    slds[i] = L::kDataBytes + 256 * 4 * op + 64 * 4 * (J & 3);
  }

  const uint32_t smem_base = lds_addr(smem);
  auto issue_stage = [&](int st) {
    const uint32_t buf = smem_base + (st % kNumBuf) * L::kStageBytes;
#pragma unroll
    for (int o = 0; o < L::kOps; ++o)
#pragma unroll
      for (int t = 0; t < 2; ++t)
        dma16(dsrc[o][t] + (int64_t)st * kRowBytes,
              __builtin_amdgcn_readfirstlane(buf + dlds[o][t]));
#pragma unroll
    for (int i = 0; i < L::kScaleInstr; ++i)
      dma4(ssrc[i] + 4 * (int64_t)st, __builtin_amdgcn_readfirstlane(buf + slds[i]));
  };

  v4f acc[kFM][kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i)
#pragma unroll
    for (int j = 0; j < kFN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  const int frow = lane & 15, g = lane >> 4;

  issue_stage(0);
  if (nstages > 1) issue_stage(1);

  for (int st = 0; st < nstages; ++st) {
    // This thread's loads of stage st are done once at most one stage's
    // worth of loads is outstanding; the barrier then covers every wave's.
    if (st + 1 < nstages) {
      if constexpr (L::kLoads == 8)
        asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
      else
        asm volatile("s_waitcnt vmcnt(5)" ::: "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (st + 2 < nstages) issue_stage(st + 2);

    const uint8_t *buf = smem + (st % kNumBuf) * L::kStageBytes;
    const uint8_t *sc = buf + L::kDataBytes;
    v8i wf[kFN];
    int wsc[kFN];
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      const int r = L::kWRow + wn * kTN + 16 * j + frow;
      const uint4 d = *reinterpret_cast<const uint4 *>(buf + chunk_off(r, g));
      wf[j] = v8i{(int)d.x, (int)d.y, (int)d.z, (int)d.w, 0, 0, 0, 0};
      wsc[j] = sc[(RES ? 2 : 1) * 1024 + (wn * kTN + 16 * j + frow) * 4 + g];
    }
#pragma unroll
    for (int i = 0; i < kFM; ++i) {
      const int r = wm * kTM + 16 * i + frow;
      const uint4 d = *reinterpret_cast<const uint4 *>(buf + chunk_off(r, g));
      const v8i af = v8i{(int)d.x, (int)d.y, (int)d.z, (int)d.w, 0, 0, 0, 0};
      const int asc = sc[r * 4 + g];
#pragma unroll
      for (int j = 0; j < kFN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
            wf[j], af, acc[i][j], kFmtFp4, kFmtFp4, 0, wsc[j], 0, asc);
      if constexpr (RES) {
        const int rr = 256 + r;
        const uint4 e = *reinterpret_cast<const uint4 *>(buf + chunk_off(rr, g));
        const v8i rf = v8i{(int)e.x, (int)e.y, (int)e.z, (int)e.w, 0, 0, 0, 0};
        const int rsc = sc[1024 + r * 4 + g];
#pragma unroll
        for (int j = 0; j < kFN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
              wf[j], rf, acc[i][j], kFmtFp4, kFmtFp4, 0, wsc[j], 0, rsc);
      }
    }
  }

  const bool vec_ok = (N & 3) == 0;
#pragma unroll
  for (int i = 0; i < kFM; ++i) {
    const int64_t m = m0 + wm * kTM + 16 * i + frow;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < kFN; ++j)
      store4<ZBF16>(z, m, n0 + wn * kTN + 16 * j + 4 * g, N, vec_ok, acc[i][j]);
  }
}

template <bool RES, bool ZBF16>
hipError_t launch(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc,
                  const uint8_t *rs, const uint8_t *wc, const uint8_t *ws,
                  int64_t M, int64_t N, int64_t K, void *z, hipStream_t stream) {
  using L = Layout<RES>;
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
                        const uint8_t *w_scales, int64_t K) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(q_scales) |
                      reinterpret_cast<uintptr_t>(r_scales) |
                      reinterpret_cast<uintptr_t>(w_scales);
  return (K % kStageK) == 0 && (a & 3) == 0;
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
