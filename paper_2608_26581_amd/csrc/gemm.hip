// RFQ product on the gfx950 block-scaled FP4 matrix cores (Eq. 11,
// Algorithm 1 with the fallback indicator phi = 1, or phi = 0 without the
// residual operand):
//
//   Z[m][n] = sum_k q[m][k] w[n][k] * Sq[m][k/32] Sw[n][k/32]
//           + sum_k r[m][k] w[n][k] * Sr[m][k/32] Sw[n][k/32]
//
// Instruction: v_mfma_scale_f32_16x16x128_f8f6f4 with both operands in E2M1
// (format code 4).  Lane l of a 16x16x128 operand holds row (l mod 16) and 32
// consecutive K values (one MX block, 16 bytes, element 2j in the low nibble of
// byte j) and supplies that block's E8M0 scale in a byte of its scale VGPR
// selected by op_sel.  The weight fragment is the A operand and the
// activation fragment the B operand, so the 16x16 fp32 result in lane l holds
// Z[m = l mod 16][n = 4*(l/16) .. +3]: four consecutive outputs of one row.
//
// Because the contraction order inside one instruction is irrelevant, the K
// values given to the four lane groups may be permuted as long as weights and
// activations use the same permutation: in a stage of 256 K values (8 blocks),
// lane group g takes blocks 2g (first instruction) and 2g+1 (second), so its
// two scale bytes are adjacent and one 16-bit LDS read serves both.
//
// Data flow per workgroup (output tile BM x BN, 4 waves as 2 x 2, each wave a
// (BM/2) x (BN/2) sub-tile): each stage copies 128 code bytes per row of the
// q, r and w tiles plus 8 scale bytes per row from global memory into LDS
// (double buffered; the next stage's global loads are in flight while the
// current stage is multiplied).  The residual contraction reuses every
// weight fragment read from LDS: per weight fragment two MFMAs are issued,
// one against q and one against r.  16-byte chunks are XOR-swizzled by row
// inside LDS so that the 16 rows read by one fragment hit distinct banks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "gemm_common.h"
#include "rfq_internal.h"

namespace rfq {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kStageK = 256;                 // K values per stage
constexpr int kRowBytes = kStageK / 2;       // code bytes per row per stage
constexpr int kRowChunks = kRowBytes / 16;   // 16-byte chunks per row
constexpr int kRowScales = kStageK / 32;     // scale bytes per row per stage
constexpr int kFmtFp4 = 4;                   // E2M1 operand format code

template <int BM, int BN, bool RES>
struct Smem {
  static constexpr int kRows = (RES ? 2 : 1) * BM + BN;   // q, r, w rows
  static constexpr int kDataBytes = kRows * kRowBytes;
  static constexpr int kScaleBytes = kRows * kRowScales;
  static constexpr int kStageBytes = kDataBytes + kScaleBytes;
  static constexpr int kBytes = 2 * kStageBytes;
};

// LDS serves a 16-byte access of 16 lanes at a time across 256 bytes of
// banks (two 128-byte rows): the XOR with (row >> 1) & 7 gives the 16
// consecutive rows of a fragment read 16 distinct slots (row & 7 let rows r
// and r + 8 collide); the stores (2 rows x 8 chunks per 16 lanes) stay
// conflict-free.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * kRowBytes + 16 * (chunk ^ ((row >> 1) & 7));
}

// Fallback-indicator map: one byte per tile of 64 activation rows (a wave's
// rows) by 256 reduction columns (a stage).
constexpr int kPhiRows = 64;
constexpr int kPhiMapMaxBytes = 2 * ((1 << 20) / kStageK);   // two rows, K up to 2^20

template <int BM, int BN, bool RES, bool ZBF16, bool PHI = false>
__global__ __launch_bounds__(256) void rfq_gemm_kernel(
    const uint8_t *__restrict__ qc, const uint8_t *__restrict__ qs,
    const uint8_t *__restrict__ rc, const uint8_t *__restrict__ rs,
    const uint8_t *__restrict__ wc, const uint8_t *__restrict__ ws,
    int64_t M, int64_t N, int64_t K, void *__restrict__ z,
    const uint8_t *__restrict__ phi) {
  constexpr int kThreads = 256;
  constexpr int TM = BM / 2, TN = BN / 2;     // wave sub-tile
  constexpr int FM = TM / 16, FN = TN / 16;   // 16x16 fragments per wave
  using S = Smem<BM, BN, RES>;
  constexpr int kRows = S::kRows;
  constexpr int kChunksPerStage = kRows * kRowChunks;
  static_assert(kChunksPerStage % kThreads == 0, "chunk split");
  constexpr int kLoads = kChunksPerStage / kThreads;
  constexpr int kScaleLoads = (kRows + kThreads - 1) / kThreads;

  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

  // ---- tile order: consecutive tiles on one XCD, grouped by 8 tile rows.
  const int ntm = (int)((M + BM - 1) / BM), ntn = (int)((N + BN - 1) / BN);
  const int ntiles = ntm * ntn;
  int t = blockIdx.x;
  if ((ntiles & 7) == 0) t = (t & 7) * (ntiles >> 3) + (t >> 3);
  constexpr int GM = 8;
  const int group = t / (GM * ntn);
  const int first_m = group * GM;
  const int gsize = min(ntm - first_m, GM);
  const int in_group = t - group * GM * ntn;
  const int tm = first_m + in_group % gsize;
  const int tn = in_group / gsize;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t kbytes = K / 2, kblocks = K / 32;
  const int nstages = (int)((K + kStageK - 1) / kStageK);
  const bool fast_scales =
      (kblocks % kRowScales) == 0 &&
      ((reinterpret_cast<uintptr_t>(qs) | reinterpret_cast<uintptr_t>(rs) |
        reinterpret_cast<uintptr_t>(ws)) & 7) == 0;

  // Row r of the stage tile: [0, BM) q, [BM, 2BM) r (RES), then BN rows of w.
  constexpr int kWRow0 = (RES ? 2 : 1) * BM;
  auto src_codes = [&](int r) { return r >= kWRow0 ? wc : (RES && r >= BM ? rc : qc); };
  auto src_scales = [&](int r) { return r >= kWRow0 ? ws : (RES && r >= BM ? rs : qs); };
  auto src_row = [&](int r) -> int64_t {
    return r >= kWRow0 ? n0 + (r - kWRow0) : m0 + (RES && r >= BM ? r - BM : r);
  };
  auto src_limit = [&](int r) -> int64_t { return r >= kWRow0 ? N : M; };

  uint4 pref[kLoads];
  uint2 spref[kScaleLoads];

  auto load_stage = [&](int st) {
    const int64_t kb0 = (int64_t)st * kRowBytes;   // byte offset in a row
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int c = tid + i * kThreads;
      const int r = c / kRowChunks, ch = c % kRowChunks;
      const int64_t grow = src_row(r);
      const int64_t kb = kb0 + 16 * ch;
      if (grow < src_limit(r) && kb < kbytes)
        pref[i] = *reinterpret_cast<const uint4 *>(src_codes(r) + grow * kbytes + kb);
      else
        pref[i] = make_uint4(0, 0, 0, 0);
    }
    const int64_t sb0 = (int64_t)st * kRowScales;
#pragma unroll
    for (int i = 0; i < kScaleLoads; ++i) {
      const int r = tid + i * kThreads;
      uint2 v = make_uint2(0, 0);
      if (r < kRows) {
        const int64_t grow = src_row(r);
        if (grow < src_limit(r)) {
          const uint8_t *p = src_scales(r) + grow * kblocks + sb0;
          if (fast_scales) {
            v = *reinterpret_cast<const uint2 *>(p);
          } else {
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              if (sb0 + b < kblocks) lo |= (uint32_t)p[b] << (8 * b);
              if (sb0 + 4 + b < kblocks) hi |= (uint32_t)p[4 + b] << (8 * b);
            }
            v = make_uint2(lo, hi);
          }
        }
      }
      spref[i] = v;
    }
  };

  auto store_stage = [&](int buf) {
    uint8_t *base = smem + buf * S::kStageBytes;
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int c = tid + i * kThreads;
      const int r = c / kRowChunks, ch = c % kRowChunks;
      *reinterpret_cast<uint4 *>(base + swz(r, ch)) = pref[i];
    }
#pragma unroll
    for (int i = 0; i < kScaleLoads; ++i) {
      const int r = tid + i * kThreads;
      if (r < kRows)
        *reinterpret_cast<uint2 *>(base + S::kDataBytes + r * kRowScales) = spref[i];
    }
  };

  v4f acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  const int frow = lane & 15, g = lane >> 4;

  static_assert(!PHI || BM == 2 * kPhiRows, "a wave's rows are one indicator row");
  // The indicator rows of this workgroup's two wave rows, behind the stage
  // buffers in LDS (published by the barrier after the first stage store).
  const int pcols = nstages;
  uint8_t *phi_lds = smem + S::kBytes;
  if constexpr (PHI) {
    const int64_t prow0 = m0 / kPhiRows, prows = (M + kPhiRows - 1) / kPhiRows;
    for (int i = tid; i < 2 * pcols; i += kThreads) {
      const int64_t pr = prow0 + i / pcols;
      phi_lds[i] = pr < prows ? phi[pr * pcols + i % pcols] : (uint8_t)0;
    }
  }
  const int wm_u = __builtin_amdgcn_readfirstlane(wm);

  // One instruction step: blocks 2g+SUB of the stage for every lane group;
  // `res_on` (wave-uniform) switches the residual MFMAs of the stage.
  auto mma_step = [&](const uint8_t *base, auto sub_tag, bool res_on) {
    constexpr int SUB = decltype(sub_tag)::value;
    const uint8_t *sc = base + S::kDataBytes;
    v8i wf[FN];
    int wsc[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int r = (RES ? 2 : 1) * BM + wn * TN + 16 * j + frow;
      const uint4 d = *reinterpret_cast<const uint4 *>(base + swz(r, 2 * g + SUB));
      wf[j] = v8i{(int)d.x, (int)d.y, (int)d.z, (int)d.w, 0, 0, 0, 0};
      wsc[j] = *reinterpret_cast<const uint16_t *>(sc + r * kRowScales + 2 * g);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int r = wm * TM + 16 * i + frow;
      const uint4 d = *reinterpret_cast<const uint4 *>(base + swz(r, 2 * g + SUB));
      const v8i af = v8i{(int)d.x, (int)d.y, (int)d.z, (int)d.w, 0, 0, 0, 0};
      const int asc = *reinterpret_cast<const uint16_t *>(sc + r * kRowScales + 2 * g);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
            wf[j], af, acc[i][j], kFmtFp4, kFmtFp4, SUB, wsc[j], SUB, asc);
      if (RES && res_on) {
        const int rr = BM + r;
        const uint4 e = *reinterpret_cast<const uint4 *>(base + swz(rr, 2 * g + SUB));
        const v8i rf = v8i{(int)e.x, (int)e.y, (int)e.z, (int)e.w, 0, 0, 0, 0};
        const int rsc = *reinterpret_cast<const uint16_t *>(sc + rr * kRowScales + 2 * g);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
              wf[j], rf, acc[i][j], kFmtFp4, kFmtFp4, SUB, wsc[j], SUB, rsc);
      }
    }
  };

  load_stage(0);
  store_stage(0);
  __syncthreads();
  for (int st = 0; st < nstages; ++st) {
    const bool more = st + 1 < nstages;
    if (more) load_stage(st + 1);
    const uint8_t *base = smem + (st & 1) * S::kStageBytes;
    const bool res_on =
        !PHI || __builtin_amdgcn_readfirstlane((int)phi_lds[wm_u * pcols + st]) != 0;
    mma_step(base, std::integral_constant<int, 0>{}, res_on);
    mma_step(base, std::integral_constant<int, 1>{}, res_on);
    if (more) store_stage((st + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds Z[m][n .. n+3] for every fragment pair.
  const bool vec_ok = (N & 3) == 0;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int64_t m = m0 + wm * TM + 16 * i + frow;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t n = n0 + wn * TN + 16 * j + 4 * g;
      const v4f a = acc[i][j];
      if constexpr (ZBF16) {
        uint16_t *zp = reinterpret_cast<uint16_t *>(z) + m * N + n;
        if (vec_ok && n + 3 < N) {
          uint2 w;
          w.x = bf16x2_rne(a[0], a[1]);
          w.y = bf16x2_rne(a[2], a[3]);
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
  }
}

template <int BM, int BN, bool RES, bool ZBF16, bool PHI = false>
hipError_t launch_tile(const uint8_t *qc, const uint8_t *qs, const uint8_t *rc,
                       const uint8_t *rs, const uint8_t *wc, const uint8_t *ws,
                       int64_t M, int64_t N, int64_t K, void *z,
                       hipStream_t stream, const uint8_t *phi = nullptr) {
  using S = Smem<BM, BN, RES>;
  auto kern = rfq_gemm_kernel<BM, BN, RES, ZBF16, PHI>;
  constexpr int kMaxBytes = S::kBytes + (PHI ? kPhiMapMaxBytes : 0);
  const int phi_bytes = PHI ? (int)((2 * ((K + kStageK - 1) / kStageK) + 15) / 16 * 16) : 0;
  // The dynamic-LDS limit is an attribute of the kernel function, set once
  // per device; setting it twice from racing threads is harmless.
  static std::atomic<bool> attr_done[kMaxDevices];
  const hipError_t e = set_lds_limit(attr_done, reinterpret_cast<const void *>(kern), kMaxBytes);
  if (e != hipSuccess) return e;
  const int64_t ntiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  kern<<<dim3((unsigned)ntiles), dim3(256), S::kBytes + phi_bytes, stream>>>(
      qc, qs, rc, rs, wc, ws, M, N, K, z, phi);
  return hipGetLastError();
}

}  // namespace

// The few-row kernel takes the product (shape conditions only; alignment and
// size conditions of the kernels are checked where they are dispatched).
static bool few_rows_chosen(int64_t M, int64_t N, int64_t K) {
  return M <= kSkinnyMaxRows && (K % 512) == 0 && !large_tiles_beat_few_rows(M, N);
}

// With a workspace the split product replaces the few-row kernel where it
// splits, from 33 rows; from 24 where K >= 12288, and from 17 where the
// few-row grid is uneven (between one and two workgroups per CU) and K >=
// 8192 (20 rows x 9216 x 4096: 13.6 us few-row against 14.9 split; x 4608 x
// 8192 19.6 against 14.6).  Measured,
// bf16 Z, few-row against split: 64 rows x 4096 x 12288 32.5 against 18.1
// us, 32 rows 19.3 against 16.5, 24 rows 16.8 against 16.0, 16 rows 13.0
// against 15.8; 24 rows x 5120 x 13824 31.4 against 21.0, 16 rows (the
// few-row kernel split over K) 19.3 against 20.5; 32 rows x 4096 x 8192 13.7
// against 13.6, 24 rows 11.9 against 13.2.  Not where the few-row kernel runs
// 64 weight rows per workgroup below N = 16384 (48 rows x 12288 x 4096: 15.4
// us few-row against 18.4 split, 64 rows 17.1 against 19.5).
static bool few_rows_beat_split(int64_t M, int64_t N, int64_t K) {
  if (skinny_four_fragments(M, N) && N < 16384) return true;
  const int64_t min_rows = (skinny_grid_uneven(M, N) && K >= 8192) ? 17 : (K >= 12288 ? 24 : 33);
  return M < min_rows;
}

int64_t gemm_split_bytes(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || (K % 512) != 0) return 0;
  if (few_rows_chosen(M, N, K) && few_rows_beat_split(M, N, K)) {
    const int parts = skinny_split_parts(M, N, K);
    return parts > 1 ? int64_t(parts) * M * N * 4 : 0;
  }
  const SplitPlan p = splitk_plan(M, N, K);
  return p.parts > 1 ? p.work_bytes : 0;
}

hipError_t launch_gemm(const uint8_t *q_codes, const uint8_t *q_scales,
                       const uint8_t *r_codes, const uint8_t *r_scales,
                       const uint8_t *w_codes, const uint8_t *w_scales,
                       int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                       hipStream_t stream, float *work, int64_t work_bytes) {
  const bool large = gemm_large_applies(q_scales, r_scales, w_scales, M, N, K);
  SplitPlan plan{1, K, 0};
  if (large && work) {
    plan = splitk_plan(M, N, K);
    if (plan.work_bytes > work_bytes) plan = SplitPlan{1, K, 0};
  }
  const bool split = plan.parts > 1 && !(few_rows_chosen(M, N, K) && few_rows_beat_split(M, N, K));
  if (gemm_skinny_applies(q_scales, r_scales, w_scales, M, N, K) && !split &&
      !(large && large_tiles_beat_few_rows(M, N))) {
    const int parts = work ? skinny_split_parts(M, N, K) : 1;
    if (parts > 1 && int64_t(parts) * M * N * 4 <= work_bytes)
      return launch_gemm_skinny_split(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M,
                                      N, K, z, z_bf16, parts, work, stream);
    return launch_gemm_skinny(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K,
                              z, z_bf16, stream);
  }
  if (large) {
    if (plan.parts > 1)
      return launch_gemm_large_split(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M,
                                     N, K, z, z_bf16, plan, work, stream);
    return launch_gemm_large(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K,
                             z, z_bf16, stream);
  }
  constexpr int BM = 128, BN = 128;
  if (r_codes) {
    if (z_bf16)
      return launch_tile<BM, BN, true, true>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
    return launch_tile<BM, BN, true, false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
  }
  if (z_bf16)
    return launch_tile<BM, BN, false, true>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
  return launch_tile<BM, BN, false, false>(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, M, N, K, z, stream);
}

hipError_t launch_gemm_phi(const uint8_t *q_codes, const uint8_t *q_scales,
                           const uint8_t *r_codes, const uint8_t *r_scales,
                           const uint8_t *w_codes, const uint8_t *w_scales, const uint8_t *phi,
                           int64_t M, int64_t N, int64_t K, void *z, bool z_bf16,
                           hipStream_t stream) {
  if (gemm_large_applies(q_scales, r_scales, w_scales, M, N, K))
    return launch_gemm_large_phi(q_codes, q_scales, r_codes, r_scales, w_codes, w_scales, phi, M,
                                 N, K, z, z_bf16, stream);
  constexpr int BM = 128, BN = 128;
  if (z_bf16)
    return launch_tile<BM, BN, true, true, true>(q_codes, q_scales, r_codes, r_scales, w_codes,
                                                 w_scales, M, N, K, z, stream, phi);
  return launch_tile<BM, BN, true, false, true>(q_codes, q_scales, r_codes, r_scales, w_codes,
                                                w_scales, M, N, K, z, stream, phi);
}

}  // namespace rfq
