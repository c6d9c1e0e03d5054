// Selector block scoring kernels (paper Section 2.1).
//  * score_kernel: one query row against a run of key blocks per wavefront
//    (the per-wavefront core is in score_core.h) -- the decode case, a GEMV
//    per sequence, and the 4-bit selector formats.
//  * score_tile_kernel: many query rows per sequence (prefill: one row per
//    query block) with a BF16 selector cache -- per head a GEMM
//    S_h = Q_h K_h^T on the matrix cores, then sum_h w_h ReLU(S_h) per
//    (query block, key block) tile (the query-block x key-block matmul).
#include "score_core.h"

namespace spot {
namespace {

constexpr int kUnroll = 8;          // blocks per wavefront
constexpr int kWavesPerWG = 4;
constexpr int kBlocksPerWG = kUnroll * kWavesPerWG;

// grid: x = row (n_seq * rows_per_seq), y = chunk of kBlocksPerWG blocks;
// wave w scores kUnroll consecutive blocks.
// QFMT: the queries' format (BF16, or MXFP4 / MXFP8 codes with q_scale).
template <int KFMT, int LPH, int QFMT = SPOT_KFMT_BF16>
__global__ __launch_bounds__(256) void score_kernel(const uint8_t* __restrict__ q_sel,
                                                    const float* __restrict__ w,
                                                    const uint8_t* __restrict__ k_sel,
                                                    const uint8_t* __restrict__ k_scale,
                                                    int rows_per_seq, int nblk,
                                                    const int32_t* __restrict__ n_valid,
                                                    float* __restrict__ scores,
                                                    const uint8_t* __restrict__ q_scale) {
  const int row = blockIdx.x;
  const int j0 = blockIdx.y * kBlocksPerWG + (threadIdx.x >> 6) * kUnroll;
  int nv = n_valid ? n_valid[row] : nblk;
  nv = nv < 0 ? 0 : (nv > nblk ? nblk : nv);
  if (j0 >= nblk) return;
  score_blocks<KFMT, LPH, kUnroll, QFMT>(q_sel, w, k_sel, k_scale, row, row / rows_per_seq, nblk,
                                         nv, j0, nblk, scores, nullptr, threadIdx.x & 63,
                                         q_scale);
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// One 16 x 16 (query row x key block) tile per wavefront, a 2 x 2 group of
// tiles per workgroup.  For head h, v_mfma_f32_16x16x32_bf16 with
//   A = Q_h (16 rows x 32 dims): lane l holds row l%16, dims 8(l/16) ..+7,
//   B = K_h^T (32 dims x 16 keys): lane l holds key l%16, dims 8(l/16) ..+7,
// both 16 contiguous bytes of the row-major caches, read straight from
// global memory; D gives lane l rows 4(l/16)+i of key column l%16.  The head
// sum w_h ReLU(S_h) is accumulated in head order.  Keys at or past a row's
// n_valid score -inf; a tile whose keys all lie past every row's n_valid
// only writes -inf.
template <int DS>
__global__ __launch_bounds__(256) void score_tile_kernel(
    const uint16_t* __restrict__ q_sel, const float* __restrict__ w,
    const uint16_t* __restrict__ k_sel, int rows, int rows_per_seq, int nblk,
    const int32_t* __restrict__ n_valid, float* __restrict__ scores) {
  constexpr int HS = 512 / DS, KS = DS / 32;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.x * 32 + (wave >> 1) * 16;    // first row of the tile
  const int j0 = blockIdx.y * 32 + (wave & 1) * 16;     // first key block of the tile
  const int r16 = lane & 15, G = lane >> 4;
  // This lane's output rows 4G + i and key column r16.
  int nv[4];
  int nv_max = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = r0 + 4 * G + i;
    int v = r < rows ? (n_valid ? n_valid[r] : nblk) : 0;
    v = v < 0 ? 0 : (v > nblk ? nblk : v);
    nv[i] = v;
    nv_max = max(nv_max, v);
  }
  nv_max = (int)wave_max_u((uint32_t)nv_max);
  const int key = j0 + r16;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  if (j0 < nv_max) {
    const int ra = r0 + r16;                            // A row of this lane
    const bool a_ok = ra < rows, b_ok = key < nblk;
    // The 16 rows of a tile share one sequence (the launcher requires
    // rows_per_seq % 16 == 0), whose key cache is the B operand for all.
    const int seq = min(r0, rows - 1) / rows_per_seq;
    const uint16_t* qa = q_sel + (size_t)(a_ok ? ra : 0) * 512 + 8 * G;
    const uint16_t* kb = k_sel + ((size_t)seq * nblk + (b_ok ? key : 0)) * 512 + 8 * G;
    const float* wr = w + (size_t)(r0 + 4 * G) * HS;
    u32x4 af[HS][KS], bfr[HS][KS];
#pragma unroll
    for (int h = 0; h < HS; ++h)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 z = {0u, 0u, 0u, 0u};
        af[h][ks] = a_ok ? *reinterpret_cast<const u32x4*>(qa + h * DS + ks * 32) : z;
        bfr[h][ks] = b_ok ? *reinterpret_cast<const u32x4*>(kb + h * DS + ks * 32) : z;
      }
#pragma unroll
    for (int h = 0; h < HS; ++h) {
      f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, af[h][ks]),
                                                    __builtin_bit_cast(bf16x8_t, bfr[h][ks]), s,
                                                    0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float wi = r0 + 4 * G + i < rows ? wr[i * HS + h] : 0.f;
        acc[i] = fmaf(wi, fmaxf(s[i], 0.f), acc[i]);
      }
    }
  }
  if (key < nblk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = r0 + 4 * G + i;
      if (r < rows) scores[(size_t)r * nblk + key] = key < nv[i] ? acc[i] : -INFINITY;
    }
  }
}

template <int KFMT, int QFMT = SPOT_KFMT_BF16>
hipError_t launch_fmt(int lph, dim3 grid, hipStream_t s, const uint8_t* q, const float* w,
                      const uint8_t* k, const uint8_t* ks, int rows_per_seq, int nblk,
                      const int32_t* nv, float* out, const uint8_t* qs = nullptr) {
  if (lph == 8)
    hipLaunchKernelGGL((score_kernel<KFMT, 8, QFMT>), grid, dim3(256), 0, s, q, w, k, ks,
                       rows_per_seq, nblk, nv, out, qs);
  else
    hipLaunchKernelGGL((score_kernel<KFMT, 16, QFMT>), grid, dim3(256), 0, s, q, w, k, ks,
                       rows_per_seq, nblk, nv, out, qs);
  return hipGetLastError();
}

// Row kernel for any key format with queries in format QFMT.
template <int QFMT>
hipError_t launch_row_q(int kfmt, int lph, dim3 grid, hipStream_t s, const uint8_t* q,
                        const uint8_t* qs, const float* w, const uint8_t* k, const uint8_t* ks,
                        int rows_per_seq, int nblk, const int32_t* nv, float* out) {
  switch (kfmt) {
    case SPOT_KFMT_BF16:
      return launch_fmt<SPOT_KFMT_BF16, QFMT>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk, nv,
                                              out, qs);
    case SPOT_KFMT_INT4_G32:
      return launch_fmt<SPOT_KFMT_INT4_G32, QFMT>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                                  nv, out, qs);
    case SPOT_KFMT_INT8_G32:
      return launch_fmt<SPOT_KFMT_INT8_G32, QFMT>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                                  nv, out, qs);
    case SPOT_KFMT_MXFP8_G32:
      return launch_fmt<SPOT_KFMT_MXFP8_G32, QFMT>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                                   nv, out, qs);
    default:
      return launch_fmt<SPOT_KFMT_MXFP4_G32, QFMT>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                                   nv, out, qs);
  }
}

typedef int32_t i32x8_t __attribute__((ext_vector_type(8)));

// Query-block x key-block tiles with queries and keys both in one MX format
// (MXFP4 or MXFP8, one E8M0 scale per 32 elements) and d_s = 128: per head one
// v_mfma_scale_f32_16x16x128_f8f6f4, the matrix cores applying both operands'
// block scales.  Tiling as score_tile_kernel: one 16 x 16 tile per wave, 2 x 2
// per workgroup.  A = Q_h: lane l holds query row l%16, dims 32(l/16) .. +31
// of head h -- exactly one scale group, whose E8M0 byte the lane passes;
// B = K_h^T likewise for key block l%16 (8-bit codes: see the operand
// layout below).  D gives lane l rows 4(l/16)+i of key column l%16.
template <int FMT>
__global__ __launch_bounds__(256) void score_tile_mx_kernel(
    const uint8_t* __restrict__ q, const uint8_t* __restrict__ qs, const float* __restrict__ w,
    const uint8_t* __restrict__ k, const uint8_t* __restrict__ ks, int rows, int rows_per_seq,
    int nblk, const int32_t* __restrict__ n_valid, float* __restrict__ scores) {
  constexpr int HS = 4;                                        // 4 heads x 128 dims
  constexpr bool FP4 = FMT == SPOT_KFMT_MXFP4_G32;
  constexpr int RB = FP4 ? 256 : 512;                          // code bytes per row
  constexpr int GB = FP4 ? 16 : 32;                            // code bytes per 32-group
  constexpr int kFmtCode = FP4 ? 4 : 0;                        // E2M1 : E4M3
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = blockIdx.x * 32 + (wave >> 1) * 16;
  const int j0 = blockIdx.y * 32 + (wave & 1) * 16;
  const int r16 = lane & 15, G = lane >> 4;
  int nv[4];
  int nv_max = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = r0 + 4 * G + i;
    int v = r < rows ? (n_valid ? n_valid[r] : nblk) : 0;
    v = v < 0 ? 0 : (v > nblk ? nblk : v);
    nv[i] = v;
    nv_max = max(nv_max, v);
  }
  nv_max = (int)wave_max_u((uint32_t)nv_max);
  const int key = j0 + r16;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  if (j0 < nv_max) {
    // Rows past the end and keys past nblk read row / key 0 (in bounds);
    // their results are never stored.
    const int ra = min(r0 + r16, rows - 1);
    const int seq = min(r0, rows - 1) / rows_per_seq;
    const size_t kr = (size_t)seq * nblk + (key < nblk ? key : 0);
    // Operand bytes of lane group G within a head: E2M1, 16 bytes = dims
    // 32G .. 32G+31; E4M3, 32 bytes in two halves, dims 16G .. 16G+15 and
    // 64+16G .. 64+16G+15 (the 8-bit operand layout).  Either way the lane's
    // scale byte is that of the 32-dim group G.
    const uint8_t* qa = q + (size_t)ra * RB + G * 16;
    const uint8_t* kb = k + kr * RB + G * 16;
    const float* wr = w + (size_t)(r0 + 4 * G) * HS;
    i32x8_t A[HS], B[HS];
    int sa[HS], sb[HS];
#pragma unroll
    for (int h = 0; h < HS; ++h) {
      const u32x4 a0 = *reinterpret_cast<const u32x4*>(qa + h * 4 * GB);
      const u32x4 b0 = *reinterpret_cast<const u32x4*>(kb + h * 4 * GB);
      u32x4 a1 = {0u, 0u, 0u, 0u}, b1 = {0u, 0u, 0u, 0u};
      if constexpr (!FP4) {
        a1 = *reinterpret_cast<const u32x4*>(qa + h * 4 * GB + 64);
        b1 = *reinterpret_cast<const u32x4*>(kb + h * 4 * GB + 64);
      }
      A[h] = i32x8_t{(int)a0[0], (int)a0[1], (int)a0[2], (int)a0[3],
                     (int)a1[0], (int)a1[1], (int)a1[2], (int)a1[3]};
      B[h] = i32x8_t{(int)b0[0], (int)b0[1], (int)b0[2], (int)b0[3],
                     (int)b1[0], (int)b1[1], (int)b1[2], (int)b1[3]};
      sa[h] = qs[(size_t)ra * 16 + h * 4 + G];
      sb[h] = ks[kr * 16 + h * 4 + G];
    }
#pragma unroll
    for (int h = 0; h < HS; ++h) {
      const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
      const f32x4_t sc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
          A[h], B[h], z, kFmtCode, kFmtCode, 0, sa[h], 0, sb[h]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float wi = r0 + 4 * G + i < rows ? wr[i * HS + h] : 0.f;
        acc[i] = fmaf(wi, fmaxf(sc[i], 0.f), acc[i]);
      }
    }
  }
  if (key < nblk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = r0 + 4 * G + i;
      if (r < rows) scores[(size_t)r * nblk + key] = key < nv[i] ? acc[i] : -INFINITY;
    }
  }
}

}  // namespace

hipError_t launch_selector_score(const void* q_sel, const float* w, const void* k_sel,
                                 const void* k_scale, int kfmt, int n_seq, int rows_per_seq,
                                 int nblk, int h_s, int d_s, const int32_t* n_valid,
                                 float* scores, hipStream_t s) {
  (void)h_s;
  const int rows = n_seq * rows_per_seq;
  if (kfmt == SPOT_KFMT_BF16 && rows_per_seq > 1 && rows_per_seq % 16 == 0 &&
      (d_s == 64 || d_s == 128)) {
    const dim3 tgrid((rows + 31) / 32, (nblk + 31) / 32);
    auto q = static_cast<const uint16_t*>(q_sel);
    auto k = static_cast<const uint16_t*>(k_sel);
    if (d_s == 64)
      hipLaunchKernelGGL((score_tile_kernel<64>), tgrid, dim3(256), 0, s, q, w, k, rows,
                         rows_per_seq, nblk, n_valid, scores);
    else
      hipLaunchKernelGGL((score_tile_kernel<128>), tgrid, dim3(256), 0, s, q, w, k, rows,
                         rows_per_seq, nblk, n_valid, scores);
    return hipGetLastError();
  }
  dim3 grid(rows, (nblk + kBlocksPerWG - 1) / kBlocksPerWG);
  const int lph = d_s / 8;
  auto q = static_cast<const uint8_t*>(q_sel);
  auto k = static_cast<const uint8_t*>(k_sel);
  auto ks = static_cast<const uint8_t*>(k_scale);
  switch (kfmt) {
    case SPOT_KFMT_BF16:
      return launch_fmt<SPOT_KFMT_BF16>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk, n_valid,
                                        scores);
    case SPOT_KFMT_INT4_G32:
      return launch_fmt<SPOT_KFMT_INT4_G32>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                            n_valid, scores);
    case SPOT_KFMT_INT8_G32:
      return launch_fmt<SPOT_KFMT_INT8_G32>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                            n_valid, scores);
    case SPOT_KFMT_MXFP8_G32:
      return launch_fmt<SPOT_KFMT_MXFP8_G32>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                             n_valid, scores);
    default:
      return launch_fmt<SPOT_KFMT_MXFP4_G32>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                             n_valid, scores);
  }
}

hipError_t launch_selector_score_q(const void* q_sel, const void* q_scale, int qfmt,
                                   const float* w, const void* k_sel, const void* k_scale,
                                   int kfmt, int n_seq, int rows_per_seq, int nblk, int d_s,
                                   const int32_t* n_valid, float* scores, hipStream_t s) {
  const int rows = n_seq * rows_per_seq;
  auto q = static_cast<const uint8_t*>(q_sel);
  auto qs = static_cast<const uint8_t*>(q_scale);
  auto k = static_cast<const uint8_t*>(k_sel);
  auto ks = static_cast<const uint8_t*>(k_scale);
  if (qfmt == kfmt && (qfmt == SPOT_KFMT_MXFP4_G32 || qfmt == SPOT_KFMT_MXFP8_G32) &&
      d_s == 128 && rows_per_seq > 1 && rows_per_seq % 16 == 0) {
    const dim3 tgrid((rows + 31) / 32, (nblk + 31) / 32);
    if (qfmt == SPOT_KFMT_MXFP4_G32)
      hipLaunchKernelGGL((score_tile_mx_kernel<SPOT_KFMT_MXFP4_G32>), tgrid, dim3(256), 0, s, q,
                         qs, w, k, ks, rows, rows_per_seq, nblk, n_valid, scores);
    else
      hipLaunchKernelGGL((score_tile_mx_kernel<SPOT_KFMT_MXFP8_G32>), tgrid, dim3(256), 0, s, q,
                         qs, w, k, ks, rows, rows_per_seq, nblk, n_valid, scores);
    return hipGetLastError();
  }
  const dim3 grid(rows, (nblk + kBlocksPerWG - 1) / kBlocksPerWG);
  const int lph = d_s / 8;
  switch (qfmt) {
    case SPOT_KFMT_MXFP4_G32:
      return launch_row_q<SPOT_KFMT_MXFP4_G32>(kfmt, lph, grid, s, q, qs, w, k, ks, rows_per_seq,
                                               nblk, n_valid, scores);
    case SPOT_KFMT_MXFP8_G32:
      return launch_row_q<SPOT_KFMT_MXFP8_G32>(kfmt, lph, grid, s, q, qs, w, k, ks, rows_per_seq,
                                               nblk, n_valid, scores);
    case SPOT_KFMT_INT4_G32:
      return launch_row_q<SPOT_KFMT_INT4_G32>(kfmt, lph, grid, s, q, qs, w, k, ks, rows_per_seq,
                                              nblk, n_valid, scores);
    default:
      return launch_row_q<SPOT_KFMT_INT8_G32>(kfmt, lph, grid, s, q, qs, w, k, ks, rows_per_seq,
                                              nblk, n_valid, scores);
  }
}

}  // namespace spot
