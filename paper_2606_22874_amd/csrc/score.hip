// Selector block scoring kernel (paper Section 2.1); the per-wavefront core
// is in score_core.h.  Each wave handles kUnroll consecutive blocks.
#include "score_core.h"

namespace spot {
namespace {

constexpr int kUnroll = 8;          // blocks per wavefront
constexpr int kWavesPerWG = 4;
constexpr int kBlocksPerWG = kUnroll * kWavesPerWG;

// grid: x = row (n_seq * rows_per_seq), y = chunk of kBlocksPerWG blocks;
// wave w scores kUnroll consecutive blocks.
template <int KFMT, int LPH>
__global__ __launch_bounds__(256) void score_kernel(const uint16_t* __restrict__ q_sel,
                                                    const float* __restrict__ w,
                                                    const uint8_t* __restrict__ k_sel,
                                                    const uint8_t* __restrict__ k_scale,
                                                    int rows_per_seq, int nblk,
                                                    const int32_t* __restrict__ n_valid,
                                                    float* __restrict__ scores) {
  const int row = blockIdx.x;
  const int j0 = blockIdx.y * kBlocksPerWG + (threadIdx.x >> 6) * kUnroll;
  int nv = n_valid ? n_valid[row] : nblk;
  nv = nv < 0 ? 0 : (nv > nblk ? nblk : nv);
  if (j0 >= nblk) return;
  score_blocks<KFMT, LPH, kUnroll>(q_sel, w, k_sel, k_scale, row, row / rows_per_seq, nblk, nv,
                                   j0, nblk, scores, nullptr, threadIdx.x & 63);
}

template <int KFMT>
hipError_t launch_fmt(int lph, dim3 grid, hipStream_t s, const uint16_t* q, const float* w,
                      const uint8_t* k, const uint8_t* ks, int rows_per_seq, int nblk,
                      const int32_t* nv, float* out) {
  if (lph == 8)
    hipLaunchKernelGGL((score_kernel<KFMT, 8>), grid, dim3(256), 0, s, q, w, k, ks, rows_per_seq,
                       nblk, nv, out);
  else
    hipLaunchKernelGGL((score_kernel<KFMT, 16>), grid, dim3(256), 0, s, q, w, k, ks,
                       rows_per_seq, nblk, nv, out);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_selector_score(const void* q_sel, const float* w, const void* k_sel,
                                 const void* k_scale, int kfmt, int n_seq, int rows_per_seq,
                                 int nblk, int h_s, int d_s, const int32_t* n_valid,
                                 float* scores, hipStream_t s) {
  (void)h_s;
  const int rows = n_seq * rows_per_seq;
  dim3 grid(rows, (nblk + kBlocksPerWG - 1) / kBlocksPerWG);
  const int lph = d_s / 8;
  auto q = static_cast<const uint16_t*>(q_sel);
  auto k = static_cast<const uint8_t*>(k_sel);
  auto ks = static_cast<const uint8_t*>(k_scale);
  switch (kfmt) {
    case SPOT_KFMT_BF16:
      return launch_fmt<SPOT_KFMT_BF16>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk, n_valid,
                                        scores);
    case SPOT_KFMT_INT4_G32:
      return launch_fmt<SPOT_KFMT_INT4_G32>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                            n_valid, scores);
    default:
      return launch_fmt<SPOT_KFMT_MXFP4_G32>(lph, grid, s, q, w, k, ks, rows_per_seq, nblk,
                                             n_valid, scores);
  }
}

}  // namespace spot
