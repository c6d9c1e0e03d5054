// Block-sparse (and dense) GQA split-KV decode attention kernel; the
// per-workgroup body is in decode_core.h.
#include "decode_core.h"

namespace spot {
namespace {

using namespace dec;

// Grid: n_pairs * n_slot workgroups; workgroup i serves pair i / n_slot with
// slot i % n_slot.  SB: tokens per selected block (64, or 16 for the paper's
// selector block; sparse only).
template <int G, bool DENSE, int SB = kBlk>
__global__ __launch_bounds__(64 * kDecWaves, 2) void decode_split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ seq_len,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int k_max, int h_q,
    int h_kv, int l_cap, float scale_log2, int n_slot, float* __restrict__ ws_o,
    float* __restrict__ ws_ml, unsigned* __restrict__ counters, uint16_t* __restrict__ out,
    float* __restrict__ lse) {
  __shared__ DecodeSmem<G> sm;
  decode_body<G, DENSE, ListFromIdx, SB>(sm, ListFromIdx{idx, count, k_max},
                                         blockIdx.x / n_slot, blockIdx.x % n_slot, q, k, v,
                                         seq_len, h_q, h_kv, l_cap, scale_log2, n_slot, ws_o,
                                         ws_ml, counters, out, lse);
}

}  // namespace

// Workgroups per (sequence, KV head) pair: aim for ~2048 waves over the grid
// (8 per CU, so the whole grid is resident at once; 4 waves per workgroup
// whatever the group size), at least one, and at
// least two list entries per workgroup (with blocks of 16 tokens: two
// virtual blocks of four entries).  Never more than with per_virtual = 1, so
// a workspace sized for 64-token blocks fits.
#ifndef SPOT_DECODE_WAVE_TARGET
#define SPOT_DECODE_WAVE_TARGET 2048
#endif
int decode_num_splits(int batch, int h_kv, int max_blocks, int group, int per_virtual) {
  const int pairs = batch * h_kv;
  (void)group;
  int n = (SPOT_DECODE_WAVE_TARGET / kDecWaves + pairs - 1) / pairs;
  const int by_len = ((max_blocks + per_virtual - 1) / per_virtual + 1) / 2;
  if (n > by_len) n = by_len;
  const int min_for_ids = (max_blocks + kMaxIds - 1) / kMaxIds;  // entries per WG <= kMaxIds
  if (n < min_for_ids) n = min_for_ids;
  return n < 1 ? 1 : n;
}

// Workspace: partial o [B, h_q, n_slot, d], partial (m, l) [B, h_q, n_slot],
// then one completion counter per (sequence, KV head) pair.
size_t decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks) {
  const int G = h_q / h_kv;
  const size_t ns = (size_t)decode_num_splits(batch, h_kv, max_blocks, G, 1);
  return (size_t)batch * h_q * ns * ((size_t)d + 2) * sizeof(float) +
         (size_t)batch * h_kv * sizeof(unsigned);
}

hipError_t launch_decode(bool dense, const void* q, const void* k, const void* v,
                         const int32_t* seq_len, const int32_t* idx, const int32_t* count,
                         int k_max, int batch, int h_q, int h_kv, int l_cap, int blk,
                         float sm_scale, void* out, float* lse, void* ws, unsigned* counters,
                         hipStream_t s) {
  const int G = h_q / h_kv;
  const bool b16 = !dense && blk == 16;
  const int max_blocks = dense ? l_cap / kBlk : k_max;
  const int n_slot = decode_num_splits(batch, h_kv, max_blocks, G, b16 ? 4 : 1);
  // The workspace layout follows the 64-token split count (never smaller),
  // so the completion counters sit at the same place for either block size.
  const int n_lay = decode_num_splits(batch, h_kv, max_blocks, G, 1);
  const int n_pairs = batch * h_kv;
  float* ws_o = static_cast<float*>(ws);
  float* ws_ml = ws_o + (size_t)batch * h_q * n_lay * kD;
  if (!counters) counters = reinterpret_cast<unsigned*>(ws_ml + (size_t)batch * h_q * n_lay * 2);
  auto o16 = static_cast<uint16_t*>(out);
  const float scale_log2 = sm_scale * kLog2e;
  dim3 grid(n_pairs * n_slot);
  auto qq = static_cast<const uint16_t*>(q);
  auto kk = static_cast<const uint16_t*>(k);
  auto vv = static_cast<const uint16_t*>(v);
#define SPOT_DECODE_LAUNCH(...)                                                               \
  hipLaunchKernelGGL((decode_split_kernel<__VA_ARGS__>), grid, dim3(64 * kDecWaves), 0, s, qq, \
                     kk, vv, seq_len, idx, count, k_max, h_q, h_kv, l_cap, scale_log2, n_slot,  \
                     ws_o, ws_ml, counters, o16, lse)
#define SPOT_DECODE_CASE(GG)                 \
  case GG:                                   \
    if (b16)                                 \
      SPOT_DECODE_LAUNCH(GG, false, 16);     \
    else if (dense)                          \
      SPOT_DECODE_LAUNCH(GG, true);          \
    else                                     \
      SPOT_DECODE_LAUNCH(GG, false);         \
    break;
  // every group of up to 16 query heads per KV head (the tile's columns)
  switch (G) {
    SPOT_DECODE_CASE(1) SPOT_DECODE_CASE(2) SPOT_DECODE_CASE(3) SPOT_DECODE_CASE(4)
    SPOT_DECODE_CASE(5) SPOT_DECODE_CASE(6) SPOT_DECODE_CASE(7) SPOT_DECODE_CASE(8)
    SPOT_DECODE_CASE(9) SPOT_DECODE_CASE(10) SPOT_DECODE_CASE(11) SPOT_DECODE_CASE(12)
    SPOT_DECODE_CASE(13) SPOT_DECODE_CASE(14) SPOT_DECODE_CASE(15) SPOT_DECODE_CASE(16)
    default: return hipErrorInvalidValue;
  }
#undef SPOT_DECODE_CASE
#undef SPOT_DECODE_LAUNCH
  return hipGetLastError();
}

}  // namespace spot
