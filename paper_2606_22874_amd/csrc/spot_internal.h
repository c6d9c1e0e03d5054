// Internal declarations shared by the HIP sources of libspot (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spot.h"

namespace spot {

constexpr int kBlk = 64;      // tokens per KV block
constexpr int kWave = 64;     // CDNA wavefront width

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

// Two bf16 products summed into an fp32 accumulator (v_dot2_f32_bf16).
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                          __builtin_bit_cast(bf16x2_t, b), c, false);
}

// float -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ------------------------------------------------------ wave reductions
// Butterfly reductions over all 64 lanes; every lane receives the result.
// The combination order is fixed, so results are deterministic.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v += __shfl_xor(v, off, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}

// ------------------------------------------------------ kernel launchers
// Each returns hipSuccess or the launch error; arguments are pre-validated.
hipError_t launch_selector_score(const void* q_sel, const float* w, const void* k_sel,
                                 const void* k_scale, int kfmt, int n_seq, int rows_per_seq,
                                 int nblk, int h_s, int d_s, const int32_t* n_valid,
                                 float* scores, hipStream_t s);

hipError_t launch_select_blocks(const float* scores, int rows, int nblk, const int32_t* n_valid,
                                float top_p, int k_max, int k_min, int n_sink, int n_recent,
                                int32_t* idx, int32_t* count, float* nuc_mass, hipStream_t s);

int decode_num_splits(int batch, int h_kv, int max_blocks);
size_t decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks);

hipError_t launch_decode(bool dense, const void* q, const void* k, const void* v,
                         const int32_t* seq_len, const int32_t* idx, const int32_t* count,
                         int k_max, int batch, int h_q, int h_kv, int l_cap, float sm_scale,
                         void* out, float* lse, void* ws, hipStream_t s);

hipError_t launch_sparse_prefill(const void* q, const void* k, const void* v, int L,
                                 const int32_t* idx, const int32_t* count, int k_max,
                                 int batch, int h_q, int h_kv, float sm_scale, void* out,
                                 float* lse, hipStream_t s);

}  // namespace spot
