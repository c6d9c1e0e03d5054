// Internal declarations shared by the HIP sources of libspot (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spot.h"

namespace spot {

constexpr int kBlk = 64;      // tokens per KV block
constexpr int kWave = 64;     // CDNA wavefront width
constexpr int kMaxGroupSize = 16;   // query heads per KV head of the decode paths

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
// Cross-lane moves through DPP (quad permutes, row mirrors, row shifts) and
// v_readlane: no LDS round trip.  Every combination order is fixed, so the
// results are deterministic, and every lane receives the same value.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(dpp_i<CTRL>(__float_as_int(x)));
}
constexpr int kDppQuadXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;    // lane i <-> 7 - i within 8
constexpr int kDppMirror = 0x140;        // lane i <-> 15 - i within 16
constexpr int kDppRowShr1 = 0x111;

// Self-flagging record word of a float for readers in other workgroups of
// the same launch: the bit complement, so that no value maps to the zero
// "not written yet" word (the only float whose complement is zero, the NaN
// with every bit set, is replaced by the canonical quiet NaN first).
__device__ __forceinline__ uint32_t rec_word(float v) {
  const uint32_t u = __float_as_uint(v);
  return ~(u == 0xffffffffu ? 0x7fc00000u : u);
}
__device__ __forceinline__ float rec_value(uint32_t w) { return __uint_as_float(~w); }

__device__ __forceinline__ float readlane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<kDppQuadXor1>(v);
  v += dpp_f<kDppQuadXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return (readlane_f(v, 0) + readlane_f(v, 16)) + (readlane_f(v, 32) + readlane_f(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<kDppQuadXor1>(v));
  v = fmaxf(v, dpp_f<kDppQuadXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return fmaxf(fmaxf(readlane_f(v, 0), readlane_f(v, 16)),
               fmaxf(readlane_f(v, 32), readlane_f(v, 48)));
}
__device__ __forceinline__ int wave_sum_i(int v) {
  v += dpp_i<kDppQuadXor1>(v);
  v += dpp_i<kDppQuadXor2>(v);
  v += dpp_i<kDppHalfMirror>(v);
  v += dpp_i<kDppMirror>(v);
  return (__builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16)) +
         (__builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48));
}
__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
  v = max(v, (uint32_t)dpp_i<kDppQuadXor1>((int)v));
  v = max(v, (uint32_t)dpp_i<kDppQuadXor2>((int)v));
  v = max(v, (uint32_t)dpp_i<kDppHalfMirror>((int)v));
  v = max(v, (uint32_t)dpp_i<kDppMirror>((int)v));
  const uint32_t a = max((uint32_t)__builtin_amdgcn_readlane((int)v, 0),
                         (uint32_t)__builtin_amdgcn_readlane((int)v, 16));
  const uint32_t b = max((uint32_t)__builtin_amdgcn_readlane((int)v, 32),
                         (uint32_t)__builtin_amdgcn_readlane((int)v, 48));
  return max(a, b);
}
__device__ __forceinline__ uint32_t wave_min_u(uint32_t v) {
  v = min(v, (uint32_t)dpp_i<kDppQuadXor1>((int)v));
  v = min(v, (uint32_t)dpp_i<kDppQuadXor2>((int)v));
  v = min(v, (uint32_t)dpp_i<kDppHalfMirror>((int)v));
  v = min(v, (uint32_t)dpp_i<kDppMirror>((int)v));
  const uint32_t a = min((uint32_t)__builtin_amdgcn_readlane((int)v, 0),
                         (uint32_t)__builtin_amdgcn_readlane((int)v, 16));
  const uint32_t b = min((uint32_t)__builtin_amdgcn_readlane((int)v, 32),
                         (uint32_t)__builtin_amdgcn_readlane((int)v, 48));
  return min(a, b);
}
// Inclusive prefix sum over lanes 0..63 (row shifts within 16 lanes, then the
// row totals carried across rows).
__device__ __forceinline__ int wave_incl_scan_i(int x) {
  const int lane = __lane_id();
  x += dpp_i<0x111>(x);  // row_shr:1
  x += dpp_i<0x112>(x);  // row_shr:2
  x += dpp_i<0x114>(x);  // row_shr:4
  x += dpp_i<0x118>(x);  // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(x, 15);
  const int r1 = __builtin_amdgcn_readlane(x, 31);
  const int r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = lane >> 4;
  return x + (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
}

// ------------------------------------------------------ kernel launchers
// Each returns hipSuccess or the launch error; arguments are pre-validated.
hipError_t launch_selector_score(const void* q_sel, const float* w, const void* k_sel,
                                 const void* k_scale, int kfmt, int n_seq, int rows_per_seq,
                                 int nblk, int h_s, int d_s, const int32_t* n_valid,
                                 float* scores, hipStream_t s);

hipError_t launch_selector_score_q(const void* q_sel, const void* q_scale, int qfmt,
                                   const float* w, const void* k_sel, const void* k_scale,
                                   int kfmt, int n_seq, int rows_per_seq, int nblk, int d_s,
                                   const int32_t* n_valid, float* scores, hipStream_t s);

hipError_t launch_selector_score_tokens(const void* q_sel, const float* w, const void* k_tok,
                                        const void* k_scale, int kfmt, int n_seq,
                                        int rows_per_seq, int l_cap, int blk, int d_s,
                                        const int32_t* seq_len, float* scores, hipStream_t s);

hipError_t launch_selector_project(const void* h, const void* w_q, const void* w_k,
                                   const void* w_w, const int32_t* pos, int rows, int d_model,
                                   int h_s, int d_s, int rope_dim, float rope_base, void* q_out,
                                   float* w_out, void* k_cache, int rows_per_seq, int l_cap,
                                   void* k_pool, const int32_t* seq_len,
                                   hipStream_t s);
hipError_t launch_selector_pool(const void* k_tok, void* k_pool, int n_seq, int l_cap,
                                const int32_t* seq_len, const int32_t* first_block,
                                int max_blocks, hipStream_t s);

hipError_t launch_select_blocks(const float* scores, int rows, int nblk, const int32_t* n_valid,
                                float top_p, int k_max, int k_min, int n_sink, int n_recent,
                                int32_t* idx, int32_t* count, float* nuc_mass, hipStream_t s);

// per_virtual: list entries per loop step (1; 4 for 16-token blocks)
int decode_num_splits(int batch, int h_kv, int max_blocks, int group, int per_virtual = 1);
size_t decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks);

// Byte offsets in a decode step's workspace: the control region [0, ctrl)
// (completion counters, expiry word, score records, bitmaps; zero between
// calls) and the partials from `part` to `total`.
struct StepWs {
  size_t cnt, sticky, srec, brec, ctrl, part, total;
};
StepWs step_layout(int batch, int h_q, int h_kv, int k_max, size_t ctrl_cap);
size_t step_workspace_bytes(int batch, int h_q, int h_kv, int d, int k_max);
// The layout of the static scratch: its partials start at a fixed offset.
StepWs step_static_layout(int batch, int h_q, int h_kv, int k_max);
bool step_static_fits(int batch, int h_q, int h_kv, int k_max);
void step_force_expiry(int on);
size_t static_scratch_bytes();
// Device address of the current device's static scratch; with setup, looked
// up and zero-filled on `s` by the first call on the device (else NULL until
// then).
hipError_t static_scratch(void** out, bool setup, hipStream_t s);
bool step_fusable(int h_q, int h_kv, int nblk, int k_max);
hipError_t launch_decode_step(const void* q_sel, const void* q_scale, int qfmt, const float* w,
                              const void* k_sel, const void* k_scale, int kfmt, int d_s,
                              const int32_t* n_valid,
                              float top_p, int k_max, int k_min, int n_sink, int n_recent,
                              const void* q, const void* k, const void* v,
                              const int32_t* seq_len, int batch, int h_q, int h_kv, int l_cap,
                              float sm_scale, float* scores, int32_t* idx, int32_t* count,
                              float* nuc_mass, void* out, float* lse, void* ws, bool static_ws,
                              hipStream_t s);
// ws holds the partials, then (when counters is NULL) the completion
// counters, as decode_workspace_bytes lays them out.
hipError_t launch_decode(bool dense, const void* q, const void* k, const void* v,
                         const int32_t* seq_len, const int32_t* idx, const int32_t* count,
                         int k_max, int batch, int h_q, int h_kv, int l_cap, int blk,
                         float sm_scale, void* out, float* lse, void* ws, unsigned* counters,
                         hipStream_t s);

hipError_t launch_sparse_prefill(const void* q, const void* k, const void* v, int L,
                                 const int32_t* idx, const int32_t* count, int k_max,
                                 int batch, int h_q, int h_kv, float sm_scale, void* out,
                                 float* lse, hipStream_t s);

}  // namespace spot
