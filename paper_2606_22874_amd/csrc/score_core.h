// Selector scoring core shared by the stand-alone scoring kernel and the
// fused decode step (paper Section 2.1):
//   scores[r, j] = sum_h w[r,h] * ReLU(q_sel[r,h,:] . kbar[seq(r), j, h, :]).
// The pooled key of one block is h_s * d_s = 512 elements.  One wavefront
// covers a whole block with one load per lane: lane l owns elements
// 8l .. 8l+7 (BF16: 16 bytes; 8-bit formats: 8 bytes of codes, 4-bit
// formats: 4 bytes, plus the scale of its 32-element group), so consecutive
// lanes read consecutive bytes.  The head dot products are reduced over the LPH = d_s/8 lanes of a
// head, passed through ReLU and weighted, then summed over heads -- all with
// a fixed butterfly, so the result is deterministic.
#pragma once

#include "spot_internal.h"

namespace spot {

// FP16 bits -> float (IEEE binary16, subnormals exact).
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

// E8M0 -> 2^(e-127) as float (e = 0 gives the subnormal 2^-127).
__device__ __forceinline__ float e8m0_to_f32(uint32_t e) {
  return e ? __uint_as_float(e << 23) : __uint_as_float(0x00400000u);
}

// Eight signed 4-bit codes of one word, nibble i (bits 4i .. 4i+3) holding
// element i, as floats scaled by 1/16: v_cvt_off_f32_i4 turns the low four
// bits of its operand into n / 16 (exact), and reading byte b of the word and
// of the word rotated right by 4 picks nibbles 2b and 2b+1 with a byte select
// on the operand, so the eight values cost nine instructions.  A sum of
// q_i * (n_i / 16) scaled by 16 equals the sum of q_i * n_i bit for bit
// (scaling by a power of two commutes with every rounding step).
__device__ __forceinline__ void int4_sixteenths(uint32_t w, float (&v)[8]) {
  const uint32_t odd = __builtin_amdgcn_alignbit(w, w, 4);
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    v[2 * b] = __builtin_amdgcn_cvt_off_f32_i4((int)((w >> (8 * b)) & 0xffu));
    v[2 * b + 1] = __builtin_amdgcn_cvt_off_f32_i4((int)((odd >> (8 * b)) & 0xffu));
  }
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Global loads, optionally non-temporal (NT: the line is not kept in the
// caches -- for data streamed exactly once, which then does not evict
// anything reused).
template <bool NT, class T>
__device__ __forceinline__ T ld(const void* p) {
  if constexpr (NT)
    return __builtin_nontemporal_load(reinterpret_cast<const T*>(p));
  else
    return *reinterpret_cast<const T*>(p);
}

template <int KFMT>
struct KeyLoad;

// BF16: 16 bytes per lane.
template <>
struct KeyLoad<SPOT_KFMT_BF16> {
  uint4 raw;
  template <bool NT = false>
  __device__ __forceinline__ void load(const uint8_t* kb, const uint8_t*, size_t blk, int lane) {
    const u32x4 t = ld<NT, u32x4>(kb + blk * 1024 + lane * 16);
    raw = make_uint4(t[0], t[1], t[2], t[3]);
  }
  __device__ __forceinline__ float dot(const uint4& qraw, const float*) const {
    float a = dot2_bf16(qraw.x, raw.x, 0.f);
    a = dot2_bf16(qraw.y, raw.y, a);
    a = dot2_bf16(qraw.z, raw.z, a);
    return dot2_bf16(qraw.w, raw.w, a);
  }
  // FP32 queries (integer query codes, which BF16 cannot hold exactly).
  __device__ __forceinline__ float dot_f(const float* qf) const {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
    float a = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a = fmaf(qf[2 * i], bf16_lo(w[i]), a);
      a = fmaf(qf[2 * i + 1], bf16_hi(w[i]), a);
    }
    return a;
  }
};

// INT4: 4 bytes of codes (element 2i in the low nibble) and one FP16 scale.
template <>
struct KeyLoad<SPOT_KFMT_INT4_G32> {
  uint32_t codes;
  uint16_t scale;
  template <bool NT = false>
  __device__ __forceinline__ void load(const uint8_t* kb, const uint8_t* ks, size_t blk, int lane) {
    codes = ld<NT, uint32_t>(kb + blk * 256 + lane * 4);
    scale = ld<NT, uint16_t>(ks + (blk * 16 + (lane >> 2)) * 2);
  }
  __device__ __forceinline__ float dot(const uint4&, const float* qf) const {
    float v[8];
    int4_sixteenths(codes, v);
    float a = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) a = fmaf(qf[i], v[i], a);
    return a * 16.f * f16_to_f32(scale);
  }
  __device__ __forceinline__ float dot_f(const float* qf) const { return dot(uint4{}, qf); }
};

// MXFP4: 4 bytes of E2M1 codes and one E8M0 scale.
template <>
struct KeyLoad<SPOT_KFMT_MXFP4_G32> {
  uint32_t codes;
  uint8_t scale;
  template <bool NT = false>
  __device__ __forceinline__ void load(const uint8_t* kb, const uint8_t* ks, size_t blk, int lane) {
    codes = ld<NT, uint32_t>(kb + blk * 256 + lane * 4);
    scale = ld<NT, uint8_t>(ks + blk * 16 + (lane >> 2));
  }
  __device__ __forceinline__ float dot(const uint4&, const float* qf) const {
    // v_cvt_scalef32_pk_f32_fp4 (scale 1): byte b of the codes -> the exact
    // E2M1 values of its low and high nibble (elements 2b, 2b+1); the E8M0
    // scale is applied once to the sum, in FP32.
    const f32x2 v0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, 1.0f, 0);
    const f32x2 v1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, 1.0f, 1);
    const f32x2 v2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, 1.0f, 2);
    const f32x2 v3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, 1.0f, 3);
    float a = fmaf(qf[0], v0[0], 0.f);
    a = fmaf(qf[1], v0[1], a);
    a = fmaf(qf[2], v1[0], a);
    a = fmaf(qf[3], v1[1], a);
    a = fmaf(qf[4], v2[0], a);
    a = fmaf(qf[5], v2[1], a);
    a = fmaf(qf[6], v3[0], a);
    a = fmaf(qf[7], v3[1], a);
    return a * e8m0_to_f32(scale);
  }
  __device__ __forceinline__ float dot_f(const float* qf) const { return dot(uint4{}, qf); }
};

// INT8: 8 bytes of two's-complement codes and one FP16 scale.
template <>
struct KeyLoad<SPOT_KFMT_INT8_G32> {
  u32x2 codes;
  uint16_t scale;
  template <bool NT = false>
  __device__ __forceinline__ void load(const uint8_t* kb, const uint8_t* ks, size_t blk, int lane) {
    codes = ld<NT, u32x2>(kb + blk * 512 + lane * 8);
    scale = ld<NT, uint16_t>(ks + (blk * 16 + (lane >> 2)) * 2);
  }
  __device__ __forceinline__ float dot(const uint4&, const float* qf) const {
    float a = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int code = (int)(codes[i >> 2] << (24 - 8 * (i & 3))) >> 24;  // sign-extend byte
      a = fmaf(qf[i], (float)code, a);
    }
    return a * f16_to_f32(scale);
  }
  __device__ __forceinline__ float dot_f(const float* qf) const { return dot(uint4{}, qf); }
};

// MXFP8: 8 bytes of OCP E4M3 codes and one E8M0 scale.
template <>
struct KeyLoad<SPOT_KFMT_MXFP8_G32> {
  u32x2 codes;
  uint8_t scale;
  template <bool NT = false>
  __device__ __forceinline__ void load(const uint8_t* kb, const uint8_t* ks, size_t blk, int lane) {
    codes = ld<NT, u32x2>(kb + blk * 512 + lane * 8);
    scale = ld<NT, uint8_t>(ks + blk * 16 + (lane >> 2));
  }
  __device__ __forceinline__ float dot(const uint4&, const float* qf) const {
    // v_cvt_scalef32_pk_f32_fp8 (scale 1): the two E4M3 bytes of the low or
    // high half-word -> their exact values; the E8M0 scale multiplies the sum.
    const f32x2 v0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(codes[0], 1.0f, false);
    const f32x2 v1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(codes[0], 1.0f, true);
    const f32x2 v2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(codes[1], 1.0f, false);
    const f32x2 v3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(codes[1], 1.0f, true);
    float a = fmaf(qf[0], v0[0], 0.f);
    a = fmaf(qf[1], v0[1], a);
    a = fmaf(qf[2], v1[0], a);
    a = fmaf(qf[3], v1[1], a);
    a = fmaf(qf[4], v2[0], a);
    a = fmaf(qf[5], v2[1], a);
    a = fmaf(qf[6], v3[0], a);
    a = fmaf(qf[7], v3[1], a);
    return a * e8m0_to_f32(scale);
  }
  __device__ __forceinline__ float dot_f(const float* qf) const { return dot(uint4{}, qf); }
};

// One wavefront scores blocks j0 .. min(j0 + U, jend) - 1 of query row `row`
// (sequence `seq`), all key loads issued before any arithmetic; blocks at or
// past nv score -inf.  A non-null rec (the row's record words, indexed by
// block; rec_copies runs of them rec_stride words apart) also receives
// rec_word() of each valid block's score in every run, stored at device
// scope (readers in other workgroups of the same launch poll these words:
// zero means not written yet).  A null `scores` stores no scores.  Returns,
// in lane u < U, the score of block j0 + u (-inf in the other lanes and past
// jend).
// This lane's 8 query elements of row `row` (head lane / LPH, dims
// 8*(lane % LPH) ..).  BF16 and MX queries: BF16 bits in qraw and floats in
// qf, qsc = 1 (MX codes -- E2M1 or E4M3, one E8M0 scale per 32 -- times a
// power of two fit BF16, so they are decoded exactly into both).  INT4 / INT8
// queries (one FP16 scale per 32): the integer codes as floats in qf (exact)
// and the group's scale in qsc, applied to the lane's partial dot product;
// qraw is unused.
template <int QFMT>
__device__ __forceinline__ void load_query(const uint8_t* __restrict__ q,
                                           const uint8_t* __restrict__ q_scale, int row,
                                           int lane, uint4& qraw, float (&qf)[8], float& qsc) {
  qsc = 1.f;
  if constexpr (QFMT == SPOT_KFMT_BF16) {
    qraw = *reinterpret_cast<const uint4*>(q + (size_t)row * 1024 + lane * 16);
    qf[0] = bf16_lo(qraw.x); qf[1] = bf16_hi(qraw.x);
    qf[2] = bf16_lo(qraw.y); qf[3] = bf16_hi(qraw.y);
    qf[4] = bf16_lo(qraw.z); qf[5] = bf16_hi(qraw.z);
    qf[6] = bf16_lo(qraw.w); qf[7] = bf16_hi(qraw.w);
  } else if constexpr (QFMT == SPOT_KFMT_INT4_G32 || QFMT == SPOT_KFMT_INT8_G32) {
    qraw = make_uint4(0u, 0u, 0u, 0u);
    qsc = f16_to_f32(*reinterpret_cast<const uint16_t*>(q_scale + ((size_t)row * 16 + (lane >> 2)) * 2));
    if constexpr (QFMT == SPOT_KFMT_INT4_G32) {
      const uint32_t c = *reinterpret_cast<const uint32_t*>(q + (size_t)row * 256 + lane * 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) qf[i] = (float)((int)(c << (28 - 4 * i)) >> 28);
    } else {
      const u32x2 c = *reinterpret_cast<const u32x2*>(q + (size_t)row * 512 + lane * 8);
#pragma unroll
      for (int i = 0; i < 8; ++i) qf[i] = (float)((int)(c[i >> 2] << (24 - 8 * (i & 3))) >> 24);
    }
  } else {
    static_assert(QFMT == SPOT_KFMT_MXFP4_G32 || QFMT == SPOT_KFMT_MXFP8_G32,
                  "queries: BF16, INT4, INT8 or an MX format");
    const float sf = e8m0_to_f32(q_scale[(size_t)row * 16 + (lane >> 2)]);
    f32x2 v[4];
    if constexpr (QFMT == SPOT_KFMT_MXFP4_G32) {
      const uint32_t c = *reinterpret_cast<const uint32_t*>(q + (size_t)row * 256 + lane * 4);
      v[0] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, sf, 0);
      v[1] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, sf, 1);
      v[2] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, sf, 2);
      v[3] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, sf, 3);
    } else {
      const u32x2 c = *reinterpret_cast<const u32x2*>(q + (size_t)row * 512 + lane * 8);
      v[0] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(c[0], sf, false);
      v[1] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(c[0], sf, true);
      v[2] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(c[1], sf, false);
      v[3] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(c[1], sf, true);
    }
    uint32_t wd[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      qf[2 * i] = v[i][0];
      qf[2 * i + 1] = v[i][1];
      wd[i] = (__float_as_uint(v[i][0]) >> 16) | (__float_as_uint(v[i][1]) & 0xffff0000u);
    }
    qraw = make_uint4(wd[0], wd[1], wd[2], wd[3]);
  }
}

// Butterfly step of the score reductions: x + (x of lane l ^ OFF) in every
// lane (both lanes of a pair form the same sum, addition being commutative).
// Without LDS: quad permutes for 1 and 2; for 4 and 8 the half-row and row
// mirrors, whose partner lane holds the same value as lane l ^ OFF once the
// groups of OFF lanes are summed; the lane-swap instructions for 16 and 32.
template <int OFF>
__device__ __forceinline__ float xor_add(float x) {
#pragma clang fp contract(off)
  if constexpr (OFF == 1) {
    return x + dpp_f<kDppQuadXor1>(x);
  } else if constexpr (OFF == 2) {
    return x + dpp_f<kDppQuadXor2>(x);
  } else if constexpr (OFF == 4) {
    return x + dpp_f<kDppHalfMirror>(x);
  } else if constexpr (OFF == 8) {
    return x + dpp_f<kDppMirror>(x);
  } else if constexpr (OFF == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  } else {
    static_assert(OFF == 32, "lane offsets 1 .. 32");
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
}
// Sum over aligned groups of END lanes, given groups of FROM lanes already
// summed (every lane of a group holding the same value).
template <int FROM, int END>
__device__ __forceinline__ float xor_sum(float x) {
  if constexpr (FROM >= END)
    return x;
  else
    return xor_sum<FROM * 2, END>(xor_add<FROM>(x));
}

template <int KFMT, int LPH, int U, int QFMT = SPOT_KFMT_BF16>
__device__ __forceinline__ float score_blocks(const void* __restrict__ q_sel,
                                             const float* __restrict__ w,
                                             const uint8_t* __restrict__ k_sel,
                                             const uint8_t* __restrict__ k_scale, int row,
                                             int seq, int nblk, int nv, int j0, int jend,
                                             float* __restrict__ scores,
                                             uint32_t* __restrict__ rec, int lane,
                                             const uint8_t* __restrict__ q_scale = nullptr,
                                             int rec_copies = 1, size_t rec_stride = 0) {
  // No product is fused into a following addition: whether the compiler
  // fuses one depends on the code around the call (it did for some runs
  // of 8 blocks and not for runs of 16), and every caller must get the same
  // bits for a block, whatever its run.
#pragma clang fp contract(off)
  constexpr int kHeads = 64 / LPH;
  constexpr bool kIntQ = QFMT == SPOT_KFMT_INT4_G32 || QFMT == SPOT_KFMT_INT8_G32;
  uint4 qraw;
  float qf[8], qsc;
  load_query<QFMT>(static_cast<const uint8_t*>(q_sel), q_scale, row, lane, qraw, qf, qsc);
  const float wh = w[(size_t)row * kHeads + lane / LPH];

  // Every slot loads (branch-free, so the loads of all U blocks fly
  // together); a slot past the last valid block rereads that block (or
  // block 0), which stays in bounds and in cache, and its score is dropped.
  KeyLoad<KFMT> key[U];
  const int jlim = min(jend, max(nv, 1)) - 1;
#pragma unroll
  for (int u = 0; u < U; ++u)
    key[u].load(k_sel, k_scale, (size_t)seq * nblk + min(j0 + u, jlim), lane);
  float res = 0.f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float part = kIntQ ? key[u].dot_f(qf) * qsc : key[u].dot(qraw, qf);
    part = xor_sum<1, LPH>(part);
    float v = wh * fmaxf(part, 0.f);
    v = xor_sum<LPH, 64>(v);
    if (lane == u) res = v;
  }
  const int j = j0 + lane;
  const float val = lane < U && j < nv && j < jend ? res : -INFINITY;
  if (lane < U && j < jend) {
    if (rec && j < nv)
      for (int c = 0; c < rec_copies; ++c)
        __hip_atomic_store(rec + c * rec_stride + j, rec_word(val), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    if (scores) scores[(size_t)row * nblk + j] = val;
  }
  return val;
}

}  // namespace spot
