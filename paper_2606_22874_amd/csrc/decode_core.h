// Split-KV decode attention core shared by the stand-alone decode kernel and
// the fused decode step.
//
// The layer attends only to the tokens of the selected 64-token blocks
// (paper Section 2 and the method figure: attention over the gathered K_I,
// V_I; one block set per query, shared by every head).
//
// Work split: grid (n_split, h_kv, batch).  A workgroup owns every n_split-th
// entry of its sequence's block list and the whole GQA group of G query
// heads of one KV head, so every K/V byte is read from HBM exactly once.  The
// workgroup has 4 waves; wave w owns token rows [16w, 16w+16) of every
// 64-token block and keeps its own online-softmax state per head.  Per block
// a wave's arithmetic is two small matrix products on the matrix cores, run
// transposed so that the scores never leave the registers (the GQA group's
// heads are the 16 columns of each tile, G of them real):
//   S^T = K Q^T       4 v_mfma_f32_16x16x32_bf16: the wave's 16 K rows are
//                     the A operand straight from global memory (16-byte
//                     loads), Q^T the B operand held for the whole loop;
//   online softmax    per head = per lane column: block maximum over the 4
//                     rows a lane holds and the 4 lane groups (two lane
//                     swaps), a lazy rescale (only when a maximum grows by
//                     more than 2^kLazy), exponentials in the log2 domain;
//   O^T += V^T P^T    8 v_mfma_f32_16x16x16_bf16: P^T goes from the score
//                     accumulators straight into the B operand (rounded to
//                     BF16), V^T comes from the wave's V rows in LDS through
//                     the transposing read ds_read_b64_tr_b16.
// The C layout of a 16x16 tile gives lane l the rows 4(l/16)..4(l/16)+3 of
// column l%16; the A/B layouts give lane l the consecutive k entries of row
// (A) or column (B) l%16 starting at k = 8(l/16) (16x16x32) or 4(l/16)
// (16x16x16).  The next two blocks' K and V rows are in flight in registers
// while one is computed.
// Blocks of 16 tokens (SB = 16, the paper's selector block): the loop runs
// over "virtual blocks" of four consecutive entries of the workgroup's list
// (the last one padded with -1), and wave w takes entry 4n + w of virtual
// block n -- the same 16-row loads; rows of a padding entry are masked like
// rows past seq_len.  Each wave keeps its own softmax state, so which
// tokens a wave sees does not matter to the merge.
// After the block loop the 4 waves' (m, l, O) states are merged in LDS into
// one partial per head; the last split to finish for a (sequence, KV head)
// merges all splits with log-sum-exp weights, rounds to BF16 and resets the
// completion counter, so the whole call is one kernel launch.
#pragma once

#include "spot_internal.h"

namespace spot {
namespace dec {


constexpr int kD = 128;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxIds = 512;     // max list entries per workgroup
static_assert(kMaxIds % 4 == 0, "16-token blocks pad the list to whole virtual blocks");

// ------------------------------------------------ coherent split partials
// Split partials cross workgroups that may run on different XCDs (each with
// its own L2).  They are written and read with relaxed device-scope atomic
// accesses, which go to the device coherence point, so no L2-wide writeback
// or invalidate is needed; a vmcnt(0) wait orders the partial stores before
// the completion-counter increment.
__device__ __forceinline__ void store_coherent(float* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_coherent(const float* p) {
  return __builtin_bit_cast(
      float2, __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Orders this wave's LDS accesses (LDS executes a wave's operations in order;
// this only stops the compiler from moving them across).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Log-sum-exp merge of n <= 16 partials of query head bh held by one wave:
// lane u < n has partial u's (m, l) in t, every lane has the partials'
// output dims 2*lane, 2*lane+1 in o[u].  Writes out (BF16) and lse; fixed
// order, so deterministic.
__device__ __forceinline__ void merge_small(float2 t, const float2 (&o)[16], int n, size_t bh,
                                            uint16_t* __restrict__ out, float* __restrict__ lse,
                                            int lane) {
  const float M = wave_max(t.y > 0.f ? t.x : -INFINITY);
  const float wgt = t.y > 0.f ? exp2f(t.x - M) : 0.f;
  const float L = wave_sum(t.y * wgt);
  float o0 = 0.f, o1 = 0.f;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    if (u < n) {
      const float wt = readlane_f(wgt, u);
      o0 = fmaf(o[u].x, wt, o0);
      o1 = fmaf(o[u].y, wt, o1);
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const uint32_t packed = (uint32_t)f32_to_bf16_rne(o0 * inv) |
                          ((uint32_t)f32_to_bf16_rne(o1 * inv) << 16);
  *reinterpret_cast<uint32_t*>(&out[bh * kD + 2 * lane]) = packed;
  if (lse && lane == 0) lse[bh] = L > 0.f ? (M + log2f(L)) * 0.6931471805599453f : -INFINITY;
}

// Log-sum-exp merge of the n_split partials of query head bh by one wave
// (lane = output dims 2*lane, 2*lane+1); fixed order, so deterministic.
__device__ __forceinline__ void merge_head(const float* __restrict__ ws_o,
                                           const float* __restrict__ ws_ml, int n_split,
                                           size_t bh, uint16_t* __restrict__ out,
                                           float* __restrict__ lse, int lane) {
  const float* ml = ws_ml + bh * n_split * 2;
  if (n_split <= 16) {
    // one round trip: every partial's (m, l) and o in flight together
    const float2 t = lane < n_split ? load_coherent(ml + 2 * lane) : make_float2(-INFINITY, 0.f);
    const float* ob = ws_o + bh * n_split * kD + 2 * lane;
    float2 o[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (u < n_split) o[u] = load_coherent(ob + (size_t)u * kD);
    merge_small(t, o, n_split, bh, out, lse, lane);
    return;
  }
  float M = -INFINITY;
  for (int s = lane; s < n_split; s += 64) {
    const float2 t = load_coherent(ml + 2 * s);
    if (t.y > 0.f) M = fmaxf(M, t.x);
  }
  M = wave_max(M);
  float L = 0.f, o0 = 0.f, o1 = 0.f;
  if (M > -INFINITY) {
    for (int base = 0; base < n_split; base += 64) {
      const int s = base + lane;
      float wgt = 0.f, lw = 0.f;
      if (s < n_split) {
        const float2 t = load_coherent(ml + 2 * s);
        if (t.y > 0.f) {
          wgt = exp2f(t.x - M);
          lw = t.y * wgt;
        }
      }
      L += wave_sum(lw);
      const int nn = min(64, n_split - base);
      const float* ob = ws_o + (bh * n_split + base) * kD + 2 * lane;
      int t = 0;
      for (; t + 8 <= nn; t += 8) {  // 8 independent loads in flight
        float2 o[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = load_coherent(ob + (size_t)(t + u) * kD);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float wt = readlane_f(wgt, t + u);
          o0 = fmaf(o[u].x, wt, o0);
          o1 = fmaf(o[u].y, wt, o1);
        }
      }
      for (; t < nn; ++t) {
        const float wt = readlane_f(wgt, t);
        const float2 o = load_coherent(ob + (size_t)t * kD);
        o0 = fmaf(o.x, wt, o0);
        o1 = fmaf(o.y, wt, o1);
      }
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const uint32_t packed = (uint32_t)f32_to_bf16_rne(o0 * inv) |
                          ((uint32_t)f32_to_bf16_rne(o1 * inv) << 16);
  *reinterpret_cast<uint32_t*>(&out[bh * kD + 2 * lane]) = packed;
  if (lse && lane == 0) lse[bh] = L > 0.f ? (M + log2f(L)) * 0.6931471805599453f : -INFINITY;
}

// ---------------------------------------------------------- LDS layout
constexpr int kDecWaves = 4;         // waves per workgroup (16 token rows each)
constexpr int kVRowBytes = kD * 2;   // one V row, 256 bytes
constexpr float kLazy = 8.f;         // rescale only when a maximum grows by more (log2)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

template <int G>
struct DecodeSmem {
  static_assert(G >= 1 && G <= 16, "the heads of a group are the columns of a 16x16 tile");
  struct Merge {
    float ml[kDecWaves][G][2];                        // [wave][head] (m, l)
    alignas(16) float o[kDecWaves][G][kD];            // [wave][head][dim]
  };
  union {
    alignas(16) unsigned char v[kDecWaves][16 * kVRowBytes];   // each wave's V rows
    Merge merge;
  };
  int ids[kMaxIds];
  int n_local;
  int last;
};

// One completion counter per (sequence, KV head) pair in the workspace.
__device__ __forceinline__ unsigned* pair_counters(unsigned* counters, int pair) {
  return counters + pair;
}

// Appends the ids of wave 0's lanes that lie in [0, nb_valid) to ids[cnt ..]
// in lane order and returns the new count (ids past kMaxIds are dropped).
__device__ __forceinline__ int append_ids(int* ids, int cnt, int j, int nb_valid) {
  const int lane = __lane_id();
  const bool ok = j >= 0 && j < nb_valid;
  const unsigned long long m = __ballot(ok);
  const int pos = cnt + __popcll(m & ((1ull << lane) - 1ull));
  if (ok && pos < kMaxIds) ids[pos] = j;
  return cnt + __popcll(m);
}

// Block list source of decode_body: entries slot, slot + n_slot, slot +
// 2 n_slot, ... of the sequence's list idx[b, 0 .. min(count[b], k_max)).
// Interleaving keeps the workgroups' shares within one entry of each other
// for any count.  Called by wave 0 only.
struct ListFromIdx {
  const int32_t* idx;
  const int32_t* count;
  int k_max;
  __device__ __forceinline__ int operator()(int* ids, int b, int g, int slot, int n_slot,
                                            int nb_valid) const {
    (void)g;
    const int lane = __lane_id();
    const int n_entries = min(count[b], k_max);
    const int32_t* lst = idx + (size_t)b * k_max;
    int cnt = 0;
    for (int base = slot; base < n_entries; base += 64 * n_slot) {
      const int e = base + lane * n_slot;
      cnt = append_ids(ids, cnt, e < n_entries ? lst[e] : -1, nb_valid);
    }
    return min(cnt, kMaxIds);
  }
};

// ---------------------------------------------------------- the body
// Physical 16-byte chunk of logical chunk c of V row r in LDS: the
// transposing read takes 8 bytes from each of 8 rows at the same column per
// half wave, so rows r and r + 1 .. r + 7 must land in different bank
// groups; XOR with 2 (r % 8) moves the chunk pairs apart and keeps each
// pair's two chunks adjacent.
__device__ __forceinline__ int swz_v(int r, int c) { return c ^ ((r & 7) << 1); }

// Two floats -> packed BF16 pair, round to nearest even.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// Cross-lane partner values without LDS: the lane swaps exchange the two
// halves / the odd-even 16-lane rows of a register.
__device__ __forceinline__ float lanes_max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float lanes_max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float lanes_sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float lanes_sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Q^T as the B operand of S^T = K Q^T: lane l holds query head l%16 of the
// group (zero past G), dims 32 kc + 8(l/16) .. +8 for kc = 0 .. 3.
struct QueryFrag {
  bf16x8_t q[4];
};
template <int G>
__device__ __forceinline__ QueryFrag load_query_heads(const uint16_t* __restrict__ q, int b,
                                                      int g, int h_q) {
  const int lane = __lane_id(), hh = lane & 15, kg = lane >> 4;
  QueryFrag f;
#pragma unroll
  for (int kc = 0; kc < 4; ++kc) {
    u32x4 t = {0u, 0u, 0u, 0u};
    if (hh < G)
      t = *reinterpret_cast<const u32x4*>(q + ((size_t)b * h_q + g * G + hh) * kD + 32 * kc +
                                          8 * kg);
    f.q[kc] = __builtin_bit_cast(bf16x8_t, t);
  }
  return f;
}

// One workgroup's partial of one query head after its 4 waves are merged:
// M and L in every lane, output dims 2*lane and 2*lane+1 in o0, o1.  L == 0
// means no token was seen.
struct HeadPartial {
  float M, L, o0, o1;
};
// The partials a wave holds after the merge: heads wave + 4j (j < HPW) of the
// group; entries for heads >= G are unused.
template <int G>
struct Partials {
  static constexpr int HPW = (G + kDecWaves - 1) / kDecWaves;
  HeadPartial h[HPW];
};

// The block loop of a workgroup: blocks blk_of(0 .. n_local-1) of the KV
// head whose caches start at kh / vh ([l_cap, 128] each), tokens below sl.
// Wave w processes token rows [16w, 16w+16) of every block; the 4 waves'
// states are merged in LDS at the end (two barriers).  issued(n) is called
// by every wave right after it issued the loads of block n, so a caller can
// act once the last block's loads are in flight.  SB = 16: n_local counts
// virtual blocks, and blk_of(e) is list entry e (-1 for padding).
template <int G, int SB = kBlk, class BlkOf, class Issued>
__device__ __forceinline__ Partials<G> attend_blocks(DecodeSmem<G>& sm, const QueryFrag& qf,
                                                     const uint16_t* __restrict__ kh,
                                                     const uint16_t* __restrict__ vh, int sl,
                                                     int n_local, const BlkOf& blk_of,
                                                     float scale_log2, const Issued& issued) {
  static_assert(SB == kBlk || SB == 16, "blocks of 64 or 16 tokens");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;   // tile column / row, lane group
  unsigned char* vs = sm.v[wave];

  // First token of this wave's 16 rows in (virtual) block n; -1 for padding.
  auto base_tok = [&](int n) -> int {
    if constexpr (SB == kBlk) {
      return blk_of(n) * kBlk + wave * 16;
    } else {
      const int id = blk_of(4 * n + wave);
      return id < 0 ? -1 : id * SB;
    }
  };
  // K rows in the A layout of 16x16x32 (row r16, dims 32 kc + 8 kg .. +8) and
  // V rows lane-contiguously (load i: row 4i + kg, chunk r16).
  auto load = [&](u32x4 (&kr)[4], u32x4 (&vr)[4], int n) {
    const int tb = max(base_tok(n), 0);
    const uint16_t* kp = kh + (size_t)(tb + r16) * kD + 8 * kg;
    const uint16_t* vp = vh + (size_t)tb * kD + lane * 8;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      kr[kc] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + 32 * kc));
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vp + i * 512));
  };

  u32x4 krA[4], vrA[4], krB[4], vrB[4];
  f32x4_t o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_lane = 0.f;

  // V rows of the stage into the wave's LDS rows (swizzled), then S^T.
  auto front = [&](const u32x4 (&kr)[4], const u32x4 (&vr)[4]) -> f32x4_t {
    wave_lds_sync();  // this wave's reads of the previous rows are issued
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + kg;
      *reinterpret_cast<u32x4*>(vs + r * kVRowBytes + (swz_v(r, r16) << 4)) = vr[i];
    }
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kr[kc]), qf.q[kc],
                                                  s, 0, 0, 0);
    wave_lds_sync();
    return s;
  };
  // Softmax of the block's scores and O^T += V^T P^T.
  auto back = [&](int n, f32x4_t s) {
    const int tb = base_tok(n);
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = tb + 4 * kg + i;
      x[i] = tb >= 0 && t < sl ? s[i] * scale_log2 : -INFINITY;
    }
    float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    mx = lanes_max_xor32(lanes_max_xor16(mx));          // the head's block maximum
    if (__ballot(mx > m_run + kLazy) != 0ull) {           // some head's maximum grew
      const float m_new = fmaxf(m_run, mx);
      const float alpha = m_new == -INFINITY ? 1.f : exp2f(m_run - m_new);
      l_lane *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[dt] *= alpha;
      m_run = m_new;
    }
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = x[i] == -INFINITY ? 0.f : exp2f(x[i] - m_run);
    l_lane += (p[0] + p[1]) + (p[2] + p[3]);
    const s16x4_t pb =
        __builtin_bit_cast(s16x4_t, u32x2_t{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])});
    // V^T fragment of d tile dt: lane (kg, r16) addresses row 4 kg + r16/4,
    // columns 16 dt + 4 (r16 % 4) .. +3 and receives column 16 dt + r16 of
    // rows 4 kg .. 4 kg + 3.
    const int vr_row = 4 * kg + (r16 >> 2);
    const unsigned char* vrow = vs + vr_row * kVRowBytes + (r16 & 1) * 8;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const int c = 2 * dt + ((r16 & 3) >> 1);
      const s16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4_t*)(vrow + (swz_v(vr_row, c) << 4)));
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pb, o[dt], 0, 0, 0);
    }
  };

  // Two register stages: while block n is computed, blocks n+1 and n+2 are
  // loading.  The steady-state loop issues both prefetches unconditionally,
  // so the compiler's wait before each stage's first use counts only that
  // stage's loads (a conditional prefetch makes it wait for every load in
  // flight, which serialises the stream); the last one or two blocks run
  // after the loop.
  int n = 0;
  if (n_local >= 4) {
    load(krA, vrA, 0);
    issued(0);
    load(krB, vrB, 1);
    issued(1);
    for (; n + 3 < n_local; n += 2) {
      f32x4_t s = front(krA, vrA);
      load(krA, vrA, n + 2);
      issued(n + 2);
      back(n, s);
      s = front(krB, vrB);
      load(krB, vrB, n + 3);
      issued(n + 3);
      back(n + 1, s);
    }
    // n_local - n is 2 or 3: blocks n and n + 1 are in flight
    f32x4_t s = front(krA, vrA);
    if (n + 2 < n_local) {
      load(krA, vrA, n + 2);
      issued(n + 2);
    }
    back(n, s);
    s = front(krB, vrB);
    back(n + 1, s);
    if (n + 2 < n_local) {
      s = front(krA, vrA);
      back(n + 2, s);
    }
  } else {
    if (n_local > 0) {
      load(krA, vrA, 0);
      issued(0);
    }
    if (n_local > 1) {
      load(krB, vrB, 1);
      issued(1);
    }
    if (n_local > 2) {
      f32x4_t s = front(krA, vrA);
      load(krA, vrA, 2);
      issued(2);
      back(0, s);
      s = front(krB, vrB);
      back(1, s);
      s = front(krA, vrA);
      back(2, s);
    } else {
      if (n_local > 0) back(0, front(krA, vrA));
      if (n_local > 1) back(1, front(krB, vrB));
    }
  }

  // ---- merge the 4 waves into one partial per head ----
  const float l_head = lanes_sum_xor32(lanes_sum_xor16(l_lane));   // column r16's sum
  __syncthreads();  // every wave is done with its V rows (aliased below)
  if (r16 < G) {
    if (kg == 0) {
      sm.merge.ml[wave][r16][0] = m_run;
      sm.merge.ml[wave][r16][1] = l_head;
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
      *reinterpret_cast<f32x4_t*>(&sm.merge.o[wave][r16][16 * dt + 4 * kg]) = o[dt];
  }
  __syncthreads();
  Partials<G> r;
#pragma unroll
  for (int j = 0; j < Partials<G>::HPW; ++j) {
    const int h = wave + kDecWaves * j;   // this wave merges head h of the group
    float M = -INFINITY, L = 0.f, o0 = 0.f, o1 = 0.f;
    if (h < G) {
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w)
        if (sm.merge.ml[w][h][1] > 0.f) M = fmaxf(M, sm.merge.ml[w][h][0]);
      if (M > -INFINITY) {
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) {
          const float lw = sm.merge.ml[w][h][1];
          const float wgt = lw > 0.f ? exp2f(sm.merge.ml[w][h][0] - M) : 0.f;
          L = fmaf(lw, wgt, L);
          const float2 ov = *reinterpret_cast<const float2*>(&sm.merge.o[w][h][2 * lane]);
          o0 = fmaf(ov.x, wgt, o0);
          o1 = fmaf(ov.y, wgt, o1);
        }
      }
    }
    r.h[j] = HeadPartial{M, L, o0, o1};
  }
  return r;
}

struct NoHook {
  __device__ __forceinline__ void operator()(int) const {}
};

// Workgroup (pair, slot): slot s takes its share of the pair's block list
// (from `list`; DENSE: the s-th contiguous run of all valid blocks); wave w
// processes token rows [16w, 16w+16) of each of those blocks.  The split
// partials go to the workspace; the last workgroup of the pair to finish
// (device-scope counter) merges them.  Returns true in that workgroup.
template <int G, bool DENSE, class List, int SB = kBlk>
__device__ __forceinline__ bool decode_body(
    DecodeSmem<G>& sm, const List& list, int pair, int slot, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const int32_t* __restrict__ seq_len, int h_q, int h_kv, int l_cap,
    float scale_log2, int n_slot, float* __restrict__ ws_o, float* __restrict__ ws_ml,
    unsigned* __restrict__ counters, uint16_t* __restrict__ out, float* __restrict__ lse) {
  const int b = pair / h_kv, g = pair % h_kv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  unsigned* pc = pair_counters(counters, pair);

  const QueryFrag qf = load_query_heads<G>(q, b, g, h_q);

  const int sl = min(seq_len[b], l_cap);
  const int nb_valid = (sl + SB - 1) / SB;
  // DENSE: this workgroup's contiguous run [e0, e1) of the valid blocks.
  const int bps = (nb_valid + n_slot - 1) / n_slot;
  const int e0 = slot * bps;
  const int e1 = min(e0 + bps, nb_valid);
  if (!DENSE && wave == 0) {
    int n = list(sm.ids, b, g, slot, n_slot, nb_valid);
    if constexpr (SB != kBlk) {
      // pad the last virtual block of four entries (kMaxIds is a multiple of 4)
      if (lane < 3 && n + lane < ((n + 3) & ~3)) sm.ids[n + lane] = -1;
      n = (n + 3) / 4;
    }
    if (lane == 0) sm.n_local = n;
  }
  __syncthreads();
  const int n_local = DENSE ? max(e1 - e0, 0) : sm.n_local;
  const size_t head_base = ((size_t)b * h_kv + g) * (size_t)l_cap * kD;
  auto blk_of = [&](int n) { return DENSE ? e0 + n : sm.ids[n]; };
  const Partials<G> hp = attend_blocks<G, SB>(sm, qf, k + head_base, v + head_base, sl,
                                              n_local, blk_of, scale_log2, NoHook{});
#pragma unroll
  for (int j = 0; j < Partials<G>::HPW; ++j) {
    const int h = wave + kDecWaves * j;
    if (h < G) {
      const size_t ps = ((size_t)b * h_q + g * G + h) * n_slot + slot;
      store_coherent(&ws_o[ps * kD + 2 * lane], make_float2(hp.h[j].o0, hp.h[j].o1));
      if (lane == 0) store_coherent(&ws_ml[ps * 2], make_float2(hp.h[j].M, hp.h[j].L));
    }
  }

  // ---- the last workgroup of the pair merges all slots ----
  wait_stores();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&pc[0], 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    sm.last = prev == (unsigned)(n_slot - 1);
  }
  __syncthreads();
  if (!sm.last) return false;
#pragma unroll
  for (int j = 0; j < Partials<G>::HPW; ++j) {
    const int h = wave + kDecWaves * j;
    if (h < G) merge_head(ws_o, ws_ml, n_slot, (size_t)b * h_q + g * G + h, out, lse, lane);
  }
  if (tid == 0) __hip_atomic_store(&pc[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

}  // namespace dec
}  // namespace spot
