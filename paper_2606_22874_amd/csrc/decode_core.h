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
// workgroup has G waves; wave w owns token rows [w*T, (w+1)*T) (T = 64/G) of
// every 64-token block, and its lanes are (head h, token t) = (lane / T,
// lane % T):
//   * each wave streams its own contiguous T-row slices of K and V (16-byte
//     coalesced loads, the next block's slice already in flight in registers)
//     through a wave-private LDS region -- no workgroup barrier per block;
//   * Q.K: lane (h, t) takes the full 128-dim dot product of query head h with
//     key row t using packed BF16 dot2; the G lanes reading the same key row
//     are served by one LDS broadcast;
//   * online softmax per head in the log2 domain over the T lanes of the head
//     (DPP reductions), lane-local running sums;
//   * P.V: lane = pair of output dims, all G heads, probabilities broadcast
//     from LDS.
// Blocks of 16 tokens (SB = 16, the paper's selector block): the loop runs
// over "virtual blocks" of four consecutive entries of the workgroup's list
// (the last one padded with -1), and wave row r of virtual block n is row
// (wT + r) % 16 of entry 4n + (wT + r) / 16 -- the same slice shapes, loads
// and LDS layout, with a per-row token address; rows of a padding entry are
// masked like rows past seq_len.  Each wave keeps its own softmax state, so
// which tokens a wave sees does not matter to the merge.
// After the block loop the G waves' (m, l, o) states are merged in LDS into
// one partial per head; the last split to finish for a (sequence, KV head)
// merges all splits with log-sum-exp weights, rounds to BF16 and resets the
// completion counter, so the whole call is one kernel launch.
#pragma once

#include "spot_internal.h"

namespace spot {
namespace dec {


constexpr int kD = 128;
constexpr int kKRow = kD + 8;    // padded K row in LDS (272 bytes)
// Occupancy target in waves per SIMD (caps VGPRs without spilling).
constexpr int waves_per_eu(int G) { return G >= 4 ? 2 : 1; }
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

// ------------------------------------------- reductions over T-lane groups
// Max / sum over the T consecutive lanes of a group (T in {8, 16, 32, 64});
// every lane of the group receives the result.
template <int T>
__device__ __forceinline__ float group_max(float v) {
  v = fmaxf(v, dpp_f<kDppQuadXor1>(v));
  v = fmaxf(v, dpp_f<kDppQuadXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  if (T >= 16) v = fmaxf(v, dpp_f<kDppMirror>(v));
  if (T >= 32) v = fmaxf(v, __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F)));
  if (T >= 64) v = fmaxf(readlane_f(v, 0), readlane_f(v, 32));
  return v;
}
template <int T>
__device__ __forceinline__ float group_sum(float v) {
  v += dpp_f<kDppQuadXor1>(v);
  v += dpp_f<kDppQuadXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  if (T >= 16) v += dpp_f<kDppMirror>(v);
  if (T >= 32) v += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F));
  if (T >= 64) v = readlane_f(v, 0) + readlane_f(v, 32);
  return v;
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

// One T-row slice of a block's K and of its V (contiguous T x 256 bytes each)
// into registers: 16-byte chunk c = i * 64 + lane.
template <int NLD>
__device__ __forceinline__ void load_slice(u32x4 (&kr)[NLD], u32x4 (&vr)[NLD],
                                           const uint16_t* __restrict__ kw,
                                           const uint16_t* __restrict__ vw, int blk, int lane) {
  const size_t base = (size_t)blk * kBlk * kD;
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int c = i * 64 + lane;
    kr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kw + base + c * 8));
    vr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vw + base + c * 8));
  }
}

// ---------------------------------------------------------- LDS layout
template <int G>
struct DecodeSmem {
  static constexpr int T = 64 / G;                    // token rows per wave
  struct Wave {
    uint16_t k[T * kKRow];                            // K slice, padded rows
    uint16_t v[T * kD];                               // V slice
    float p[T][G];                                    // probabilities [token][head]
  };
  struct Merge {
    float ml[G][G][2];                                // [wave][head] (m, l)
    float o[G][G][kD];                                // [wave][head][dim]
  };
  union {
    Wave wave[G];
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
// The G query heads of KV head g of sequence b: lane (h, t) of every wave
// holds query head g*G + h (h = lane / T) as 64 packed BF16 pairs.
template <int G>
__device__ __forceinline__ void load_query_heads(uint32_t (&qv)[kD / 2],
                                                 const uint16_t* __restrict__ q, int b, int g,
                                                 int h_q) {
  constexpr int T = 64 / G;
  const int hh = __lane_id() / T;
  const u32x4* qp = reinterpret_cast<const u32x4*>(q + ((size_t)b * h_q + g * G + hh) * kD);
#pragma unroll
  for (int i = 0; i < kD / 8; ++i) {
    const u32x4 t = qp[i];
    qv[4 * i + 0] = t.x; qv[4 * i + 1] = t.y; qv[4 * i + 2] = t.z; qv[4 * i + 3] = t.w;
  }
}

// One workgroup's partial of one query head after its G waves are merged:
// wave w holds head w of the group (M and L in every lane, output dims
// 2*lane and 2*lane+1 in o0, o1).  L == 0 means no token was seen.
struct HeadPartial {
  float M, L, o0, o1;
};

// The block loop of a workgroup: blocks blk_of(0 .. n_local-1) of the KV
// head whose caches start at kh / vh ([l_cap, 128] each), tokens below sl.
// Wave w processes token rows [w*T, (w+1)*T) of every block; the G waves'
// states are merged in LDS at the end (two barriers).  issued(n) is called
// by every wave right after it issued the loads of block n, so a caller can
// act once the last block's loads are in flight.  SB = 16: n_local counts
// virtual blocks, and blk_of(e) is list entry e (-1 for padding).
template <int G, int SB = kBlk, class BlkOf, class Issued>
__device__ __forceinline__ HeadPartial attend_blocks(DecodeSmem<G>& sm,
                                                     const uint32_t (&qv)[kD / 2],
                                                     const uint16_t* __restrict__ kh,
                                                     const uint16_t* __restrict__ vh, int sl,
                                                     int n_local, const BlkOf& blk_of,
                                                     float scale_log2, const Issued& issued) {
  constexpr int T = 64 / G;               // token rows per wave per block
  constexpr int NLD = T * kD * 2 / 1024;  // 16-byte loads per lane per slice
  static_assert(NLD >= 1, "slice smaller than one wave load");
  static_assert(SB == kBlk || SB == 16, "blocks of 64 or 16 tokens");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane / T, tt = lane % T;  // this lane's (head, token row)

  // This wave's slice of a block starts at token row wave * T.
  const uint16_t* kw = kh + (size_t)wave * T * kD;
  const uint16_t* vw = vh + (size_t)wave * T * kD;
  auto& W = sm.wave[wave];

  // Loads of (virtual) block n into a register stage; 16-byte chunk
  // c = i * 64 + lane is row c / 16, column chunk c % 16 of the wave's slice.
  auto load = [&](u32x4 (&kr)[NLD], u32x4 (&vr)[NLD], int n) {
    if constexpr (SB == kBlk) {
      load_slice<NLD>(kr, vr, kw, vw, blk_of(n), lane);
    } else {
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const int wr = wave * T + 4 * i + (lane >> 4);
        const int id = blk_of(4 * n + (wr >> 4));
        const size_t off = (size_t)(id < 0 ? 0 : id * SB + (wr & (SB - 1))) * kD + (lane & 15) * 8;
        kr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kh + off));
        vr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vh + off));
      }
    }
  };
  // This lane's token (row tt of the wave's slice) in (virtual) block n; -1
  // for a padding entry.
  auto tok_of = [&](int n) {
    if constexpr (SB == kBlk) {
      return blk_of(n) * kBlk + wave * T + tt;
    } else {
      const int wr = wave * T + tt;
      const int id = blk_of(4 * n + (wr >> 4));
      return id < 0 ? -1 : id * SB + (wr & (SB - 1));
    }
  };

  // Register stages A and B hold the two blocks of the current chunk.
  u32x4 krA[NLD], vrA[NLD], krB[NLD], vrB[NLD];
  float m_run = -INFINITY, l_lane = 0.f;
  float acc[G][2];
#pragma unroll
  for (int h = 0; h < G; ++h) acc[h][0] = acc[h][1] = 0.f;

  auto consume = [&](const u32x4 (&kr)[NLD], const u32x4 (&vr)[NLD]) {
    wave_lds_sync();  // this wave's reads of the previous slice are issued
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int c = i * 64 + lane;
      *reinterpret_cast<u32x4*>(&W.k[(c >> 4) * kKRow + (c & 15) * 8]) = kr[i];
      *reinterpret_cast<u32x4*>(&W.v[c * 8]) = vr[i];
    }
    wave_lds_sync();
  };
  auto compute = [&](int tok) {
    // Q.K for (head hh, token row tt)
    const u32x4* krow = reinterpret_cast<const u32x4*>(&W.k[tt * kKRow]);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kD / 8; ++i) {
      const u32x4 kk = krow[i];
      s = dot2_bf16(qv[4 * i + 0], kk.x, s);
      s = dot2_bf16(qv[4 * i + 1], kk.y, s);
      s = dot2_bf16(qv[4 * i + 2], kk.z, s);
      s = dot2_bf16(qv[4 * i + 3], kk.w, s);
    }
    const bool tok_ok = (SB == kBlk || tok >= 0) && tok < sl;
    const float x = tok_ok ? s * scale_log2 : -INFINITY;
    const float m_new = fmaxf(m_run, group_max<T>(x));
    // A slice whose rows all lie past seq_len leaves the state unchanged.
    const bool live = m_new > -INFINITY;
    const float pr = live ? exp2f(x - m_new) : 0.f;
    const float alpha = live ? exp2f(m_run - m_new) : 1.f;
    m_run = m_new;
    l_lane = l_lane * alpha + pr;
    W.p[tt][hh] = pr;
    float al[G];
#pragma unroll
    for (int h = 0; h < G; ++h) al[h] = readlane_f(alpha, h * T);
    wave_lds_sync();

    // P.V: lane = output dims 2*lane, 2*lane+1 for every head of the group
#pragma unroll
    for (int h = 0; h < G; ++h) {
      acc[h][0] *= al[h];
      acc[h][1] *= al[h];
    }
#pragma unroll 4
    for (int t = 0; t < T; ++t) {
      float pt[G];
      if constexpr (G >= 4) {
#pragma unroll
        for (int h4 = 0; h4 < G; h4 += 4) {
          const float4 p4 = *reinterpret_cast<const float4*>(&W.p[t][h4]);
          pt[h4] = p4.x; pt[h4 + 1] = p4.y; pt[h4 + 2] = p4.z; pt[h4 + 3] = p4.w;
        }
      } else {
#pragma unroll
        for (int h = 0; h < G; ++h) pt[h] = W.p[t][h];
      }
      const uint32_t vv = *reinterpret_cast<const uint32_t*>(&W.v[t * kD + 2 * lane]);
      const float v0 = bf16_lo(vv), v1 = bf16_hi(vv);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        acc[h][0] = fmaf(pt[h], v0, acc[h][0]);
        acc[h][1] = fmaf(pt[h], v1, acc[h][1]);
      }
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
      consume(krA, vrA);
      load(krA, vrA, n + 2);
      issued(n + 2);
      compute(tok_of(n));
      consume(krB, vrB);
      load(krB, vrB, n + 3);
      issued(n + 3);
      compute(tok_of(n + 1));
    }
    // n_local - n is 2 or 3: blocks n and n + 1 are in flight
    consume(krA, vrA);
    if (n + 2 < n_local) {
      load(krA, vrA, n + 2);
      issued(n + 2);
    }
    compute(tok_of(n));
    consume(krB, vrB);
    compute(tok_of(n + 1));
    if (n + 2 < n_local) {
      consume(krA, vrA);
      compute(tok_of(n + 2));
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
      consume(krA, vrA);
      compute(tok_of(0));
      load(krA, vrA, 2);
      issued(2);
      consume(krB, vrB);
      compute(tok_of(1));
      consume(krA, vrA);
      compute(tok_of(2));
    } else {
      if (n_local > 0) {
        consume(krA, vrA);
        compute(tok_of(0));
      }
      if (n_local > 1) {
        consume(krB, vrB);
        compute(tok_of(1));
      }
    }
  }

  // ---- merge the G waves (token slices) into one partial per head ----
  const float l_grp = group_sum<T>(l_lane);
  __syncthreads();  // every wave is done with its slice buffers (aliased below)
  if (tt == 0) {
    sm.merge.ml[wave][hh][0] = m_run;
    sm.merge.ml[wave][hh][1] = l_grp;
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
    *reinterpret_cast<float2*>(&sm.merge.o[wave][h][2 * lane]) = make_float2(acc[h][0], acc[h][1]);
  __syncthreads();
  HeadPartial r;
  {
    const int h = wave;  // wave w merges head w of the group
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < G; ++w)
      if (sm.merge.ml[w][h][1] > 0.f) M = fmaxf(M, sm.merge.ml[w][h][0]);
    float L = 0.f, o0 = 0.f, o1 = 0.f;
    if (M > -INFINITY) {
#pragma unroll
      for (int w = 0; w < G; ++w) {
        const float lw = sm.merge.ml[w][h][1];
        const float wgt = lw > 0.f ? exp2f(sm.merge.ml[w][h][0] - M) : 0.f;
        L = fmaf(lw, wgt, L);
        const float2 o = *reinterpret_cast<const float2*>(&sm.merge.o[w][h][2 * lane]);
        o0 = fmaf(o.x, wgt, o0);
        o1 = fmaf(o.y, wgt, o1);
      }
    }
    r = HeadPartial{M, L, o0, o1};
  }
  return r;
}

struct NoHook {
  __device__ __forceinline__ void operator()(int) const {}
};

// Workgroup (pair, slot): slot s takes its share of the pair's block list
// (from `list`; DENSE: the s-th contiguous run of all valid blocks); wave w
// processes token rows [w*T, (w+1)*T) of each of those blocks.  The split
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

  uint32_t qv[kD / 2];
  load_query_heads<G>(qv, q, b, g, h_q);

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
  const HeadPartial hp = attend_blocks<G, SB>(sm, qv, k + head_base, v + head_base, sl,
                                              n_local, blk_of, scale_log2, NoHook{});
  {
    const int h = wave;
    const size_t ps = ((size_t)b * h_q + g * G + h) * n_slot + slot;
    store_coherent(&ws_o[ps * kD + 2 * lane], make_float2(hp.o0, hp.o1));
    if (lane == 0) store_coherent(&ws_ml[ps * 2], make_float2(hp.M, hp.L));
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
  merge_head(ws_o, ws_ml, n_slot, (size_t)b * h_q + g * G + wave, out, lse, lane);
  if (tid == 0) __hip_atomic_store(&pc[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

}  // namespace dec
}  // namespace spot
