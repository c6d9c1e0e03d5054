// Block-sparse (and dense) GQA split-KV decode attention.
//
// The layer attends only to the tokens of the selected 64-token blocks
// (paper Section 2 and the method figure: attention over the gathered K_I,
// V_I; one block set per query, shared by every head).
//
// Work split: grid (n_split, h_kv, batch).  A workgroup of 256 threads owns a
// contiguous run of entries of the sequence's block list and the whole GQA
// group of query heads of one KV head, so each K/V block is read from HBM
// once and shared by all its query heads through LDS.  Per block:
//   * the 4 waves copy the 64 x 128 BF16 K and V tiles (16 KiB each) into LDS
//     with 16-byte coalesced loads; the next block's loads are already in
//     flight in registers while the current one is computed;
//   * Q.K: wave w handles query head(s) of the group, lane = token, the
//     128-dim dot product with packed BF16 dot2 instructions;
//   * online softmax in the log2 domain (running max, lane-local running sum);
//   * P.V: lane = pair of output dims, probabilities broadcast from LDS.
// Each split writes an unnormalised partial (m, l, o) and bumps a completion
// counter of its (sequence, KV head); the last split to arrive merges all of
// them with log-sum-exp weights, rounds to BF16 and resets the counter, so the
// whole call is one kernel launch.
#include "spot_internal.h"

namespace spot {
namespace {

constexpr int kD = 128;
constexpr int kThreads = 256;
constexpr int kRowU16 = kD + 8;        // padded LDS row (272 bytes)
constexpr int kMaxBps = 256;           // max block-list entries per split
constexpr float kLog2e = 1.4426950408889634f;

struct alignas(16) DecodeSmem {
  uint16_t k[kBlk * kRowU16];
  uint16_t v[kBlk * kRowU16];
  float p[4][2][kBlk];
  int ids[kMaxBps];
};

// Register staging of one 64 x 128 BF16 K tile and V tile: 4 x 16 bytes of
// each per thread, chunk c = p * 256 + tid covering row c / 16, dims
// 8 * (c % 16) .. +8 -- consecutive threads read consecutive 16-byte chunks.
__device__ __forceinline__ void load_tile(u32x4 (&kr)[4], u32x4 (&vr)[4],
                                          const uint16_t* __restrict__ kh,
                                          const uint16_t* __restrict__ vh, int blk, int tid) {
  const size_t base = (size_t)blk * kBlk * kD;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int c = p * kThreads + tid;
    const size_t off = base + (size_t)(c >> 4) * kD + (c & 15) * 8;
    kr[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kh + off));
    vr[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vh + off));
  }
}

__device__ __forceinline__ void store_tile(const u32x4 (&kr)[4], const u32x4 (&vr)[4],
                                           uint16_t* sk, uint16_t* sv, int tid) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int c = p * kThreads + tid;
    *reinterpret_cast<u32x4*>(&sk[(c >> 4) * kRowU16 + (c & 15) * 8]) = kr[p];
    *reinterpret_cast<u32x4*>(&sv[(c >> 4) * kRowU16 + (c & 15) * 8]) = vr[p];
  }
}

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

// Log-sum-exp merge of the n_split partials of query head bh by one wave
// (lane = output dims 2*lane, 2*lane+1); fixed order, so deterministic.
__device__ __forceinline__ void merge_head(const float* __restrict__ ws_o,
                                           const float* __restrict__ ws_ml, int n_split,
                                           size_t bh, uint16_t* __restrict__ out,
                                           float* __restrict__ lse, int lane) {
  const float* ml = ws_ml + bh * n_split * 2;
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

// G = query heads per KV head; HPW = query heads per wave (G <= 4: one head
// per wave and 4 - G idle waves; G = 8: two heads per wave).
template <int G, bool DENSE>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ seq_len,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int k_max, int h_q,
    int h_kv, int l_cap, float scale_log2, int bps, int n_split, float* __restrict__ ws_o,
    float* __restrict__ ws_ml, unsigned* __restrict__ counters, uint16_t* __restrict__ out,
    float* __restrict__ lse) {
  constexpr int HPW = G > 4 ? G / 4 : 1;
  __shared__ DecodeSmem sm;
  __shared__ int n_local_s;
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool active = wave * HPW < G;

  const int sl = min(seq_len[b], l_cap);
  const int nb_valid = (sl + kBlk - 1) / kBlk;
  const int n_entries = DENSE ? nb_valid : min(count[b], k_max);
  const int e0 = split * bps;
  const int e1 = min(e0 + bps, n_entries);

  // Valid block ids of this split, compacted in list order (ids outside
  // [0, nb_valid) are dropped, so no load can leave the cache).
  int n_local;
  if (DENSE) {
    n_local = max(e1 - e0, 0);
  } else {
    if (wave == 0) {
      int cnt = 0;
      for (int base = e0; base < e1; base += 64) {
        const int e = base + lane;
        const int j = e < e1 ? idx[(size_t)b * k_max + e] : -1;
        const bool ok = j >= 0 && j < nb_valid;
        const unsigned long long m = __ballot(ok);
        const int pos = cnt + __popcll(m & ((1ull << lane) - 1ull));
        if (ok) sm.ids[pos] = j;
        cnt += __popcll(m);
      }
      if (lane == 0) n_local_s = cnt;
    }
  }

  // Query heads of this wave: full 128-dim vectors as packed BF16 pairs.
  uint32_t qv[HPW][kD / 2];
  float m_run[HPW], l_lane[HPW], acc0[HPW], acc1[HPW];
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
    const int hq = g * G + min(wave * HPW + hh, G - 1);
    const uint4* qp = reinterpret_cast<const uint4*>(q + ((size_t)b * h_q + hq) * kD);
#pragma unroll
    for (int i = 0; i < kD / 8; ++i) {
      const uint4 t = qp[i];
      qv[hh][4 * i + 0] = t.x; qv[hh][4 * i + 1] = t.y;
      qv[hh][4 * i + 2] = t.z; qv[hh][4 * i + 3] = t.w;
    }
    m_run[hh] = -INFINITY;
    l_lane[hh] = 0.f;
    acc0[hh] = 0.f;
    acc1[hh] = 0.f;
  }
  __syncthreads();
  if (!DENSE) n_local = n_local_s;

  const size_t head_base = ((size_t)b * h_kv + g) * (size_t)l_cap * kD;
  const uint16_t* kh = k + head_base;
  const uint16_t* vh = v + head_base;

  u32x4 kr[4], vr[4];
  if (n_local > 0) load_tile(kr, vr, kh, vh, DENSE ? e0 : sm.ids[0], tid);

  for (int n = 0; n < n_local; ++n) {
    const int blk = DENSE ? e0 + n : sm.ids[n];
    __syncthreads();  // the previous block's LDS reads are done
    store_tile(kr, vr, sm.k, sm.v, tid);
    __syncthreads();
    if (n + 1 < n_local) load_tile(kr, vr, kh, vh, DENSE ? e0 + n + 1 : sm.ids[n + 1], tid);

    if (active) {
      const bool tok_ok = blk * kBlk + lane < sl;
      const uint4* krow = reinterpret_cast<const uint4*>(&sm.k[lane * kRowU16]);
      float s[HPW];
#pragma unroll
      for (int hh = 0; hh < HPW; ++hh) s[hh] = 0.f;
#pragma unroll
      for (int i = 0; i < kD / 8; ++i) {
        const uint4 kk = krow[i];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
          s[hh] = dot2_bf16(qv[hh][4 * i + 0], kk.x, s[hh]);
          s[hh] = dot2_bf16(qv[hh][4 * i + 1], kk.y, s[hh]);
          s[hh] = dot2_bf16(qv[hh][4 * i + 2], kk.z, s[hh]);
          s[hh] = dot2_bf16(qv[hh][4 * i + 3], kk.w, s[hh]);
        }
      }
#pragma unroll
      for (int hh = 0; hh < HPW; ++hh) {
        const float x = tok_ok ? s[hh] * scale_log2 : -INFINITY;
        // Every listed block has >= 1 valid token, so m_new is finite.
        const float m_new = fmaxf(m_run[hh], wave_max(x));
        const float pr = exp2f(x - m_new);
        const float alpha = exp2f(m_run[hh] - m_new);
        m_run[hh] = m_new;
        l_lane[hh] = l_lane[hh] * alpha + pr;
        acc0[hh] *= alpha;
        acc1[hh] *= alpha;
        sm.p[wave][hh][lane] = pr;
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll 4
      for (int t = 0; t < kBlk; t += 4) {
        float4 pp[HPW];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh)
          pp[hh] = *reinterpret_cast<const float4*>(&sm.p[wave][hh][t]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t vv =
              *reinterpret_cast<const uint32_t*>(&sm.v[(t + u) * kRowU16 + 2 * lane]);
          const float v0 = bf16_lo(vv), v1 = bf16_hi(vv);
#pragma unroll
          for (int hh = 0; hh < HPW; ++hh) {
            const float pu = u == 0 ? pp[hh].x : u == 1 ? pp[hh].y : u == 2 ? pp[hh].z : pp[hh].w;
            acc0[hh] = fmaf(pu, v0, acc0[hh]);
            acc1[hh] = fmaf(pu, v1, acc1[hh]);
          }
        }
      }
    }
  }

  // ---- partial (m, l, o) of this split, one slot per query head ----
  if (active) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      if (wave * HPW + hh >= G) continue;
      const int hq = g * G + wave * HPW + hh;
      const size_t slot = ((size_t)b * h_q + hq) * n_split + split;
      const float l = wave_sum(l_lane[hh]);
      store_coherent(&ws_o[slot * kD + 2 * lane], make_float2(acc0[hh], acc1[hh]));
      if (lane == 0) store_coherent(&ws_ml[slot * 2], make_float2(m_run[hh], l));
    }
  }

  // ---- the last split to finish merges all splits of this (b, g) ----
  wait_stores();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&counters[(size_t)b * h_kv + g], 1u,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    n_local_s = prev == (unsigned)(n_split - 1);
  }
  __syncthreads();
  if (!n_local_s) return;
  if (active) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      if (wave * HPW + hh >= G) continue;
      const size_t bh = (size_t)b * h_q + g * G + wave * HPW + hh;
      merge_head(ws_o, ws_ml, n_split, bh, out, lse, lane);
    }
  }
  if (tid == 0)
    __hip_atomic_store(&counters[(size_t)b * h_kv + g], 0u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

// Splits per (sequence, KV head): aim for ~4 workgroups per CU over the whole
// grid while keeping at least 2 blocks per split.
int decode_num_splits(int batch, int h_kv, int max_blocks) {
  const int pairs = batch * h_kv;
  int target = (1024 + pairs - 1) / pairs;
  int by_len = (max_blocks + 1) / 2;
  int n = target < by_len ? target : by_len;
  if (n < 1) n = 1;
  const int min_for_cap = (max_blocks + kMaxBps - 1) / kMaxBps;  // bps <= kMaxBps
  if (n < min_for_cap) n = min_for_cap;
  return n;
}

// Workspace: partial o [B, h_q, n_split, d], partial (m, l) [B, h_q, n_split],
// then one completion counter per (sequence, KV head).
size_t decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks) {
  const size_t ns = (size_t)decode_num_splits(batch, h_kv, max_blocks);
  return (size_t)batch * h_q * ns * ((size_t)d + 2) * sizeof(float) +
         (size_t)batch * h_kv * sizeof(unsigned);
}

hipError_t launch_decode(bool dense, const void* q, const void* k, const void* v,
                         const int32_t* seq_len, const int32_t* idx, const int32_t* count,
                         int k_max, int batch, int h_q, int h_kv, int l_cap, float sm_scale,
                         void* out, float* lse, void* ws, hipStream_t s) {
  const int max_blocks = dense ? l_cap / kBlk : k_max;
  const int n_split = decode_num_splits(batch, h_kv, max_blocks);
  const int bps = (max_blocks + n_split - 1) / n_split;
  float* ws_o = static_cast<float*>(ws);
  float* ws_ml = ws_o + (size_t)batch * h_q * n_split * kD;
  unsigned* counters = reinterpret_cast<unsigned*>(ws_ml + (size_t)batch * h_q * n_split * 2);
  auto o16 = static_cast<uint16_t*>(out);
  const float scale_log2 = sm_scale * kLog2e;
  const int G = h_q / h_kv;
  dim3 grid(n_split, h_kv, batch), block(kThreads);
  auto qq = static_cast<const uint16_t*>(q);
  auto kk = static_cast<const uint16_t*>(k);
  auto vv = static_cast<const uint16_t*>(v);
#define SPOT_DECODE_CASE(GG)                                                                   \
  if (G == GG) {                                                                               \
    if (dense)                                                                                 \
      hipLaunchKernelGGL((decode_split_kernel<GG, true>), grid, block, 0, s, qq, kk, vv,       \
                         seq_len, idx, count, k_max, h_q, h_kv, l_cap, scale_log2, bps,        \
                         n_split, ws_o, ws_ml, counters, o16, lse);                            \
    else                                                                                       \
      hipLaunchKernelGGL((decode_split_kernel<GG, false>), grid, block, 0, s, qq, kk, vv,      \
                         seq_len, idx, count, k_max, h_q, h_kv, l_cap, scale_log2, bps,        \
                         n_split, ws_o, ws_ml, counters, o16, lse);                            \
  }
  SPOT_DECODE_CASE(1)
  SPOT_DECODE_CASE(2)
  SPOT_DECODE_CASE(4)
  SPOT_DECODE_CASE(8)
#undef SPOT_DECODE_CASE
  return hipGetLastError();
}

}  // namespace spot
