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
// Each split writes an unnormalised partial (m, l, o); a merge kernel
// combines the splits with log-sum-exp weights and rounds to BF16.
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

// HPW = query heads per wave (G = 4 * HPW, or G < 4 with idle waves).
template <int G, bool DENSE>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ seq_len,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ count, int k_max, int h_q,
    int h_kv, int l_cap, float scale_log2, int bps, int n_split, float* __restrict__ ws_o,
    float* __restrict__ ws_ml) {
  constexpr int HPW = G > 4 ? G / 4 : 1;
  __shared__ DecodeSmem sm;
  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool active = wave * HPW < G;

  const int sl = min(seq_len[b], l_cap);
  const int nb_valid = (sl + kBlk - 1) / kBlk;
  const int n_entries = DENSE ? nb_valid : min(count[b], k_max);
  const int e0 = split * bps;
  const int e1 = min(e0 + bps, n_entries);

  // Block list of this split (sparse); invalid ids become -1 (skipped).
  if (!DENSE) {
    for (int i = tid; i < e1 - e0; i += kThreads) {
      const int j = idx[(size_t)b * k_max + e0 + i];
      sm.ids[i] = (j >= 0 && j < nb_valid) ? j : -1;
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

  const size_t head_base = ((size_t)b * h_kv + g) * (size_t)l_cap * kD;
  const uint16_t* kh = k + head_base;
  const uint16_t* vh = v + head_base;

  auto block_id = [&](int e) -> int { return DENSE ? e : sm.ids[e - e0]; };

  // Register staging for one block: 4 x 16 B of K and of V per thread.
  uint4 kr[4], vr[4];
  auto issue = [&](int blk) {
    const size_t base = (size_t)blk * kBlk * kD;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int c = p * kThreads + tid;  // 16-byte chunk of the 16 KiB tile
      const size_t off = base + (size_t)(c >> 4) * kD + (c & 15) * 8;
      kr[p] = *reinterpret_cast<const uint4*>(kh + off);
      vr[p] = *reinterpret_cast<const uint4*>(vh + off);
    }
  };

  int e = e0;
  while (e < e1 && block_id(e) < 0) ++e;
  if (e < e1) issue(block_id(e));

  while (e < e1) {
    const int blk = block_id(e);
    int en = e + 1;
    while (en < e1 && block_id(en) < 0) ++en;

    __syncthreads();  // previous block's LDS reads are done
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int c = p * kThreads + tid;
      *reinterpret_cast<uint4*>(&sm.k[(c >> 4) * kRowU16 + (c & 15) * 8]) = kr[p];
      *reinterpret_cast<uint4*>(&sm.v[(c >> 4) * kRowU16 + (c & 15) * 8]) = vr[p];
    }
    __syncthreads();
    if (en < e1) issue(block_id(en));  // next block in flight during compute

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
        const float m_new = fmaxf(m_run[hh], wave_max(x));
        // m_new is finite: every block in the list has >= 1 valid token.
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
        for (int hh = 0; hh < HPW; ++hh) pp[hh] = *reinterpret_cast<const float4*>(&sm.p[wave][hh][t]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t vv = *reinterpret_cast<const uint32_t*>(&sm.v[(t + u) * kRowU16 + 2 * lane]);
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
    e = en;
  }

  if (active) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      if (wave * HPW + hh >= G) continue;
      const int hq = g * G + wave * HPW + hh;
      const size_t slot = ((size_t)b * h_q + hq) * n_split + split;
      const float l = wave_sum(l_lane[hh]);
      *reinterpret_cast<float2*>(&ws_o[slot * kD + 2 * lane]) = make_float2(acc0[hh], acc1[hh]);
      if (lane == 0) *reinterpret_cast<float2*>(&ws_ml[slot * 2]) = make_float2(m_run[hh], l);
    }
  }
}

// One wave per (sequence, query head): log-sum-exp merge of the splits.
__global__ __launch_bounds__(64) void decode_merge_kernel(const float* __restrict__ ws_o,
                                                          const float* __restrict__ ws_ml,
                                                          int n_split, uint16_t* __restrict__ out,
                                                          float* __restrict__ lse) {
  const int bh = blockIdx.x, lane = threadIdx.x;
  const float* ml = ws_ml + (size_t)bh * n_split * 2;
  float M = -INFINITY;
  for (int s = 0; s < n_split; ++s)
    if (ml[2 * s + 1] > 0.f) M = fmaxf(M, ml[2 * s]);
  float L = 0.f, o0 = 0.f, o1 = 0.f;
  if (M > -INFINITY) {
    for (int s = 0; s < n_split; ++s) {
      const float l = ml[2 * s + 1];
      if (!(l > 0.f)) continue;
      const float wgt = exp2f(ml[2 * s] - M);
      L = fmaf(l, wgt, L);
      const float2 o = *reinterpret_cast<const float2*>(&ws_o[((size_t)bh * n_split + s) * kD + 2 * lane]);
      o0 = fmaf(o.x, wgt, o0);
      o1 = fmaf(o.y, wgt, o1);
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const uint32_t packed = (uint32_t)f32_to_bf16_rne(o0 * inv) |
                          ((uint32_t)f32_to_bf16_rne(o1 * inv) << 16);
  *reinterpret_cast<uint32_t*>(&out[(size_t)bh * kD + 2 * lane]) = packed;
  if (lse && lane == 0) lse[bh] = L > 0.f ? (M + log2f(L)) * 0.6931471805599453f : -INFINITY;
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

size_t decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks) {
  const size_t ns = (size_t)decode_num_splits(batch, h_kv, max_blocks);
  return (size_t)batch * h_q * ns * ((size_t)d + 2) * sizeof(float);
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
                         n_split, ws_o, ws_ml);                                                \
    else                                                                                       \
      hipLaunchKernelGGL((decode_split_kernel<GG, false>), grid, block, 0, s, qq, kk, vv,      \
                         seq_len, idx, count, k_max, h_q, h_kv, l_cap, scale_log2, bps,        \
                         n_split, ws_o, ws_ml);                                                \
  }
  SPOT_DECODE_CASE(1)
  SPOT_DECODE_CASE(2)
  SPOT_DECODE_CASE(4)
  SPOT_DECODE_CASE(8)
#undef SPOT_DECODE_CASE
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(decode_merge_kernel, dim3(batch * h_q), dim3(64), 0, s, ws_o, ws_ml,
                     n_split, static_cast<uint16_t*>(out), lse);
  return hipGetLastError();
}

}  // namespace spot
