// Selector front end (paper Section 2.1; Appendix A for the rotary split):
//  * project_kernel: q^I = W_q h, k^I = W_k h and w = W_w h for rows of
//    hidden states, rotary position embedding on the first rope_dim dims of
//    every head (pairs (i, i + rope_dim/2) turned by pos * base^(-2i/rope_dim)),
//    q^I and w written out, k^I appended to the per-token selector cache at
//    (sequence, position);
//  * pool_kernel: the pooled selector key of a block, the mean of its
//    existing tokens' keys (FP32 sums over 16-token quarters in token order,
//    the quarters added in order, then BF16).
//
// Projection at decode is a matrix-vector product per sequence, bound by
// reading the weights (2 x 512 x d_model BF16 + the small W_w): each
// workgroup owns one task -- two output rows of W_q or W_k that the rotation
// pairs (or two neighbouring non-rotary rows), or two rows of W_w -- and its
// 8 waves split d_model in 512-element chunks, so every weight byte is
// loaded once with all of a workgroup's loads in flight together.  Hidden
// rows are re-read from L2 by every task.  Partial dots meet in LDS and are
// summed in a fixed order (deterministic); one lane per row finishes.
#include "spot_internal.h"

namespace spot {
namespace {

constexpr int kProjWaves = 8;

__device__ __forceinline__ float dot8_bf16(const u32x4& a, const u32x4& b, float c) {
  c = dot2_bf16(a[0], b[0], c);
  c = dot2_bf16(a[1], b[1], c);
  c = dot2_bf16(a[2], b[2], c);
  return dot2_bf16(a[3], b[3], c);
}

// Tasks: [0, n_out) pairs of W_q / W_k rows (n_out/2 each), then
// ceil(h_s / 2) pairs of W_w rows.  Pair p of one head (d_s/2 pairs):
// p < rope_dim/2 -> dims (p, p + rope_dim/2), rotated; otherwise dims
// (rope_dim + 2(p - rope_dim/2), +1), not rotated.
// RP hidden rows per pass (4, 8 or 16): every pass loads its RP rows
// without branches (rows past the end re-read the last row, in cache), so
// all of a wave's loads are in flight together.
template <int RP>
__global__ __launch_bounds__(kProjWaves * 64) void project_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w_q,
    const uint16_t* __restrict__ w_k, const uint16_t* __restrict__ w_w,
    const int32_t* __restrict__ pos, int rows, int d_model, int h_s, int d_s, int rope_dim,
    double rope_base, uint16_t* __restrict__ q_out, float* __restrict__ w_out,
    uint16_t* __restrict__ k_cache, int rows_per_seq, int l_cap) {
  __shared__ float part[kProjWaves][RP][2];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_out = h_s * d_s;
  const int task = blockIdx.x;
  const int half = rope_dim / 2;

  // This task's two weight rows and where their results go.
  int kind, ra, rb, dim_a = 0, dim_b = 0, head = 0;
  bool rotate = false;
  const uint16_t* wmat;
  if (task < n_out) {
    kind = task < n_out / 2 ? 0 : 1;               // 0: q, 1: k
    const int p = task % (n_out / 2);
    head = p / (d_s / 2);
    const int pp = p % (d_s / 2);
    if (pp < half) {
      dim_a = pp;
      dim_b = pp + half;
      rotate = true;
    } else {
      dim_a = rope_dim + 2 * (pp - half);
      dim_b = dim_a + 1;
    }
    ra = head * d_s + dim_a;
    rb = head * d_s + dim_b;
    wmat = kind == 0 ? w_q : w_k;
  } else {
    kind = 2;
    ra = 2 * (task - n_out);
    rb = min(ra + 1, h_s - 1);
    wmat = w_w;
  }
  const uint16_t* wa = wmat + (size_t)ra * d_model;
  const uint16_t* wb = wmat + (size_t)rb * d_model;
  // the pair's frequency (FP64), computed while the first loads are in flight
  const double freq = rotate ? pow(rope_base, -2.0 * dim_a / rope_dim) : 0.0;

  for (int r0 = 0; r0 < rows; r0 += RP) {
    const int nr = min(RP, rows - r0);
    // the finishing lane's (row r0 + lane) rotation, also ahead of the dots
    float c_rot = 1.f, s_rot = 0.f;
    int p_row = 0;
    if (wave == 0 && lane < nr && kind != 2) {
      p_row = pos[r0 + lane];
      if (rotate) {
        double sn, cs;
        sincos((double)p_row * freq, &sn, &cs);   // pos up to ~1e6 times freq <= 1
        c_rot = (float)cs;
        s_rot = (float)sn;
      }
    }
    float acc_a[RP], acc_b[RP];
#pragma unroll
    for (int i = 0; i < RP; ++i) acc_a[i] = acc_b[i] = 0.f;
    for (int c = wave * 512 + lane * 8; c < d_model; c += kProjWaves * 512) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(wa + c);
      const u32x4 b = *reinterpret_cast<const u32x4*>(wb + c);
      u32x4 x[RP];
#pragma unroll
      for (int i = 0; i < RP; ++i)
        x[i] = *reinterpret_cast<const u32x4*>(h + (size_t)min(r0 + i, rows - 1) * d_model + c);
#pragma unroll
      for (int i = 0; i < RP; ++i) {
        acc_a[i] = dot8_bf16(a, x[i], acc_a[i]);
        acc_b[i] = dot8_bf16(b, x[i], acc_b[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < RP; ++i) {
      if (i < nr) {
        const float sa = wave_sum(acc_a[i]), sb = wave_sum(acc_b[i]);
        if (lane == 0) {
          part[wave][i][0] = sa;
          part[wave][i][1] = sb;
        }
      }
    }
    __syncthreads();
    if (wave == 0 && lane < nr) {
      const int r = r0 + lane;
      float A = 0.f, B = 0.f;
#pragma unroll
      for (int w = 0; w < kProjWaves; ++w) {
        A += part[w][lane][0];
        B += part[w][lane][1];
      }
      if (kind == 2) {
        w_out[(size_t)r * h_s + ra] = A;
        if (ra + 1 < h_s) w_out[(size_t)r * h_s + ra + 1] = B;
      } else {
        const int p = p_row;
        if (rotate) {
          const float A2 = A * c_rot - B * s_rot;
          const float B2 = B * c_rot + A * s_rot;
          A = A2;
          B = B2;
        }
        uint16_t* dst;
        if (kind == 0) {
          dst = q_out + (size_t)r * n_out;
        } else {
          dst = (p >= 0 && p < l_cap)
                    ? k_cache + ((size_t)(r / rows_per_seq) * l_cap + p) * n_out
                    : nullptr;
        }
        if (dst) {
          dst[head * d_s + dim_a] = f32_to_bf16_rne(A);
          dst[head * d_s + dim_b] = f32_to_bf16_rne(B);
        }
      }
    }
    __syncthreads();   // part[] is reused by the next pass
  }
}

// One workgroup of 4 waves per (sequence, block to pool): block
// j = first_block[b] + y.  Wave w sums tokens [16w, 16w + 16) of the block
// (all 16 rows in flight), lane l elements 8l .. 8l+7, in token order; the
// four partial sums are added in wave order, divided by the token count and
// rounded to BF16.
__global__ __launch_bounds__(256) void pool_kernel(const uint16_t* __restrict__ k_tok,
                                                   uint16_t* __restrict__ k_pool, int l_cap,
                                                   const int32_t* __restrict__ seq_len,
                                                   const int32_t* __restrict__ first_block) {
  __shared__ float part[4][512];
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nblk = l_cap / kBlk;
  int len = seq_len ? seq_len[b] : l_cap;
  len = len < 0 ? 0 : (len > l_cap ? l_cap : len);
  const int j = (first_block ? first_block[b] : 0) + (int)blockIdx.y;
  const int lo = j * kBlk, hi = min(lo + kBlk, len);
  if (j < 0 || j >= nblk || hi <= lo) return;
  const int n = hi - lo;
  const int t0 = wave * 16;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  if (t0 < n) {
    const uint16_t* src = k_tok + ((size_t)b * l_cap + lo) * 512 + lane * 8;
    u32x4 x[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
      x[u] = *reinterpret_cast<const u32x4*>(src + (size_t)min(t0 + u, n - 1) * 512);
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (t0 + u < n) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[2 * i] += bf16_lo(x[u][i]);
          acc[2 * i + 1] += bf16_hi(x[u][i]);
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[wave][lane * 8 + e] = acc[e];
  __syncthreads();
  if (wave == 0) {
    const float cnt = (float)n;
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int e = lane * 8 + 2 * i + k;
        v[k] = ((part[0][e] + part[1][e]) + part[2][e]) + part[3][e];
      }
      o[i] = (uint32_t)f32_to_bf16_rne(v[0] / cnt) | ((uint32_t)f32_to_bf16_rne(v[1] / cnt) << 16);
    }
    *reinterpret_cast<u32x4*>(k_pool + ((size_t)b * nblk + j) * 512 + lane * 8) = o;
  }
}

}  // namespace

hipError_t launch_selector_project(const void* h, const void* w_q, const void* w_k,
                                   const void* w_w, const int32_t* pos, int rows, int d_model,
                                   int h_s, int d_s, int rope_dim, float rope_base, void* q_out,
                                   float* w_out, void* k_cache, int rows_per_seq, int l_cap,
                                   hipStream_t s) {
  const int tasks = h_s * d_s + (h_s + 1) / 2;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(tasks), dim3(kProjWaves * 64), 0, s,
                       static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w_q),
                       static_cast<const uint16_t*>(w_k), static_cast<const uint16_t*>(w_w), pos,
                       rows, d_model, h_s, d_s, rope_dim, (double)rope_base,
                       static_cast<uint16_t*>(q_out), w_out, static_cast<uint16_t*>(k_cache),
                       rows_per_seq, l_cap);
  };
  if (rows <= 4)
    go(project_kernel<4>);
  else if (rows <= 8)
    go(project_kernel<8>);
  else
    go(project_kernel<16>);
  return hipGetLastError();
}

hipError_t launch_selector_pool(const void* k_tok, void* k_pool, int n_seq, int l_cap,
                                const int32_t* seq_len, const int32_t* first_block,
                                int max_blocks, hipStream_t s) {
  hipLaunchKernelGGL(pool_kernel, dim3(n_seq, max_blocks), dim3(256), 0, s,
                     static_cast<const uint16_t*>(k_tok), static_cast<uint16_t*>(k_pool), l_cap,
                     seq_len, first_block);
  return hipGetLastError();
}

}  // namespace spot
