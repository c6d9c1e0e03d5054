// Selector front end (paper Section 2.1; Appendix A for the rotary split):
//  * project_kernel: q^I = W_q h, k^I = W_k h and w = W_w h for rows of
//    hidden states, rotary position embedding on the first rope_dim dims of
//    every head (pairs (i, i + rope_dim/2) turned by pos * base^(-2i/rope_dim)),
//    q^I and w written out, k^I appended to the per-token selector cache at
//    (sequence, position);
//  * pool_kernel: the pooled selector key of a block, the mean of its
//    existing tokens' keys (FP32 pairwise sums over each 16-token quarter,
//    the quarters added in order, then BF16).
//
// Projection at decode is a matrix-vector product per sequence, bound by
// reading the weights (2 x 512 x d_model BF16 + the small W_w): each
// workgroup owns one task -- two output rows of W_q or W_k that the rotation
// pairs (or two neighbouring non-rotary rows), the first tasks also two rows
// of W_w -- and its 8 waves split d_model in 512-element chunks, so every
// weight byte is loaded once with all of a workgroup's loads in flight
// together, and the 512 workgroups are resident at once.  Hidden
// rows are re-read from L2 by every task.  Partial dots meet in LDS and are
// summed in a fixed order (deterministic); one lane per row finishes.  The
// rotation angle only needs the position and the pair's frequency (FP64,
// from the host), so it is formed while the weight loads are in flight.
//
// Pooled sums (pool_kernel, and project_kernel with POOL): each 16-token
// quarter of the block is summed as a pairwise tree -- (t0 + t1) + (t2 + t3)
// at the first two levels, then groups of 4 and 8 -- and the four quarter
// sums are added in order; absent tokens count as -0.0, the exact identity
// of addition.  With lane = token the tree is four DPP steps (adjacent lane,
// lane pair, half-row mirror, row mirror; addition is commutative, so every
// lane of a group holds the same sum).
#include <cmath>

#include "spot_internal.h"

namespace spot {
namespace {

constexpr int kProjWaves = 8;
constexpr int kMaxRopePairs = 64;

// base^(-2i / rope_dim) for the rotary pairs i < rope_dim / 2 (FP64).
struct RopeFreq {
  double f[kMaxRopePairs];
};

// Sum over each aligned group of 16 lanes as the pairwise tree above; every
// lane of the group ends with the group's sum.
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF,
                                                        false));
}
__device__ __forceinline__ float quarter_tree_sum(float x) {
  x = dpp_add<0xB1>(x);      // quad_perm [1, 0, 3, 2]: lane ^ 1
  x = dpp_add<0x4E>(x);      // quad_perm [2, 3, 0, 1]: lane ^ 2
  x = dpp_add<0x141>(x);     // row_half_mirror: the other group of 4 in the half row
  return dpp_add<0x140>(x);  // row_mirror: the other half of the row
}

// The same tree over 16 values held by one lane.
__device__ __forceinline__ float tree_sum16(const float (&t)[16]) {
  float a[8], b[4];
#pragma unroll
  for (int k = 0; k < 8; ++k) a[k] = t[2 * k] + t[2 * k + 1];
#pragma unroll
  for (int k = 0; k < 4; ++k) b[k] = a[2 * k] + a[2 * k + 1];
  return (b[0] + b[1]) + (b[2] + b[3]);
}

__device__ __forceinline__ float dot8_bf16(const u32x4& a, const u32x4& b, float c) {
  c = dot2_bf16(a[0], b[0], c);
  c = dot2_bf16(a[1], b[1], c);
  c = dot2_bf16(a[2], b[2], c);
  return dot2_bf16(a[3], b[3], c);
}

// Tasks: n_out pairs of W_q / W_k rows (n_out/2 each); the first ceil(h_s/2)
// tasks also take a pair of W_w rows, so that the grid (n_out = 512
// workgroups of 8 waves) fits the device at once.  Pair p of one head (d_s/2 pairs):
// p < rope_dim/2 -> dims (p, p + rope_dim/2), rotated; otherwise dims
// (rope_dim + 2(p - rope_dim/2), +1), not rotated.
// RP hidden rows per pass (4, 8 or 16): every pass loads its RP rows
// without branches (rows past the end re-read the last row, in cache), so
// all of a wave's loads are in flight together.
// POOL (one row per sequence): a W_k task also pools its two dims of the
// block each row's key lands in.  Wave w holds (row, dim) pairs w, w + 8, ..
// of the pass with lane = token of the block: the other tokens' values are
// loaded before the weights (and waited for only at the end), the new key's
// value joins its lane, and each pair is summed in pool_kernel's order
// exactly (16-token quarters in token order, then the quarters in order;
// tokens at or past the block's count hold -0.0, the exact identity of
// addition), so the pooled key is the one spot_selector_pool would compute
// after the append.
template <int RP, bool POOL>
__global__ __launch_bounds__(kProjWaves * 64) void project_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w_q,
    const uint16_t* __restrict__ w_k, const uint16_t* __restrict__ w_w,
    const int32_t* __restrict__ pos, int rows, int d_model, int h_s, int d_s, int rope_dim,
    RopeFreq freq, uint16_t* __restrict__ q_out, float* __restrict__ w_out,
    uint16_t* __restrict__ k_cache, int rows_per_seq, int l_cap,
    uint16_t* __restrict__ k_pool, const int32_t* __restrict__ seq_len) {
  __shared__ float part[kProjWaves][RP][4];   // [wave][row][row a, b, W_w c, d]
  __shared__ float pool_new[POOL ? RP : 1][2];   // the new key's value, [row][dim a/b]
  constexpr int kPairs = POOL ? (2 * RP + kProjWaves - 1) / kProjWaves : 1;   // per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_out = h_s * d_s;
  const int task = blockIdx.x;
  const int half = rope_dim / 2;

  // This task's two weight rows and where their results go (dims a, b of
  // q or k), plus W_w rows c, d for the first tasks.
  int dim_a = 0, dim_b = 0, head = 0;
  bool rotate = false;
  const int kind = task < n_out / 2 ? 0 : 1;       // 0: q, 1: k
  {
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
  }
  const uint16_t* wmat = kind == 0 ? w_q : w_k;
  const uint16_t* wa = wmat + (size_t)(head * d_s + dim_a) * d_model;
  const uint16_t* wb = wmat + (size_t)(head * d_s + dim_b) * d_model;
  const bool with_w = task < (h_s + 1) / 2;
  const int rc = 2 * task, rd = min(rc + 1, h_s - 1);
  const uint16_t* wc = w_w + (size_t)(with_w ? rc : 0) * d_model;
  const uint16_t* wd = w_w + (size_t)(with_w ? rd : 0) * d_model;
  for (int r0 = 0; r0 < rows; r0 += RP) {
    const int nr = min(RP, rows - r0);
    // 1. the finishing lane's (row r0 + lane) position, then the first
    // chunk's weight and hidden loads
    int p_row = 0;
    if (wave == 0 && lane < nr) p_row = pos[r0 + lane];
    int c = wave * 512 + lane * 8;
    bool have = c < d_model;
    u32x4 a, b, cw, dw, x[RP];
    auto load_chunk = [&]() {
      a = *reinterpret_cast<const u32x4*>(wa + c);
      b = *reinterpret_cast<const u32x4*>(wb + c);
      if (with_w) {
        cw = *reinterpret_cast<const u32x4*>(wc + c);
        dw = *reinterpret_cast<const u32x4*>(wd + c);
      }
#pragma unroll
      for (int i = 0; i < RP; ++i)
        x[i] = *reinterpret_cast<const u32x4*>(h + (size_t)min(r0 + i, rows - 1) * d_model + c);
    };
    if (have) load_chunk();
    // 2. the rotation of the finishing lane's row: angle pos * freq in FP64,
    // reduced to [-pi, pi] in FP64 (two-part 2 pi), sin and cos in FP32
    float s_rot = 0.f, c_rot = 1.f;
    if (rotate && wave == 0 && lane < nr) {
      const double theta = (double)p_row * freq.f[dim_a];
      const double k = rint(theta * 0.15915494309189535);   // 1 / (2 pi)
      double red = fma(-k, 6.283185307179586, theta);       // 2 pi, high part
      red = fma(-k, 2.4492935982947064e-16, red);           // 2 pi, low part
      sincosf((float)red, &s_rot, &c_rot);
    }
    // 3. for pooling, the block's other tokens: their waits come later (the
    // pooling positions are uniform scalar loads, whose wait does not hold
    // up the vector loads above)
    float pv[kPairs];   // POOL, W_k task: pair wave + 8m's value at token `lane`
#pragma unroll
    for (int m = 0; m < kPairs; ++m) {
      pv[m] = -0.f;
      const int pr = wave + kProjWaves * m, i = pr >> 1, sel = pr & 1;
      if (POOL && kind == 1 && i < nr) {
        const int r = r0 + i, p = pos[r];
        if (p >= 0 && p < l_cap && lane != p % kBlk)
          pv[m] = bf16_lo(k_cache[((size_t)r * l_cap + p / kBlk * kBlk + lane) * n_out +
                                  head * d_s + (sel ? dim_b : dim_a)]);
      }
    }
    // 4. the dot products, chunk by chunk
    float acc_a[RP], acc_b[RP], acc_c[RP], acc_d[RP];
#pragma unroll
    for (int i = 0; i < RP; ++i) acc_a[i] = acc_b[i] = acc_c[i] = acc_d[i] = 0.f;
    while (have) {
#pragma unroll
      for (int i = 0; i < RP; ++i) {
        acc_a[i] = dot8_bf16(a, x[i], acc_a[i]);
        acc_b[i] = dot8_bf16(b, x[i], acc_b[i]);
        if (with_w) {
          acc_c[i] = dot8_bf16(cw, x[i], acc_c[i]);
          acc_d[i] = dot8_bf16(dw, x[i], acc_d[i]);
        }
      }
      c += kProjWaves * 512;
      have = c < d_model;
      if (have) load_chunk();
    }
#pragma unroll
    for (int i = 0; i < RP; ++i) {
      if (i < nr) {
        const float sa = wave_sum(acc_a[i]), sb = wave_sum(acc_b[i]);
        if (lane == 0) {
          part[wave][i][0] = sa;
          part[wave][i][1] = sb;
        }
        if (with_w) {
          const float sc = wave_sum(acc_c[i]), sd = wave_sum(acc_d[i]);
          if (lane == 0) {
            part[wave][i][2] = sc;
            part[wave][i][3] = sd;
          }
        }
      }
    }
    __syncthreads();
    if (wave == 0 && lane < nr) {
      const int r = r0 + lane;
      float A = 0.f, B = 0.f, C = 0.f, D = 0.f;
#pragma unroll
      for (int w = 0; w < kProjWaves; ++w) {
        A += part[w][lane][0];
        B += part[w][lane][1];
        if (with_w) {
          C += part[w][lane][2];
          D += part[w][lane][3];
        }
      }
      if (with_w) {
        w_out[(size_t)r * h_s + rc] = C;
        if (rc + 1 < h_s) w_out[(size_t)r * h_s + rc + 1] = D;
      }
      {
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
          const uint16_t ha = f32_to_bf16_rne(A), hb = f32_to_bf16_rne(B);
          dst[head * d_s + dim_a] = ha;
          dst[head * d_s + dim_b] = hb;
          if (POOL && kind == 1) {
            pool_new[lane][0] = bf16_lo(ha);
            pool_new[lane][1] = bf16_lo(hb);
          }
        }
      }
    }
    __syncthreads();   // part[] is reused by the next pass; pool_new is complete
    if (POOL && kind == 1) {
#pragma unroll
      for (int m = 0; m < kPairs; ++m) {
        const int pr = wave + kProjWaves * m, i = pr >> 1, sel = pr & 1;
        if (i >= nr) continue;
        const int r = r0 + i, p = pos[r];
        int len = seq_len ? seq_len[r] : p + 1;
        len = len > l_cap ? l_cap : len;
        const int lo = p / kBlk * kBlk, n = min(len - lo, kBlk);
        if (p < 0 || p >= l_cap || n <= 0) continue;
        float x = lane == p % kBlk ? pool_new[i][sel] : pv[m];
        if (lane >= n) x = -0.f;
        x = quarter_tree_sum(x);
        float q4[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
          q4[qq] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), qq * 16));
        if (lane == 0) {
          const float v = ((q4[0] + q4[1]) + q4[2]) + q4[3];
          const int nblk = l_cap / kBlk;
          k_pool[((size_t)r * nblk + p / kBlk) * n_out + head * d_s + (sel ? dim_b : dim_a)] =
              f32_to_bf16_rne(v / (float)n);
        }
      }
    }
    if (POOL) __syncthreads();   // pool_new is reused by the next pass
  }
}

// One workgroup of 4 waves per (sequence, block to pool): block
// j = first_block[b] + y.  Wave w sums tokens [16w, 16w + 16) of the block
// (all 16 rows in flight), lane l elements 8l .. 8l+7, as the pairwise tree;
// the four partial sums are added in wave order, divided by the token count
// and rounded to BF16.
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
  for (int e = 0; e < 8; ++e) acc[e] = -0.f;
  if (t0 < n) {
    const uint16_t* src = k_tok + ((size_t)b * l_cap + lo) * 512 + lane * 8;
    u32x4 x[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
      x[u] = *reinterpret_cast<const u32x4*>(src + (size_t)min(t0 + u, n - 1) * 512);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float t[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const uint32_t wd = x[u][e >> 1];
        t[u] = t0 + u < n ? ((e & 1) ? bf16_hi(wd) : bf16_lo(wd)) : -0.f;
      }
      acc[e] = tree_sum16(t);
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
                                   void* k_pool, const int32_t* seq_len, hipStream_t s) {
  const int tasks = h_s * d_s;   // h_s * d_s / 2 >= ceil(h_s / 2) tasks carry the W_w rows
  if (rope_dim / 2 > kMaxRopePairs) return hipErrorInvalidValue;
  RopeFreq freq;
  const double lb = std::log2((double)rope_base);
  for (int i = 0; i < kMaxRopePairs; ++i)
    freq.f[i] = i < rope_dim / 2 ? std::exp2(-2.0 * i / rope_dim * lb) : 0.0;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(tasks), dim3(kProjWaves * 64), 0, s,
                       static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w_q),
                       static_cast<const uint16_t*>(w_k), static_cast<const uint16_t*>(w_w), pos,
                       rows, d_model, h_s, d_s, rope_dim, freq,
                       static_cast<uint16_t*>(q_out), w_out, static_cast<uint16_t*>(k_cache),
                       rows_per_seq, l_cap, static_cast<uint16_t*>(k_pool), seq_len);
  };
  if (k_pool) {   // one row per sequence (the caller checks rows_per_seq == 1)
    if (rows <= 4)
      go(project_kernel<4, true>);
    else if (rows <= 8)
      go(project_kernel<8, true>);
    else
      go(project_kernel<16, true>);
  } else if (rows <= 4) {
    go(project_kernel<4, false>);
  } else if (rows <= 8) {
    go(project_kernel<8, false>);
  } else {
    go(project_kernel<16, false>);
  }
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
