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
// of W_w -- and its 4 waves split d_model in passes of 4 x CH chunks of 512
// elements (one pass at d_model = 4096), every chunk's weight and hidden
// loads issued before the first product, so every weight byte is loaded once
// with all of a wave's loads in flight together, and the 512 workgroups are
// resident at once (a grid row per pass of RP hidden rows).  Hidden rows are
// re-read from L2 by every task.  Partial
// dots meet in LDS and are summed in a fixed order (deterministic); one lane
// per row finishes.  The rows' positions (and lengths) are the first loads
// of a pass, so that nothing after them waits for a late scalar load; the
// rotation angle only needs the position and the pair's frequency (FP64,
// from the host), so it is formed while the weight loads are in flight.
// (Against 8 waves of one chunk, with the positions read where they are
// used and loads behind branches, this takes 3.8 instead of 4.9 us for the
// B = 4, d_model = 4096 decode projection, and 4.5 instead of 6.0 us with
// the pooling, replayed in a HIP graph.)
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

constexpr int kProjWaves = 4;
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
// workgroups of 4 waves) fits the device at once.  Pair p of one head (d_s/2 pairs):
// p < rope_dim/2 -> dims (p, p + rope_dim/2), rotated; otherwise dims
// (rope_dim + 2(p - rope_dim/2), +1), not rotated.
// RP hidden rows per row pass (4, 8 or 16): every pass loads its RP rows
// without branches (rows past the end re-read the last row, in cache), so
// all of a wave's loads are in flight together.  CH chunks of 512 elements
// per wave and d pass; lanes past d_model load nothing and add zeros.
// POOL (one row per sequence): a W_k task also pools its two dims of the
// block each row's key lands in.  Wave w gathers rows w, w + 4, .. of the
// pass, both dims (one 4-byte load when they are neighbours), with lane =
// token of the block: the loads go out after the first d pass's weight
// loads and are waited for only at the end; the new key's value joins its
// lane, and each dim is summed in pool_kernel's order exactly (16-token
// quarters in token order, then the quarters in order; tokens at or past
// the block's count hold -0.0, the exact identity of addition), so the
// pooled key is the one spot_selector_pool would compute after the append.
template <int RP, int CH, bool POOL>
__global__ __launch_bounds__(kProjWaves * 64) void project_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w_q,
    const uint16_t* __restrict__ w_k, const uint16_t* __restrict__ w_w,
    const int32_t* __restrict__ pos, int rows, int d_model, int h_s, int d_s, int rope_dim,
    RopeFreq freq, uint16_t* __restrict__ q_out, float* __restrict__ w_out,
    uint16_t* __restrict__ k_cache, int rows_per_seq, int l_cap,
    uint16_t* __restrict__ k_pool, const int32_t* __restrict__ seq_len, int row_base) {
  static_assert(RP >= kProjWaves && (RP & (RP - 1)) == 0, "RP: a power of two >= the waves");
  __shared__ float part[kProjWaves][RP][4];   // [wave][row][row a, b, W_w c, d]
  __shared__ float pool_new[POOL ? RP : 1][2];   // the new key's value, [row][dim a/b]
  constexpr int kRows = POOL ? RP / kProjWaves : 1;   // rows gathered per wave
  constexpr int kPass = kProjWaves * 512 * CH;        // d elements per pass
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Row pass blockIdx.y (RP rows from row_base + RP * blockIdx.y).
  // 1. every lane: position and length (the position again without
  // seq_len) of row r0 + lane % RP (the last row for lanes past the end),
  // the first loads; lane r of wave 0 finishes row r0 + r, wave w gathers
  // rows r0 + w + 4m.  Every load is unconditional (addresses clamped into
  // their buffers, unused values masked where they are used), so that no
  // branch join makes a wave wait for a load before it issues the next ones.
  const int r0 = row_base + (int)blockIdx.y * RP;
  const int nr = min(RP, rows - r0);
  const int lr = r0 + min(lane & (RP - 1), nr - 1);
  const int pos_l = pos[lr];
  const int len_l = (seq_len ? seq_len : pos)[lr];

  // This task's two weight rows and where their results go (dims a, b of
  // q or k), plus W_w rows c, d for the first tasks.  n_out (512) and the
  // d_s / 2 pairs of a head are powers of two.
  const int n_out = h_s * d_s;
  const int task = blockIdx.x;
  const int half = rope_dim / 2;
  // 0: q, 1: k; with pooling the k tasks, which also gather and pool, are
  // dispatched first
  const int kind = (task < (n_out >> 1)) == POOL ? 1 : 0;
  const int p_task = task & ((n_out >> 1) - 1);
  const int head = p_task >> __builtin_ctz(d_s >> 1);
  const int pp = p_task & ((d_s >> 1) - 1);
  const bool rotate = pp < half;
  const int dim_a = rotate ? pp : rope_dim + 2 * (pp - half);
  const int dim_b = rotate ? pp + half : dim_a + 1;
  const bool pool_task = POOL && kind == 1;
  const uint16_t* wmat = kind == 0 ? w_q : w_k;
  const uint16_t* wa = wmat + (size_t)(head * d_s + dim_a) * d_model;
  const uint16_t* wb = wmat + (size_t)(head * d_s + dim_b) * d_model;
  // W_w rows ride on the first q tasks (with pooling, the k tasks are the
  // heavier ones)
  const int wt = task - (POOL ? n_out >> 1 : 0);
  const bool with_w = wt >= 0 && wt < (h_s + 1) / 2;
  const int rc = with_w ? 2 * wt : 0, rd = min(rc + 1, h_s - 1);
  const uint16_t* wc = w_w + (size_t)(with_w ? rc : 0) * d_model;
  const uint16_t* wd = w_w + (size_t)(with_w ? rd : 0) * d_model;
  {
    // the finishing lane's sequence
    const int seq_l = rows_per_seq == 1 ? lr : lr / rows_per_seq;
    float acc_a[RP], acc_b[RP], acc_c[RP], acc_d[RP];
#pragma unroll
    for (int i = 0; i < RP; ++i) acc_a[i] = acc_b[i] = acc_c[i] = acc_d[i] = 0.f;
    uint16_t pga[kRows], pgb[kRows];   // POOL, W_k task: row w + 4m's dims at token `lane`
    float s_rot = 0.f, c_rot = 1.f;
    for (int c0 = 0; c0 < d_model; c0 += kPass) {
      // 2. this pass's weight and hidden loads, all in flight together
      // (chunks past d_model re-read the last 8 elements and are skipped)
      u32x4 a[CH], b[CH], cw[CH], dw[CH], x[CH][RP];
#pragma unroll
      for (int cc = 0; cc < CH; ++cc) {
        const int c = min(c0 + (cc * kProjWaves + wave) * 512 + lane * 8, d_model - 8);
        a[cc] = *reinterpret_cast<const u32x4*>(wa + c);
        b[cc] = *reinterpret_cast<const u32x4*>(wb + c);
        if (with_w) {
          cw[cc] = *reinterpret_cast<const u32x4*>(wc + c);
          dw[cc] = *reinterpret_cast<const u32x4*>(wd + c);
        }
#pragma unroll
        for (int i = 0; i < RP; ++i)
          x[cc][i] = *reinterpret_cast<const u32x4*>(
              h + (size_t)min(r0 + i, rows - 1) * d_model + c);
      }
      if (c0 == 0) {
        // 3. pooling: the block's tokens at both dims (waited for at the
        // end); tasks and rows without pooling read one cache word
#pragma unroll
        for (int m = 0; m < kRows; ++m) {
          const int i = wave + kProjWaves * m;
          const int p = __builtin_amdgcn_readlane(pos_l, min(i, nr - 1));
          const bool live = pool_task && i < nr && p >= 0 && p < l_cap;
          const uint16_t* src =
              live ? k_cache + ((size_t)(r0 + i) * l_cap + p / kBlk * kBlk + lane) * n_out +
                         head * d_s
                   : k_cache;
          pga[m] = src[dim_a];
          pgb[m] = src[dim_b];
        }
        // 4. the rotation of the finishing lane's row: angle pos * freq in
        // FP64, reduced to [-pi, pi] in FP64 (two-part 2 pi), sin and cos in
        // FP32
        if (rotate && wave == 0 && lane < nr) {
          const double theta = (double)pos_l * freq.f[dim_a];
          const double k = rint(theta * 0.15915494309189535);   // 1 / (2 pi)
          double red = fma(-k, 6.283185307179586, theta);       // 2 pi, high part
          red = fma(-k, 2.4492935982947064e-16, red);           // 2 pi, low part
          sincosf((float)red, &s_rot, &c_rot);
        }
      }
      // 5. the dot products of this pass
#pragma unroll
      for (int cc = 0; cc < CH; ++cc) {
        if (c0 + (cc * kProjWaves + wave) * 512 + lane * 8 >= d_model) continue;
#pragma unroll
        for (int i = 0; i < RP; ++i) {
          acc_a[i] = dot8_bf16(a[cc], x[cc][i], acc_a[i]);
          acc_b[i] = dot8_bf16(b[cc], x[cc][i], acc_b[i]);
          if (with_w) {
            acc_c[i] = dot8_bf16(cw[cc], x[cc][i], acc_c[i]);
            acc_d[i] = dot8_bf16(dw[cc], x[cc][i], acc_d[i]);
          }
        }
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
        const int p = pos_l;
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
                    ? k_cache + ((size_t)seq_l * l_cap + p) * n_out
                    : nullptr;
        }
        if (dst) {
          const uint16_t ha = f32_to_bf16_rne(A), hb = f32_to_bf16_rne(B);
          dst[head * d_s + dim_a] = ha;
          dst[head * d_s + dim_b] = hb;
          if (pool_task) {
            pool_new[lane][0] = bf16_lo(ha);
            pool_new[lane][1] = bf16_lo(hb);
          }
        }
      }
    }
    if (pool_task) __syncthreads();   // pool_new is complete
    if (pool_task) {
#pragma unroll
      for (int m = 0; m < kRows; ++m) {
        const int i = wave + kProjWaves * m;
        if (i >= nr) continue;
        const int p = __builtin_amdgcn_readlane(pos_l, i);
        int len = seq_len ? __builtin_amdgcn_readlane(len_l, i) : p + 1;
        len = len > l_cap ? l_cap : len;
        const int lo = p / kBlk * kBlk, n = min(len - lo, kBlk);
        if (p < 0 || p >= l_cap || n <= 0) continue;
        const int r = r0 + i;
#pragma unroll
        for (int sel = 0; sel < 2; ++sel) {
          float x = lane == p % kBlk ? pool_new[i][sel] : bf16_lo(sel ? pgb[m] : pga[m]);
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
    }
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
  const int rp = rows <= 4 ? 4 : (rows <= 8 ? 8 : 16);
  const int passes = (rows + rp - 1) / rp;
  // one row pass per workgroup row; more than 65535 passes take more launches
  for (int p0 = 0; p0 < passes; p0 += 65535) {
    const dim3 grid(tasks, passes - p0 < 65535 ? passes - p0 : 65535);
    auto go = [&](auto kern) {
      hipLaunchKernelGGL(kern, grid, dim3(kProjWaves * 64), 0, s,
                         static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w_q),
                         static_cast<const uint16_t*>(w_k), static_cast<const uint16_t*>(w_w),
                         pos, rows, d_model, h_s, d_s, rope_dim, freq,
                         static_cast<uint16_t*>(q_out), w_out, static_cast<uint16_t*>(k_cache),
                         rows_per_seq, l_cap, static_cast<uint16_t*>(k_pool), seq_len, p0 * rp);
    };
    if (k_pool) {   // one row per sequence (the caller checks rows_per_seq == 1)
      if (rp == 4)
        go(project_kernel<4, 2, true>);
      else if (rp == 8)
        go(project_kernel<8, 2, true>);
      else
        go(project_kernel<16, 1, true>);
    } else if (rp == 4) {
      go(project_kernel<4, 2, false>);
    } else if (rp == 8) {
      go(project_kernel<8, 2, false>);
    } else {
      go(project_kernel<16, 1, false>);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
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
