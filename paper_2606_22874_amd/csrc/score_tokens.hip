// Per-token selector scores reduced to one value per block (paper Section
// 2.3): the value of block b for query row r is the largest head-weighted
// ReLU score (Section 2.1) of r against the selector keys of b's visible
// tokens,
//     sbar[r, b] = max_{t in b, t < seq_len[r]} sum_h w[r,h] ReLU(q[r,h,:] . k[seq(r), t, h, :]).
//
// The per-token cache is a streamed read (1 KiB per BF16 token), so the kernel
// is bound by HBM and runs on the vector ALUs: with BF16 keys two wavefronts
// share a 64-token block, 32 tokens each, and meet in LDS (quantized keys: one
// wave per block); the loads are non-temporal (read
// once, they should not evict anything).  Each lane reads the same 16 bytes
// (8 elements) of every token row, so a load instruction moves one whole
// token row, coalesced.  Tokens are
// taken 8 at a time; the 8 per-lane partial dot products are folded across
// the LPH lanes of a head by a reduce-scatter (each butterfly step halves the
// tokens a lane keeps and exchanges the other half with its partner), which
// leaves every lane with the full head dot of one token in 7 exchanges where
// per-token reductions would need 8 x log2(LPH).  The ReLU and weight follow,
// then the head sum: inside a 16-lane row with one DPP move, across rows by a
// second reduce-scatter over the wave's groups, once per wave.  A wave
// maximum, then the maximum over the block's waves, gives the block value.
// Every exchange order is fixed, so the result is deterministic.
//
// Token loads past the last visible token re-read that token (in bounds, in
// cache); a duplicate of a visible token cannot change a maximum, so ragged
// blocks need no masking.
//
// Blocks of 16 tokens (SB = 16, the paper's selector block, Appendix A): the
// kernels walk the same 64-token spans and keep one maximum per 16-token
// block instead of one per span.  The folds above leave each lane with the
// scores of tokens from one 16-token block, so a block's value is the
// maximum over the lanes that hold its tokens (every copy of a score
// included, as in the 64-token maximum, so that both block sizes pick the
// largest of the same values); a 16-token block whose first token is not
// visible gets -inf (it may have been handed duplicates of an earlier
// block's last token).
#include "score_core.h"

namespace spot {
namespace {

constexpr int kTokWavesPerWG = 4;
constexpr int kTokTPW = 32;         // tokens per wave, BF16 keys (two waves per block)
// Quantized keys decode with more ALU work per byte, and a wave that owns a
// whole block (16 loads of 4 tokens in flight, 4-bit) overlaps its decode with
// the loads of the others better than two half-block waves: measured 26.5 vs
// 30.8 us (INT4) and 24.3 vs 28.4 us (MXFP4) over 4 x 131072 tokens.
constexpr int kTok8TPW = 64;        // tokens per wave, 8-bit keys (one wave per block)
constexpr int kTok4TPW = 64;        // tokens per wave, 4-bit keys (one wave per block)

// Butterfly exchange partner moves, all DPP inside a 16-lane row: the partner
// differs from the lane in the bit being folded (half-mirror 7 - i flips bit
// 2, mirror 15 - i flips bit 3, quad swaps flip bits 1 and 0); the other bits
// it flips are folded later, so each lane still sums every lane of its head.
template <int CTRL, int N>
__device__ __forceinline__ void fold_half(const float (&in)[2 * N], float (&out)[N], bool hi) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const float keep = hi ? in[i + N] : in[i];
    const float send = hi ? in[i] : in[i + N];
    out[i] = keep + dpp_f<CTRL>(send);
  }
}

// Same fold across 16-lane rows (partner lane ^ 16 or ^ 32).
template <int XOR, int N>
__device__ __forceinline__ void fold_half_rows(const float (&in)[2 * N], float (&out)[N],
                                               bool hi) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const float keep = hi ? in[i + N] : in[i];
    const float send = hi ? in[i] : in[i + N];
    out[i] = keep + __shfl_xor(send, XOR, 64);
  }
}

// Cross-row head sum of the G group values of a lane (G = 2, 4 or 8) and the
// maximum over them: after the folds over lane bits 4 and 5 each lane holds
// complete scores (G/4 of them, or one for G = 2), covering every token of
// the wave between the lanes.
template <int G>
__device__ __forceinline__ float rows_sum_max(const float (&y)[G], int lane) {
  if constexpr (G == 8) {
    float z[4], v[2];
    fold_half_rows<16, 4>(y, z, lane & 16);
    fold_half_rows<32, 2>(z, v, lane & 32);
    return fmaxf(v[0], v[1]);
  } else if constexpr (G == 4) {
    float z[2], v[1];
    fold_half_rows<16, 2>(y, z, lane & 16);
    fold_half_rows<32, 1>(z, v, lane & 32);
    return v[0];
  } else {
    float z[1];
    fold_half_rows<16, 1>(y, z, lane & 16);
    return z[0] + __shfl_xor(z[0], 32, 64);
  }
}

__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp_f<kDppQuadXor1>(v));
  v = fmaxf(v, dpp_f<kDppQuadXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  return fmaxf(v, dpp_f<kDppMirror>(v));
}

// Per-16-token-block maxima of a wave's G groups of 8 tokens after the head
// sums.  G = 4 (32 tokens): rows_sum_max leaves lane l with group
// 2 bit4(l) + bit5(l), so 16-token block bit4(l) of the wave; G = 8 (64
// tokens): it leaves the larger of groups 4 bit4 + 2 bit5 + {0, 1}, i.e.
// 16-token block 2 bit4 + bit5, the same for every lane of a 16-lane row.
// Returns that block's maximum in every lane.
template <int G>
__device__ __forceinline__ float sub16_max(const float (&y)[G], int lane) {
  float c = row_max16(rows_sum_max<G>(y, lane));
  if constexpr (G == 4) c = fmaxf(c, __shfl_xor(c, 32, 64));
  return c;
}
// Which of the wave's 16-token blocks lane l holds after sub16_max.
template <int G>
__device__ __forceinline__ int sub16_of_lane(int lane) {
  return G == 4 ? (lane >> 4) & 1 : 2 * ((lane >> 4) & 1) + (lane >> 5);
}

// TPW tokens per wavefront (16, 32 or 64): a block is shared by 64 / TPW
// waves of one workgroup, whose partial maxima meet in LDS.
//
// Launch order: work units u = (sequence, run of the 4 * TPW / 64 blocks of
// one workgroup) and the rows_per_seq query rows of a sequence.  Workgroup
// ids go round-robin over the 8 XCDs, so the rows that read the same keys
// are given ids 8 apart -- the same XCD, hence the same L2 -- and
// consecutive units alternate XCDs.
template <int KFMT, int LPH, int TPW, int SB>
__global__ __launch_bounds__(256) void score_tokens_kernel(
    const uint16_t* __restrict__ q_sel, const float* __restrict__ w,
    const uint8_t* __restrict__ k_tok, const uint8_t* __restrict__ k_scale, int n_seq,
    int rows_per_seq, int l_cap, int nblk, int runs, const int32_t* __restrict__ seq_len,
    float* __restrict__ scores) {
  constexpr int kHeads = 64 / LPH;
  constexpr int G = TPW / 8;                 // groups of 8 tokens per wave
  constexpr int WPB = 64 / TPW;              // waves per block
  constexpr int BPW = kTokWavesPerWG / WPB;  // blocks per workgroup
  static_assert(SB == 64 || (SB == 16 && (G == 4 || G == 8)),
                "16-token blocks need 32 or 64 tokens per wave");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gsize = 8 * rows_per_seq;
  const int id = blockIdx.x;
  const int unit = (id / gsize) * 8 + (id & 7);
  const int rr = (id % gsize) >> 3;
  if (unit >= n_seq * runs) return;
  const int seq = unit / runs;
  const int j = (unit % runs) * BPW + wave / WPB;   // 64-token span
  const int row = seq * rows_per_seq + rr;
  int len = seq_len ? seq_len[row] : l_cap;
  len = len < 0 ? 0 : (len > l_cap ? l_cap : len);
  const int t0 = j * 64 + (wave % WPB) * TPW;  // this wave's first token

  float m = -INFINITY;
  if (j < nblk && t0 < len) {
    const int tlim = min(j * 64 + 64, len) - 1;
    const size_t base = (size_t)seq * l_cap;
    const uint4 qraw = *reinterpret_cast<const uint4*>(q_sel + (size_t)row * 512 + lane * 8);
    float qf[8];
    qf[0] = bf16_lo(qraw.x); qf[1] = bf16_hi(qraw.x);
    qf[2] = bf16_lo(qraw.y); qf[3] = bf16_hi(qraw.y);
    qf[4] = bf16_lo(qraw.z); qf[5] = bf16_hi(qraw.z);
    qf[6] = bf16_lo(qraw.w); qf[7] = bf16_hi(qraw.w);
    const float wh = w[(size_t)row * kHeads + lane / LPH];

    // y[g]: the in-row head sum of this lane's token of group g (tokens
    // t0 + 8g .. t0 + 8g + 7; the lane holds token (LPH == 8 ? lane : lane >> 1) & 7).
    float y[G];
    KeyLoad<KFMT> key[2][8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      key[0][u].template load<true>(k_tok, k_scale, base + min(t0 + u, tlim), lane);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (g + 1 < G) {
#pragma unroll
        for (int u = 0; u < 8; ++u)
          key[(g + 1) & 1][u].template load<true>(k_tok, k_scale,
                                                  base + min(t0 + 8 * (g + 1) + u, tlim), lane);
      }
      float p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) p[u] = key[g & 1][u].dot(qraw, qf);
      float d;
      if constexpr (LPH == 8) {
        // Head lanes are lane bits 0..2.
        float a[4], c[2], e[1];
        fold_half<kDppHalfMirror, 4>(p, a, lane & 4);
        fold_half<kDppQuadXor2, 2>(a, c, lane & 2);
        fold_half<kDppQuadXor1, 1>(c, e, lane & 1);
        d = wh * fmaxf(e[0], 0.f);
        d += dpp_f<0x128>(d);  // row_ror:8 -- the other head of this 16-lane row
      } else {
        // Head lanes are lane bits 0..3.
        float a[4], c[2], e[1];
        fold_half<kDppMirror, 4>(p, a, lane & 8);
        fold_half<kDppHalfMirror, 2>(a, c, lane & 4);
        fold_half<kDppQuadXor2, 1>(c, e, lane & 2);
        const float h = e[0] + dpp_f<kDppQuadXor1>(e[0]);
        d = wh * fmaxf(h, 0.f);
      }
      y[g] = d;
    }
    if constexpr (SB == 64)
      m = wave_max(rows_sum_max<G>(y, lane));
    else
      m = sub16_max<G>(y, lane);
  }
  if constexpr (SB == 16) {
    // 16-token block J = the wave's first one + sub16_of_lane; one writer
    // lane per block (lanes 0, 16 (, 32, 48)).
    const int J = t0 / 16 + sub16_of_lane<G>(lane);
    if ((lane & 15) == 0 && (G == 8 || lane < 32) && j < nblk)
      scores[(size_t)row * nblk * 4 + J] = J * 16 < len ? m : -INFINITY;
    return;
  }
  float* dst = scores + (size_t)row * nblk + j;
  if constexpr (WPB == 1) {
    if (lane == 0 && j < nblk) *dst = m;
  } else {
    __shared__ float part[kTokWavesPerWG];
    if (lane == 0) part[wave] = m;
    __syncthreads();
    if (lane == 0 && wave % WPB == 0 && j < nblk) {
      float b = part[wave];
#pragma unroll
      for (int i = 1; i < WPB; ++i) b = fmaxf(b, part[wave + i]);
      *dst = b;
    }
  }
}

// 4-bit caches (INT4-g32, MXFP4-g32), 256 code bytes per token: a 16-byte
// load per lane moves four tokens, so lane l takes token slot l/16 and the
// 32-element scale group l%16 -- its 16 code bytes and its one scale.  The
// lane keeps the 32 query elements of its group in registers.  Per load:
// the group's dot, summed over the LG = d_s/32 lanes of a head (quad DPP
// moves), ReLU and w_h, then over the heads of the 16-lane row by DPP row
// rotations (rotating by 8, 4 (and 2) visits one lane of every head), which
// leaves every lane of the row with its token's score.  Tokens past the last
// visible one re-read it, as in score_tokens_kernel.
template <int KFMT, int LG, int TPW, int SB>
__global__ __launch_bounds__(256) void score_tokens4_kernel(
    const uint16_t* __restrict__ q_sel, const float* __restrict__ w,
    const uint8_t* __restrict__ k_tok, const uint8_t* __restrict__ k_scale, int n_seq,
    int rows_per_seq, int l_cap, int nblk, int runs, const int32_t* __restrict__ seq_len,
    float* __restrict__ scores) {
  constexpr int NL = TPW / 4;                // loads per wave (4 tokens each)
  constexpr int WPB = 64 / TPW;              // waves per block
  constexpr int BPW = kTokWavesPerWG / WPB;  // blocks per workgroup
  constexpr int kHeads = 16 / LG;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tq = lane >> 4, gi = lane & 15;
  const int gsize = 8 * rows_per_seq;
  const int id = blockIdx.x;
  const int unit = (id / gsize) * 8 + (id & 7);
  const int rr = (id % gsize) >> 3;
  if (unit >= n_seq * runs) return;
  const int seq = unit / runs;
  const int j = (unit % runs) * BPW + wave / WPB;
  const int row = seq * rows_per_seq + rr;
  int len = seq_len ? seq_len[row] : l_cap;
  len = len < 0 ? 0 : (len > l_cap ? l_cap : len);
  const int t0 = j * 64 + (wave % WPB) * TPW;
  static_assert(SB == 64 || (SB == 16 && TPW == 64), "16-token blocks: one wave per span");

  float m = -INFINITY;
  float ms[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};   // SB == 16
  if (j < nblk && t0 < len) {
    const int tlim = min(j * 64 + 64, len) - 1;
    const size_t base = (size_t)seq * l_cap;
    u32x4 code[NL];
    uint32_t sc[NL];
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const size_t t = base + min(t0 + 4 * u + tq, tlim);
      code[u] = ld<true, u32x4>(k_tok + t * 256 + gi * 16);
      if constexpr (KFMT == SPOT_KFMT_INT4_G32)
        sc[u] = ld<true, uint16_t>(k_scale + (t * 16 + gi) * 2);
      else
        sc[u] = ld<true, uint8_t>(k_scale + t * 16 + gi);
    }
    float qf[32];
    {
      const u32x4* qp = reinterpret_cast<const u32x4*>(q_sel + (size_t)row * 512 + gi * 32);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const u32x4 x = qp[c];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          qf[8 * c + 2 * i] = bf16_lo(x[i]);
          qf[8 * c + 2 * i + 1] = bf16_hi(x[i]);
        }
      }
    }
    const float wh = w[(size_t)row * kHeads + gi / LG];
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      float a = 0.f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t wd = code[u][c];
        if constexpr (KFMT == SPOT_KFMT_INT4_G32) {
          float v[8];
          int4_sixteenths(wd, v);
#pragma unroll
          for (int i = 0; i < 8; ++i) a = fmaf(qf[8 * c + i], v[i], a);
        } else {
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const f32x2 v = b == 0   ? __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd, 1.0f, 0)
                            : b == 1 ? __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd, 1.0f, 1)
                            : b == 2 ? __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd, 1.0f, 2)
                                     : __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd, 1.0f, 3);
            a = fmaf(qf[8 * c + 2 * b], v[0], a);
            a = fmaf(qf[8 * c + 2 * b + 1], v[1], a);
          }
        }
      }
      a *= KFMT == SPOT_KFMT_INT4_G32 ? 16.f * f16_to_f32((uint16_t)sc[u]) : e8m0_to_f32(sc[u]);
      a += dpp_f<kDppQuadXor1>(a);
      if constexpr (LG == 4) a += dpp_f<kDppQuadXor2>(a);
      float d = wh * fmaxf(a, 0.f);
      d += dpp_f<0x128>(d);                  // row_ror:8
      d += dpp_f<0x124>(d);                  // row_ror:4
      if constexpr (LG == 2) d += dpp_f<0x122>(d);   // row_ror:2
      if constexpr (SB == 64)
        m = fmaxf(m, d);
      else
        ms[u >> 2] = fmaxf(ms[u >> 2], d);   // loads 4s .. 4s+3: tokens 16s .. 16s+15
    }
    if constexpr (SB == 64) {
      m = wave_max(m);
    } else {
      // Row tq holds token slot tq's scores, but its lanes may hold them
      // rounded differently (the head sums may contract into fused
      // multiply-adds that start from a different lane's term), so each
      // block's maximum is taken over the whole wave, as wave_max does for
      // 64-token blocks: both then pick the largest of the same values.
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) ms[s4] = wave_max(ms[s4]);
    }
  }
  if constexpr (SB == 16) {
    if (lane < 4 && j < nblk) {
      const float v = lane == 0 ? ms[0] : lane == 1 ? ms[1] : lane == 2 ? ms[2] : ms[3];
      const int J = 4 * j + lane;
      scores[(size_t)row * nblk * 4 + J] = J * 16 < len ? v : -INFINITY;
    }
    return;
  }
  float* dst = scores + (size_t)row * nblk + j;
  if constexpr (WPB == 1) {
    if (lane == 0 && j < nblk) *dst = m;
  } else {
    __shared__ float part[kTokWavesPerWG];
    if (lane == 0) part[wave] = m;
    __syncthreads();
    if (lane == 0 && wave % WPB == 0 && j < nblk) {
      float b = part[wave];
#pragma unroll
      for (int i = 1; i < WPB; ++i) b = fmaxf(b, part[wave + i]);
      *dst = b;
    }
  }
}

// Grid of a per-token launch: (n_seq x runs of the workgroup's blocks),
// rounded up to a multiple of 8 units, times the query rows of a sequence.
template <int TPW>
int tok_runs(int nblk) {
  constexpr int kBlocksPerWG = kTokWavesPerWG * TPW / 64;
  return (nblk + kBlocksPerWG - 1) / kBlocksPerWG;
}
inline dim3 tok_grid(int n_seq, int runs, int rows_per_seq) {
  const long long units = (long long)n_seq * runs;
  return dim3((unsigned)(((units + 7) / 8) * 8 * rows_per_seq));
}

// nblk counts 64-token spans; with SB = 16 a row has 4 nblk output values.
template <int KFMT, int SB>
hipError_t launch_tokens_fmt(int lph, hipStream_t s, const uint16_t* q, const float* w,
                             const uint8_t* k, const uint8_t* ks, int n_seq, int rows_per_seq,
                             int l_cap, int nblk, const int32_t* seq_len, float* out) {
  if constexpr (KFMT == SPOT_KFMT_INT4_G32 || KFMT == SPOT_KFMT_MXFP4_G32) {
    // lanes per head of the 4-bit kernel: d_s / 32 = lph / 4
    const int runs = tok_runs<kTok4TPW>(nblk);
    const dim3 grid = tok_grid(n_seq, runs, rows_per_seq);
    if (lph == 8)
      hipLaunchKernelGGL((score_tokens4_kernel<KFMT, 2, kTok4TPW, SB>), grid, dim3(256), 0, s, q,
                         w, k, ks, n_seq, rows_per_seq, l_cap, nblk, runs, seq_len, out);
    else
      hipLaunchKernelGGL((score_tokens4_kernel<KFMT, 4, kTok4TPW, SB>), grid, dim3(256), 0, s, q,
                         w, k, ks, n_seq, rows_per_seq, l_cap, nblk, runs, seq_len, out);
    return hipGetLastError();
  }
  constexpr int TPW = KFMT == SPOT_KFMT_BF16 ? kTokTPW : kTok8TPW;
  const int runs = tok_runs<TPW>(nblk);
  const dim3 grid = tok_grid(n_seq, runs, rows_per_seq);
  if (lph == 8)
    hipLaunchKernelGGL((score_tokens_kernel<KFMT, 8, TPW, SB>), grid, dim3(256), 0, s, q, w, k,
                       ks, n_seq, rows_per_seq, l_cap, nblk, runs, seq_len, out);
  else
    hipLaunchKernelGGL((score_tokens_kernel<KFMT, 16, TPW, SB>), grid, dim3(256), 0, s, q, w, k,
                       ks, n_seq, rows_per_seq, l_cap, nblk, runs, seq_len, out);
  return hipGetLastError();
}

template <int SB>
hipError_t launch_tokens_sb(int kfmt, int lph, hipStream_t s, const uint16_t* q, const float* w,
                            const uint8_t* k, const uint8_t* ks, int n_seq, int rows_per_seq,
                            int l_cap, int nblk, const int32_t* seq_len, float* out) {
  switch (kfmt) {
    case SPOT_KFMT_BF16:
      return launch_tokens_fmt<SPOT_KFMT_BF16, SB>(lph, s, q, w, k, ks, n_seq, rows_per_seq,
                                                   l_cap, nblk, seq_len, out);
    case SPOT_KFMT_INT4_G32:
      return launch_tokens_fmt<SPOT_KFMT_INT4_G32, SB>(lph, s, q, w, k, ks, n_seq, rows_per_seq,
                                                       l_cap, nblk, seq_len, out);
    case SPOT_KFMT_INT8_G32:
      return launch_tokens_fmt<SPOT_KFMT_INT8_G32, SB>(lph, s, q, w, k, ks, n_seq, rows_per_seq,
                                                       l_cap, nblk, seq_len, out);
    case SPOT_KFMT_MXFP8_G32:
      return launch_tokens_fmt<SPOT_KFMT_MXFP8_G32, SB>(lph, s, q, w, k, ks, n_seq, rows_per_seq,
                                                        l_cap, nblk, seq_len, out);
    default:
      return launch_tokens_fmt<SPOT_KFMT_MXFP4_G32, SB>(lph, s, q, w, k, ks, n_seq, rows_per_seq,
                                                        l_cap, nblk, seq_len, out);
  }
}

}  // namespace

hipError_t launch_selector_score_tokens(const void* q_sel, const float* w, const void* k_tok,
                                        const void* k_scale, int kfmt, int n_seq,
                                        int rows_per_seq, int l_cap, int blk, int d_s,
                                        const int32_t* seq_len, float* scores, hipStream_t s) {
  const int nblk = l_cap / kBlk;   // 64-token spans
  const int lph = d_s / 8;
  auto q = static_cast<const uint16_t*>(q_sel);
  auto k = static_cast<const uint8_t*>(k_tok);
  auto ks = static_cast<const uint8_t*>(k_scale);
  if (blk == 16)
    return launch_tokens_sb<16>(kfmt, lph, s, q, w, k, ks, n_seq, rows_per_seq, l_cap, nblk,
                                seq_len, scores);
  return launch_tokens_sb<64>(kfmt, lph, s, q, w, k, ks, n_seq, rows_per_seq, l_cap, nblk,
                              seq_len, scores);
}

}  // namespace spot
