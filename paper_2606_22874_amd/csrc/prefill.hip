// Block-sparse causal prefill attention on the matrix cores (gfx950).
//
// Work unit: one workgroup per (sequence, query block, KV head, head chunk).
// The chunk holds up to four of the query heads that share the KV head; each
// head is split over two waves of 32 query rows.  Every selected key block of
// the query block (its ids shared by all heads, Section 2.1) is staged once
// in LDS and consumed by all waves of the workgroup, so the K/V bytes are
// fetched once per chunk rather than once per head.
//
// Per wave and key block (64 keys x 32 queries, head dim 128) the math runs
// transposed so that no score ever leaves the registers:
//   S^T = K Q^T       16 v_mfma_f32_16x16x32_bf16 tiles  (K from LDS as the
//                     A operand, Q^T held in VGPRs as the B operand)
//   online softmax    per query = per lane column; column max over the four
//                     16-lane groups with two cross-lane exchanges
//   O^T += V^T P^T    P^T goes straight from the accumulators to the B
//                     operand (keys permuted consistently on both operands);
//                     V^T comes from LDS through the transposing read
//                     ds_read_b64_tr_b16.
// The C layout of a 16x16 tile gives lane l the rows 4(l/16)..4(l/16)+3 of
// column l%16; the A/B layout gives lane l the 8 consecutive k entries
// 8(l/16).. of row (A) or column (B) l%16.
//
// K/V tiles are copied global -> LDS with 16-byte direct loads
// (global_load_lds_dwordx4): each wave instruction fills 1 KiB of LDS in lane
// order, so the tile keeps 256-byte rows and bank conflicts are avoided by
// XOR-swizzling the 16-byte chunks of a row instead of padding it.  Two tile
// buffers alternate; the next tile's loads fly while the current one is used.
#include "spot_internal.h"

namespace spot {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kD = 128;
constexpr int kRowBytes = kD * 2;               // 256
constexpr int kTileBytes = kBlk * kRowBytes;    // 16 KiB
constexpr int kPrefillMaxIds = 4096;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

struct PrefillSmem {
  alignas(16) unsigned char k[2][kTileBytes];
  alignas(16) unsigned char v[2][kTileBytes];
  int ids[kPrefillMaxIds];
  int n_local;
};

// Physical 16-byte chunk of logical chunk c in tile row r.  K is read as 16
// rows x one chunk per quarter wave, so rows must map one chunk to distinct
// bank groups (c ^ r%16).  V is read 8 bytes per lane over 8 rows x two
// adjacent chunks per half wave ((c ^ 2(r%8)) keeps the pair adjacent).
__device__ __forceinline__ int swz_k(int r, int c) { return c ^ (r & 15); }
__device__ __forceinline__ int swz_v(int r, int c) { return c ^ ((r & 7) << 1); }

typedef __attribute__((address_space(3))) void lds_void;

// Stage one 64 x 128 BF16 tile (16 KiB, contiguous in global memory) in LDS.
template <int W, bool IS_K>
__device__ __forceinline__ void stage_tile(const uint16_t* __restrict__ src, unsigned char* dst,
                                           int wave, int lane) {
#pragma unroll
  for (int u = 0; u < 16 / W; ++u) {
    const int base = (u * W + wave) * kWave;  // first physical chunk of this wave's KiB
    const int p = base + lane;
    const int r = p >> 4, pc = p & 15;
    const int lc = IS_K ? swz_k(r, pc) : swz_v(r, pc);
    __builtin_amdgcn_global_load_lds(src + r * kD + lc * 8, (lds_void*)(dst + base * 16), 16, 0,
                                     0);
  }
}

__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ float xor_f(float x, int m) { return __shfl_xor(x, m, 64); }

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return (uint32_t)f32_to_bf16_rne(a) | ((uint32_t)f32_to_bf16_rne(b) << 16);
}

template <int W>
__global__ __launch_bounds__(64 * W) void prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, int L, const int32_t* __restrict__ idx,
    const int32_t* __restrict__ count, int k_max, int batch, int h_q, int h_kv, int n_chunk,
    int n_pairs, float c, uint16_t* __restrict__ out, float* __restrict__ lse) {
  __shared__ PrefillSmem sm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Workgroups of one (sequence, query block, KV head) pair differ by a
  // multiple of 8 in their id, so they are dispatched to the same XCD and
  // share its L2; pairs are ordered heaviest query block first.
  const int inner = blockIdx.x & 7, rest = blockIdx.x >> 3;
  const int chunk = rest % n_chunk, pair = (rest / n_chunk) * 8 + inner;
  if (pair >= n_pairs) return;
  const int nqb = L / kBlk;
  const int g = pair % h_kv, rank = pair / h_kv;
  const int b = rank % batch, qb = nqb - 1 - rank / batch;
  const int row = b * nqb + qb;
  const int h = g * (h_q / h_kv) + chunk * (W / 2) + (wave >> 1);
  const int qoff = (wave & 1) * 32;
  const int G = lane >> 4, r16 = lane & 15;

  // Selected key blocks that exist for this query block (0 <= id <= qb), in
  // list order, compacted into LDS.
  if (wave == 0) {
    const int n_e = min(max(count[row], 0), k_max);
    const int32_t* ids_row = idx + (int64_t)row * k_max;
    int n = 0;
    for (int base = 0; base < n_e; base += kWave) {
      const int e = base + lane;
      const int j = e < n_e ? ids_row[e] : -1;
      const bool ok = j >= 0 && j <= qb;
      const uint64_t m = __ballot(ok);
      const int pos = n + __popcll(m & ((1ull << lane) - 1ull));
      if (ok && pos < kPrefillMaxIds) sm.ids[pos] = j;
      n += __popcll(m);
    }
    if (lane == 0) sm.n_local = min(n, kPrefillMaxIds);
  }

  // Q^T fragments (B operand): lane holds Q[row 16 qt + l%16][32 ks + 8(l/16) ..+7].
  const uint16_t* qh = q + ((int64_t)(b * h_q + h) * L + qb * kBlk + qoff) * kD;
  bf16x8 qf[2][4];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qf[qt][ks] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(qh + (qt * 16 + r16) * kD + ks * 32 + 8 * G));

  const uint16_t* kg = k + (int64_t)(b * h_kv + g) * L * kD;
  const uint16_t* vg = v + (int64_t)(b * h_kv + g) * L * kD;

  f32x4 o[2][8];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};

  __syncthreads();
  const int n_local = sm.n_local;
  if (n_local > 0) {
    const int j0 = sm.ids[0];
    stage_tile<W, true>(kg + (int64_t)j0 * kBlk * kD, sm.k[0], wave, lane);
    stage_tile<W, false>(vg + (int64_t)j0 * kBlk * kD, sm.v[0], wave, lane);
  }
  wait_vm();
  __syncthreads();

  for (int t = 0; t < n_local; ++t) {
    const int buf = t & 1;
    const int j = sm.ids[t];
    if (t + 1 < n_local) {
      const int jn = sm.ids[t + 1];
      stage_tile<W, true>(kg + (int64_t)jn * kBlk * kD, sm.k[buf ^ 1], wave, lane);
      stage_tile<W, false>(vg + (int64_t)jn * kBlk * kD, sm.v[buf ^ 1], wave, lane);
    }
    const unsigned char* Kt = sm.k[buf];
    const unsigned char* Vt = sm.v[buf];

    // S^T[key][query] for 4 key tiles x 2 query tiles.
    f32x4 s[2][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      s[0][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      s[1][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int r = kt * 16 + r16;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(Kt + r * kRowBytes +
                                                    (swz_k(r, ks * 4 + G) << 4)));
        s[0][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[0][ks], s[0][kt], 0, 0, 0);
        s[1][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[1][ks], s[1][kt], 0, 0, 0);
      }
    }

    // Online softmax per query column; P^T packed as the B operand of the
    // PV product: k entry 8(l/16)+i <-> key 32 ks + 4(l/16) + i for i < 4 and
    // key 32 ks + 16 + 4(l/16) + (i - 4) for i >= 4.
    bf16x8 pb[2][2];
    const bool diag = j == qb;
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      if (diag) {
        const int qrow = qoff + qt * 16 + r16;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (kt * 16 + 4 * G + i > qrow) s[qt][kt][i] = -INFINITY;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
        mx = fmaxf(mx, fmaxf(fmaxf(s[qt][kt][0], s[qt][kt][1]),
                             fmaxf(s[qt][kt][2], s[qt][kt][3])));
      mx = fmaxf(mx, xor_f(mx, 16));
      mx = fmaxf(mx, xor_f(mx, 32));
      const float m_new = fmaxf(m_run[qt], mx * c);
      const float mu = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run[qt] - mu);
      m_run[qt] = m_new;
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[qt][kt][i], c, -mu));
          s[qt][kt][i] = p;
          ps += p;
        }
      l_run[qt] = l_run[qt] * alpha + ps;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) o[qt][dt] *= alpha;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4 w;
        w[0] = pack_bf16(s[qt][2 * ks][0], s[qt][2 * ks][1]);
        w[1] = pack_bf16(s[qt][2 * ks][2], s[qt][2 * ks][3]);
        w[2] = pack_bf16(s[qt][2 * ks + 1][0], s[qt][2 * ks + 1][1]);
        w[3] = pack_bf16(s[qt][2 * ks + 1][2], s[qt][2 * ks + 1][3]);
        pb[qt][ks] = __builtin_bit_cast(bf16x8, w);
      }
    }

    // O^T[d][query] += V^T P^T.  The transposing read gives lane (l/16, l%16)
    // the four consecutive keys addressed by its 16-lane group, at column
    // l%16: lane k of the group addresses key row 4(l/16) + k/4, columns
    // 4(k%4)..+3 of the 16-column d tile.
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int r0 = 32 * ks + 4 * G + (r16 >> 2);
      const int lc = ((r16 & 3) >> 1);  // + 2 dt
      const int half = (r16 & 1) * 8;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const int off = r0 * kRowBytes + (swz_v(r0, 2 * dt + lc) << 4) + half;
        const s16x4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(Vt + off));
        const s16x4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4*)(Vt + off + 16 * kRowBytes));
        const u32x2 y0 = __builtin_bit_cast(u32x2, x0), y1 = __builtin_bit_cast(u32x2, x1);
        const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{y0[0], y0[1], y1[0], y1[1]});
        o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[0][ks], o[0][dt], 0, 0, 0);
        o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[1][ks], o[1][dt], 0, 0, 0);
      }
    }
    wait_vm();
    __syncthreads();
  }

  // Normalise and store: lane holds O^T[16 dt + 4(l/16) + i][query l%16].
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    float lt = l_run[qt];
    lt += xor_f(lt, 16);
    lt += xor_f(lt, 32);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int qpos = qb * kBlk + qoff + qt * 16 + r16;
    uint16_t* orow = out + ((int64_t)(b * h_q + h) * L + qpos) * kD;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      u32x2 w;
      w[0] = pack_bf16(o[qt][dt][0] * inv, o[qt][dt][1] * inv);
      w[1] = pack_bf16(o[qt][dt][2] * inv, o[qt][dt][3] * inv);
      *reinterpret_cast<u32x2*>(orow + dt * 16 + 4 * G) = w;
    }
    if (lse && G == 0)
      lse[(int64_t)(b * h_q + h) * L + qpos] =
          lt > 0.f ? (m_run[qt] + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_sparse_prefill(const void* q, const void* k, const void* v, int L,
                                 const int32_t* idx, const int32_t* count, int k_max,
                                 int batch, int h_q, int h_kv, float sm_scale, void* out,
                                 float* lse, hipStream_t s) {
  const int group = h_q / h_kv;
  const int heads_wg = group < 4 ? group : 4;
  const int W = 2 * heads_wg;
  const int n_chunk = group / heads_wg;
  const int n_pairs = batch * (L / kBlk) * h_kv;
  const dim3 grid((unsigned)((n_pairs + 7) / 8) * 8u * (unsigned)n_chunk);
  const float c = sm_scale * kLog2e;
  auto qq = static_cast<const uint16_t*>(q);
  auto kk = static_cast<const uint16_t*>(k);
  auto vv = static_cast<const uint16_t*>(v);
  auto oo = static_cast<uint16_t*>(out);
#define SPOT_PREFILL_CASE(WW)                                                                 \
  if (W == WW)                                                                                \
    hipLaunchKernelGGL((prefill_kernel<WW>), grid, dim3(64 * WW), 0, s, qq, kk, vv, L, idx,  \
                       count, k_max, batch, h_q, h_kv, n_chunk, n_pairs, c, oo, lse);
  SPOT_PREFILL_CASE(2)
  SPOT_PREFILL_CASE(4)
  SPOT_PREFILL_CASE(8)
#undef SPOT_PREFILL_CASE
  return hipGetLastError();
}

}  // namespace spot
