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
//   S^T = K Q^T       32 v_mfma_f32_16x16x32_bf16 (K from LDS as the A
//                     operand, Q^T held in VGPRs for the whole key loop as
//                     the B operand)
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
#include <type_traits>

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
constexpr float kLazy = 8.f;


// Physical 16-byte chunk of logical chunk c in tile row r.  K is read as 16
// rows x one chunk per quarter wave, so rows must map one chunk to distinct
// bank groups (c ^ r%16).  V is read 8 bytes per lane over 8 rows x two
// adjacent chunks per half wave ((c ^ 2(r%8)) keeps the pair adjacent).
__device__ __forceinline__ int swz_k(int r, int c) { return c ^ (r & 15); }
__device__ __forceinline__ int swz_v(int r, int c) { return c ^ ((r & 7) << 1); }

typedef __attribute__((address_space(3))) void lds_void;

// Stage one 64 x 128 BF16 tile (16 KiB, contiguous in global memory) in LDS,
// shared out over waves 0..NW-1 (1 KiB per wave instruction).
template <int NW, bool IS_K>
__device__ __forceinline__ void stage_tile(const uint16_t* __restrict__ src, unsigned char* dst,
                                           int wave, int lane) {
#pragma unroll
  for (int u = 0; u < 16 / NW; ++u) {
    const int base = (u * NW + wave) * kWave;  // first physical chunk of this wave's KiB
    const int p = base + lane;
    const int r = p >> 4, pc = p & 15;
    const int lc = IS_K ? swz_k(r, pc) : swz_v(r, pc);
    // unsigned lane offset: with a uniform src the load takes a scalar base
    // and a 32-bit offset instead of 64-bit lane addresses
    const uint32_t off = (uint32_t)(r * kD + lc * 8);
    __builtin_amdgcn_global_load_lds(src + off, (lds_void*)(dst + base * 16), 16, 0, 0);
  }
}

__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Two floats -> packed BF16 pair, round to nearest even (v_cvt_pk_bf16_f32).
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2_t));
}

// Cross-lane partner values within the wave without an LDS round trip:
// v_permlane32_swap / v_permlane16_swap exchange the two halves / the
// odd-even 16-lane rows of a register, so combining the swapped pair gives
// every lane the value of lane l ^ 32 (resp. l ^ 16) alongside its own.
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float max4(f32x4 x) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(x[0], x[1]),
                                       __builtin_elementwise_maximum(x[2], x[3]));
}

// 16 bytes (8 BF16) of logical chunk c of row r of a swizzled LDS tile.
__device__ __forceinline__ bf16x8 lds_frag(const unsigned char* base, int r, int c) {
  return __builtin_bit_cast(
      bf16x8, *reinterpret_cast<const u32x4*>(base + r * kRowBytes + (swz_k(r, c) << 4)));
}

// S^T[key][query] of one key block for the wave's 32 queries: 4 key tiles x
// 2 query tiles, eight independent accumulation chains, head dim outermost.
// The K fragments of step ks+1 are read from LDS before the MFMAs of step ks
// are issued, so the read latency hides behind matrix work.
__device__ __forceinline__ void qk_tile(const unsigned char* Kt, const bf16x8 (&qf)[4][2],
                                        f32x4 (&s)[2][4], int G, int r16) {
  bf16x8 a[2][4], bq[2][2];
  auto load = [&](int ks, int slot) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) a[slot][kt] = lds_frag(Kt, kt * 16 + r16, ks * 4 + G);
    bq[slot][0] = qf[ks][0];
    bq[slot][1] = qf[ks][1];
  };
  load(0, 0);
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int cur = ks & 1;
    if (ks + 1 < 4) load(ks + 1, cur ^ 1);
    // Keep the reads of step ks+1 ahead of the MFMAs of step ks.
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const f32x4 z = ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : s[0][kt];
      const f32x4 z1 = ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : s[1][kt];
      s[0][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[cur][kt], bq[cur][0], z, 0, 0, 0);
      s[1][kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[cur][kt], bq[cur][1], z1, 0, 0, 0);
    }
  }
}

// O^T[d][query] += V^T P^T over one key block.  The transposing read gives
// lane (l/16, l%16) the four consecutive keys addressed by its 16-lane group
// at column l%16: lane k of the group addresses key row 4(l/16) + k/4,
// columns 4(k%4)..+3 of the 16-column d tile.  The 16 V^T fragments are
// read in four groups of four, each group one group ahead of the MFMAs that
// use it (at most 16 reads in flight, the LDS counter's range).
__device__ __forceinline__ void pv_tile(const unsigned char* Vt, const bf16x8 (&pb)[2][2],
                                        f32x4 (&o)[2][8], int G, int r16) {
  bf16x8 a[2][8];
  auto load = [&](int ks, int dt0) {
    const int r0 = 32 * ks + 4 * G + (r16 >> 2);
    const int lc = (r16 & 3) >> 1;
    const int half = (r16 & 1) * 8;
#pragma unroll
    for (int dt = dt0; dt < dt0 + 4; ++dt) {
      const int off = r0 * kRowBytes + (swz_v(r0, 2 * dt + lc) << 4) + half;
      const s16x4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(Vt + off));
      const s16x4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4*)(Vt + off + 16 * kRowBytes));
      const u32x2 y0 = __builtin_bit_cast(u32x2, x0), y1 = __builtin_bit_cast(u32x2, x1);
      a[ks][dt] = __builtin_bit_cast(bf16x8, u32x4{y0[0], y0[1], y1[0], y1[1]});
    }
  };
  auto mma = [&](int ks, int dt0) {
#pragma unroll
    for (int dt = dt0; dt < dt0 + 4; ++dt) {
      o[0][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][dt], pb[0][ks], o[0][dt], 0, 0, 0);
      o[1][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks][dt], pb[1][ks], o[1][dt], 0, 0, 0);
    }
  };
  load(0, 0);
  load(0, 4);
  __builtin_amdgcn_sched_barrier(0);
  mma(0, 0);
  load(1, 0);
  __builtin_amdgcn_sched_barrier(0);
  mma(0, 4);
  load(1, 4);
  __builtin_amdgcn_sched_barrier(0);
  mma(1, 0);
  mma(1, 4);
}

template <int W>
struct PrefillWave {
  bf16x8 qf[4][2];           // Q^T B operand [ks][qt]
  f32x4 o[2][8];
  f32x4 s[2][4];             // scores S^T of the current tile
  float m_run[2], l_run[2];
  float c;
  int G, r16, qoff;

  bf16x8 pb[2][2];           // probabilities of the last finished tile

  // Matrix phase: O += P V of the previous tile, then S = K Q^T of the next.
  __device__ __forceinline__ void matrix_phase(bool do_qk, const unsigned char* Kt, bool do_pv,
                                               const unsigned char* Vp) {
    if (do_pv) pv_tile(Vp, pb, o, G, r16);
    if (do_qk) qk_tile(Kt, qf, s, G, r16);
  }

  // Vector phase: online softmax of the tile in s into pb.  DIAG masks keys
  // after the query (the query block's own key block).
  template <bool DIAG>
  __device__ __forceinline__ void softmax_phase() {
    if (DIAG) {
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const int qrow = qoff + qt * 16 + r16;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (kt * 16 + 4 * G + i > qrow) s[qt][kt][i] = -INFINITY;
      }
    }
    // Column max over the four 16-lane groups; the reference max only moves
    // when a column's max grows by more than kLazy (log2 units): the
    // probabilities then stay below 2^kLazy, far from FP32/BF16 overflow,
    // and most tiles skip the rescale of O and l.  The final division by l
    // uses the same reference, so the result is unchanged up to rounding.
    float mt[2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      float mx = __builtin_elementwise_maximum(
          __builtin_elementwise_maximum(max4(s[qt][0]), max4(s[qt][1])),
          __builtin_elementwise_maximum(max4(s[qt][2]), max4(s[qt][3])));
      mt[qt] = max_xor16(max_xor32(mx)) * c;
    }
    if (__ballot(mt[0] > m_run[0] + kLazy || mt[1] > m_run[1] + kLazy)) {
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const float m_new = fmaxf(m_run[qt], mt[qt]);
        const float alpha =
            __builtin_amdgcn_exp2f(m_run[qt] - (m_new == -INFINITY ? 0.f : m_new));
        m_run[qt] = m_new;
        l_run[qt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[qt][dt] *= alpha;
      }
    }
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      const float mu = m_run[qt] == -INFINITY ? 0.f : m_run[qt];
      float ps[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          s[qt][kt][i] = __builtin_amdgcn_exp2f(fmaf(s[qt][kt][i], c, -mu));
        ps[kt] = (s[qt][kt][0] + s[qt][kt][1]) + (s[qt][kt][2] + s[qt][kt][3]);
      }
      l_run[qt] += (ps[0] + ps[1]) + (ps[2] + ps[3]);
      // P^T as the B operand of the PV product: k entry 8(l/16)+i holds key
      // 32 ks + 4(l/16) + i for i < 4 and key 32 ks + 16 + 4(l/16) + (i - 4)
      // for i >= 4, matching the key order of the transposed V reads.
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
  }

  __device__ __forceinline__ void softmax_phase(bool diag) {
    if (diag)
      softmax_phase<true>();
    else
      softmax_phase<false>();
  }
};

template <int W>
__global__ __launch_bounds__(64 * W) void prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, int L, const int32_t* __restrict__ idx,
    const int32_t* __restrict__ count, int k_max, int batch, int h_q, int h_kv, int n_chunk,
    int n_pairs, float c, uint16_t* __restrict__ out, float* __restrict__ lse) {
  // Each tile buffer is a variable of its own and every access names it at
  // compile time (the loop below is unrolled by two), so the compiler can
  // tell the direct global->LDS writes into one buffer from the reads of
  // another and does not wait for the loads in flight before reading.
  __shared__ __attribute__((aligned(16))) unsigned char sk0[kTileBytes], sk1[kTileBytes];
  __shared__ __attribute__((aligned(16))) unsigned char sv0[kTileBytes], sv1[kTileBytes];
  __shared__ int s_ids[kPrefillMaxIds];
  __shared__ int s_n_local, s_has_diag;
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

  // Selected key blocks that exist for this query block: ids in [0, qb) in
  // list order, then the query block's own block qb (the only one that needs
  // the causal mask) last if it was selected.
  if (wave == 0) {
    const int n_e = min(max(count[row], 0), k_max);
    const int32_t* ids_row = idx + (int64_t)row * k_max;
    int n = 0;
    bool diag = false;
    for (int base = 0; base < n_e; base += kWave) {
      const int e = base + lane;
      const int j = e < n_e ? ids_row[e] : -1;
      const bool ok = j >= 0 && j < qb;
      const uint64_t m = __ballot(ok);
      const int pos = n + __popcll(m & ((1ull << lane) - 1ull));
      if (ok && pos < kPrefillMaxIds) s_ids[pos] = j;
      n += __popcll(m);
      diag = diag || __ballot(j == qb) != 0;
    }
    if (lane == 0) {
      n = min(n, kPrefillMaxIds - 1);
      if (diag) s_ids[n++] = qb;
      s_n_local = n;
      s_has_diag = diag;
    }
  }

  PrefillWave<W> wv;
  wv.G = lane >> 4;
  wv.r16 = lane & 15;
  wv.qoff = (wave & 1) * 32;
  wv.c = c;
  // The wave's 32 query rows stay in registers as the QK product's B
  // operand for the whole key loop: lane holds Q[16 qt + l%16][32 ks +
  // 8(l/16) ..+7] in qf[ks][qt].
  {
    const uint16_t* qh = q + ((int64_t)(b * h_q + h) * L + qb * kBlk + wv.qoff) * kD;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int qt = 0; qt < 2; ++qt)
        wv.qf[ks][qt] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(qh + (qt * 16 + wv.r16) * kD + ks * 32 +
                                                    8 * wv.G));
  }
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) wv.o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    wv.m_run[qt] = -INFINITY;
    wv.l_run[qt] = 0.f;
  }

  const uint16_t* kg = k + (int64_t)(b * h_kv + g) * L * kD;
  const uint16_t* vg = v + (int64_t)(b * h_kv + g) * L * kD;
  // The block id read from LDS is the same in every lane; readfirstlane
  // makes the tile's base address scalar, so the tile copies below take the
  // scalar-base form with a 32-bit lane offset.
  auto blk = [](const uint16_t* base, int j) {
    return base + (int64_t)__builtin_amdgcn_readfirstlane(j) * kBlk * kD;
  };

  // Ping-pong schedule.  The waves form two groups, 0..W/2-1 and W/2..W-1,
  // so the two waves sharing a SIMD belong to different groups.  A wave in
  // its matrix phase raises its issue priority (s_setprio), so that when
  // both waves of a SIMD are ready the MFMAs and LDS reads go first and the
  // softmax's VALU work fills the gaps (about 6 % faster than equal
  // priority on the 32K-token layer).  Time is cut
  // into half periods separated by workgroup barriers; in each, one group
  // runs its matrix phase (P V of tile t-1, then S of tile t) while the
  // other runs its vector phase (softmax), so MFMA work of one wave overlaps
  // VALU work of the other.  Group 1 runs the same sequence one half period
  // later.  Tile t (t = 0..n) takes half periods 2t and 2t+1:
  //   2t:   loads K(t+1) -> K buffer (t+1)%2, V(t) -> V buffer t%2;
  //         group 0 matrix(t), group 1 softmax(t-1)
  //   2t+1: group 0 softmax(t), group 1 matrix(t); loads complete.
  // Matrix(t) reads K buffer t%2 and V buffer (t-1)%2, never a buffer a load
  // in flight writes to.  Buffer parity is a compile-time constant (the loop
  // is unrolled by two, each buffer its own variable), which lets the
  // compiler skip waiting on the loads before its LDS reads.
  __syncthreads();
  const int n_local = s_n_local;
  const bool has_diag = s_has_diag;
  const bool grp1 = wave >= W / 2;
  if (n_local > 0) stage_tile<W, true>(blk(kg, s_ids[0]), sk0, wave, lane);
  wait_vm();
  __syncthreads();
  auto tile = [&](auto parity, int t) {
    constexpr int P = decltype(parity)::value;
    unsigned char* kcur = P ? sk1 : sk0;
    unsigned char* knext = P ? sk0 : sk1;
    unsigned char* vcur = P ? sv1 : sv0;
    unsigned char* vprev = P ? sv0 : sv1;
    const bool do_qk = t < n_local, do_pv = t >= 1;
    // The two groups run separate straight-line paths (the barrier counts
    // match: one mid-period barrier and one end-of-period barrier each), so
    // the compiler sees that group 1 never has a direct-to-LDS load in
    // flight; a wave with one in flight only gets full LDS waits, which
    // would serialise its matrix phase.  Group 0 therefore issues all tile
    // loads, right after its own LDS reads.
    if (!grp1) {
      __builtin_amdgcn_s_setprio(3);
      wv.matrix_phase(do_qk, kcur, do_pv, vprev);
      __builtin_amdgcn_s_setprio(0);
      if (t + 1 < n_local) stage_tile<W / 2, true>(blk(kg, s_ids[t + 1]), knext, wave, lane);
      if (t < n_local) stage_tile<W / 2, false>(blk(vg, s_ids[t]), vcur, wave, lane);
      // Phase switch only: no LDS data changes hands here, so no memory
      // fence (a fence would also wait for the tile loads in flight).
      __builtin_amdgcn_s_barrier();
      if (do_qk) wv.softmax_phase(has_diag && t + 1 == n_local);
      wait_vm();
      __syncthreads();
    } else {
      if (do_pv) wv.softmax_phase(has_diag && t == n_local);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_s_setprio(3);
      wv.matrix_phase(do_qk, kcur, do_pv, vprev);
      __builtin_amdgcn_s_setprio(0);
      __syncthreads();
    }
  };
  if (n_local > 0) {
    for (int t = 0;; t += 2) {
      tile(std::integral_constant<int, 0>(), t);
      if (t + 1 > n_local) break;
      tile(std::integral_constant<int, 1>(), t + 1);
      if (t + 2 > n_local) break;
    }
  }

  // Normalise and store: lane holds O^T[16 dt + 4(l/16) + i][query l%16].
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const float lt = sum_xor16(sum_xor32(wv.l_run[qt]));
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int qpos = qb * kBlk + wv.qoff + qt * 16 + wv.r16;
    uint16_t* orow = out + ((int64_t)(b * h_q + h) * L + qpos) * kD;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      u32x2 w;
      w[0] = pack_bf16(wv.o[qt][dt][0] * inv, wv.o[qt][dt][1] * inv);
      w[1] = pack_bf16(wv.o[qt][dt][2] * inv, wv.o[qt][dt][3] * inv);
      *reinterpret_cast<u32x2*>(orow + dt * 16 + 4 * wv.G) = w;
    }
    if (lse && wv.G == 0)
      lse[(int64_t)(b * h_q + h) * L + qpos] =
          lt > 0.f ? (wv.m_run[qt] + __log2f(lt)) * kLn2 : -INFINITY;
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
