// Selection cores shared by the stand-alone selection kernels and the fused
// decode step: order-preserving score keys, cross-lane exchanges, a
// descending bitonic sort of packed keys held in registers, and the
// workgroup (256-thread) selection of one row.
#pragma once

#include "spot_internal.h"

namespace spot {

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  u = u == 0x80000000u ? 0u : u;   // -0 and +0 are the same score (a tie)
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float order_key_inv(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}


// Value of lane (lane ^ m); m is a power of two and a compile-time constant
// after unrolling.  Needs the full wave active.
__device__ __forceinline__ uint32_t xor_lane(uint32_t x, int m) {
  switch (m) {
    case 1: return (uint32_t)dpp_i<kDppQuadXor1>((int)x);
    case 2: return (uint32_t)dpp_i<kDppQuadXor2>((int)x);
    case 4: {
      const uint32_t up = (uint32_t)dpp_i<0x104>((int)x);  // row_shl:4, lane i <- i + 4
      const uint32_t dn = (uint32_t)dpp_i<0x114>((int)x);  // row_shr:4, lane i <- i - 4
      return (__lane_id() & 4) ? dn : up;
    }
    case 8: return (uint32_t)dpp_i<0x128>((int)x);          // row_ror:8 == xor 8
    case 16: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x401F);  // xor 16
    default: return (uint32_t)__builtin_amdgcn_ds_bpermute((__lane_id() ^ 32) << 2, (int)x);
  }
}
__device__ __forceinline__ uint64_t xor_lane64(uint64_t x, int m) {
  const uint32_t lo = xor_lane((uint32_t)x, m), hi = xor_lane((uint32_t)(x >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive float prefix sum over lanes (same tree as wave_incl_scan_i).
__device__ __forceinline__ float wave_incl_scan_f(float x) {
  const int lane = __lane_id();
  x += dpp_f<0x111>(x);
  x += dpp_f<0x112>(x);
  x += dpp_f<0x114>(x);
  x += dpp_f<0x118>(x);
  const float r0 = readlane_f(x, 15), r1 = readlane_f(x, 31), r2 = readlane_f(x, 47);
  const int row = lane >> 4;
  if (row > 0) x += r0;
  if (row > 1) x += r1;
  if (row > 2) x += r2;
  return x;
}

// Descending bitonic sort of 64 * SPL packed keys; slot i = lane * SPL + t.
template <int SPL>
__device__ __forceinline__ void bitonic_desc(uint64_t (&K)[SPL]) {
  constexpr int P = 64 * SPL;
  const int lane = __lane_id();
#pragma unroll
  for (int k = 2; k <= P; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j < SPL) {
#pragma unroll
        for (int t = 0; t < SPL; ++t) {
          const int u = t ^ j;
          if (u > t) {
            const bool up = (((lane * SPL + t) & k) == 0);
            const uint64_t a = K[t], b = K[u];
            const bool swap = up ? (a < b) : (a > b);
            K[t] = swap ? b : a;
            K[u] = swap ? a : b;
          }
        }
      } else {
        const int m = j / SPL;
        const bool lower = (lane & m) == 0;
#pragma unroll
        for (int t = 0; t < SPL; ++t) {
          const uint64_t o = xor_lane64(K[t], m);
          const bool up = (((lane * SPL + t) & k) == 0);
          const bool keep_max = up == lower;
          K[t] = keep_max ? (K[t] > o ? K[t] : o) : (K[t] < o ? K[t] : o);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Workgroup (4 waves) selection for rows of up to 4096 blocks, cap <= 512
// (select_row_core below): the single-wave kernel's rule with the element-wise
// phases spread over 256 threads (EPT <= 16 consecutive ids each).
constexpr int kSelWG = 256;

// Exclusive prefix over the 256 threads in thread order; `total` = sum.
__device__ __forceinline__ int wg_excl_scan(int v, int* red, int& total) {
  const int lane = __lane_id(), wave = threadIdx.x >> 6;
  const int incl = wave_incl_scan_i(v);
  if (lane == 63) red[wave] = incl;
  __syncthreads();
  int base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kSelWG / 64; ++w) {
    const int t = red[w];
    base += w < wave ? t : 0;
    total += t;
  }
  __syncthreads();
  return base + incl - v;
}


// Score source of select_row_core: plain loads of a row of scores (never
// fails).  The fused decode step substitutes a source that polls records
// written by other workgroups of the same launch and fails when its bounded
// wait expires.
struct RowScores {
  const float* srow;
  template <int EPT>
  __device__ __forceinline__ bool operator()(float (&sv)[EPT], int j0, int nv) const {
#pragma unroll
    for (int e = 0; e < EPT; ++e) sv[e] = j0 + e < nv ? srow[j0 + e] : -INFINITY;
    return true;
  }
};

// The same row through LDS, for long rows: a thread owns EPT consecutive
// ids, so loading them directly makes every wave-wide load touch 64 cache
// lines (one per lane, each line requested again for every element) -- with
// 32 ids per thread that took ~6 us per row.  Here each wave loads its own
// 64 * EPT scores lane-contiguously (two lines per load), parks them in its
// part of stage[] and reads its threads' runs back; only the wave's own
// lanes touch its part, so no workgroup barrier is needed.
struct StagedRowScores {
  const float* srow;
  float* stage;   // kSelWG * EPT floats of LDS
  template <int EPT>
  __device__ __forceinline__ bool operator()(float (&sv)[EPT], int j0, int nv) const {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wbase = j0 - lane * EPT;          // the wave's first id
    float* st = stage + wave * 64 * EPT;
    float v[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const int j = wbase + 64 * i + lane;
      v[i] = j < nv ? srow[j] : -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) st[64 * i + lane] = v[i];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int e = 0; e < EPT; e += 4) {
      const float4 x = *reinterpret_cast<const float4*>(&st[lane * EPT + e]);
      sv[e] = x.x;
      sv[e + 1] = x.y;
      sv[e + 2] = x.z;
      sv[e + 3] = x.w;
    }
    return true;
  }
};

constexpr int kValBins = 2048;   // value bins of the threshold search

#ifndef SPOT_SEL_TS
#define SPOT_SEL_TS(i) ((void)0)
#endif

constexpr int kFine = kValBins / 64;   // value bins per coarse bin

template <int EPT, int SPL>
struct SelWgSmem {
  alignas(16) uint32_t hist[kValBins];   // value-bin counts (the fallback radix uses 256)
  uint64_t s_K[64 * (SPL > 4 ? SPL : 4)];   // threshold-bin members (64 per wave) / survivors
  uint32_t red_u[kSelWG / 64][2];
  float red_f[kSelWG / 64];
  float red_m[kSelWG / 64];       // survivors' mass partials
  int red_i[kSelWG / 64];
  int red_bad[kSelWG / 64];       // per wave: a score source failed
  int gc[kSelWG / 64];            // threshold-bin members / survivors per wave
  int bc[4];
  uint64_t cut;
  float cut_mass;
  // nucleus without a sort (cap <= 64); separate from s_K and gc, which the
  // threshold-bin ranking may still be reading when a wave gets here
  uint64_t s_sk[64];              // survivors' packed rank keys, in block order
  float s_pe[64];                 // their exp(s - M)
  int part_rk[kSelWG / 64][64];   // per wave: better survivors of its run, per survivor
  float part_mb[kSelWG / 64][64]; // per wave: their mass, per survivor
};

// What select_row_core leaves in each thread (ids [tid*EPT, tid*EPT + EPT)).
struct SelRow {
  uint32_t fin;    // bit e: id tid*EPT + e is in S
  float mass;      // nucleus mass (the same in every thread)
  bool ok;         // false: the score source failed; fin = 0
};

// Packed rank key: higher score first, then lower block id; unique per id.
__device__ __forceinline__ uint64_t rank_key(uint32_t key, int id) {
  return ((uint64_t)key << 32) | (uint64_t)(0xffffffffu - (uint32_t)id);
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// Selection of one row by the whole 256-thread workgroup: src supplies the
// row's scores (the first nv valid).  Needs min(k_max, nv) <= P = 64 * SPL
// (<= 512).  Every thread of the workgroup must call it.  Thread t owns the
// EPT consecutive ids [t*EPT, (t+1)*EPT).  Steps, with the workgroup barriers
// in brackets:
//  1. load; order-preserving keys of the residual candidates; residual max
//     M and min from per-wave partials [1]; Z = sum exp(s - M) per wave,
//     combined after the next barrier;
//  2. when the cap C binds: a histogram over 2048 equal-width value bins
//     between the candidate min and max [1]; every wave sums the bins into
//     64 coarse bins of 32 and scans the coarse and then the fine counts
//     for the bin holding the C-th best candidate (score desc, id asc); each
//     wave packs its members of that bin and sums the mass of its
//     candidates in better bins [1]; every wave ranks the members by
//     counting and derives the
//     packed cut key and the mass of the survivors.  The survivors are the
//     candidates whose packed key reaches the cut (when the cap-th best
//     candidate is the last of its bin, simply the candidates of that bin
//     and the better ones, with no packing or ranking).  A bin too crowded to
//     rank (heavy ties) falls back to an 8-bit radix select on the keys;
//  3. below top_p * Z the cap binds and the survivors are the answer;
//     otherwise the survivors are ranked by (score desc, id asc) and cut
//     where the prefix mass first reaches top_p * Z, then floored by k_min:
//     the survivors are compacted in block order [2]; up to 64 of them are
//     ranked without sorting -- wave w compares every survivor with
//     survivors 16w .. 16w+15 (how many are better, and their mass) [1],
//     and every wave adds the four parts in order and takes the same cut (a
//     survivor is in the nucleus when the mass of the better survivors is
//     still below top_p * Z); more are sorted in wave 0, prefix-summed and
//     cut [1];
// It returns, in every thread, the bits of its ids that belong to S (reserved
// + chosen) and the nucleus mass; sel_positions / sel_write turn them into
// the ascending id list [1].  A score source that fails (a bounded wait that
// expired) makes the whole workgroup return ok = false with no ids.
// Every reduction has a fixed order, so the result is deterministic.
template <int EPT, int SPL, class Src>
__device__ __forceinline__ SelRow select_row_core(SelWgSmem<EPT, SPL>& sm, const Src& src,
                                                  int nv, float top_p, int k_max, int k_min,
                                                  int n_sink, int n_recent) {
  constexpr int NT = kSelWG, NW = NT / 64;
  constexpr int P = 64 * SPL;
  constexpr float kLog2e = 1.4426950408889634f;
  static_assert(EPT <= 32, "a thread's ids must fit one 32-bit word");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sink_end = min(n_sink, nv);
  const int rec_start = max(0, nv - n_recent);
  const int n_reserved = sink_end + (nv - rec_start) - max(0, sink_end - rec_start);
  const int n_res = nv - n_reserved;
  const int cap = min(k_max - n_reserved, n_res);
  const int j0 = tid * EPT;

  // 1. scores, keys (0 = not a candidate), M and min
  SPOT_SEL_TS(0);
  float sv[EPT];
  const bool src_ok = src(sv, j0, nv);
  static_assert(kValBins == NT * 8, "two 16-byte zero stores per thread");
  reinterpret_cast<uint4*>(sm.hist)[2 * tid] = make_uint4(0u, 0u, 0u, 0u);
  reinterpret_cast<uint4*>(sm.hist)[2 * tid + 1] = make_uint4(0u, 0u, 0u, 0u);
  uint32_t key[EPT];
  uint32_t cand = 0, resv = 0;
  {
    const int lo = max(sink_end - j0, 0), hi = min(rec_start - j0, EPT);
    const int vend = min(nv - j0, EPT);
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool c = e >= lo && e < hi;
      key[e] = c ? order_key(sv[e]) : 0u;
      cand |= (uint32_t)c << e;
      resv |= (uint32_t)(e < vend && !c) << e;
    }
  }
  SPOT_SEL_TS(1);
  uint32_t kmax = 0u, kmin = 0xffffffffu;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    kmax = max(kmax, key[e]);
    kmin = min(kmin, key[e] ? key[e] : 0xffffffffu);
  }
  kmax = wave_max_u(kmax);
  kmin = wave_min_u(kmin);
  const bool wave_bad = __ballot(!src_ok) != 0ull;
  if (lane == 0) {
    sm.red_u[wave][0] = kmax;
    sm.red_u[wave][1] = kmin;
    sm.red_bad[wave] = wave_bad;
  }
  __syncthreads();
  {
    bool bad = false;
#pragma unroll
    for (int w = 0; w < NW; ++w) bad = bad || sm.red_bad[w];
    if (bad) return SelRow{0u, 0.f, false};   // uniform over the workgroup
  }
  kmax = 0u;
  kmin = 0xffffffffu;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    kmax = max(kmax, sm.red_u[w][0]);
    kmin = min(kmin, sm.red_u[w][1]);
  }
  const float M = order_key_inv(kmax);
  float pe[EPT];                                 // exp(s - M) of the candidates
#pragma unroll
  for (int e = 0; e < EPT; ++e) pe[e] = __builtin_amdgcn_exp2f((sv[e] - M) * kLog2e);
  {
    // Z's per-wave partials, read after the next barrier (every path below
    // has one before the nucleus decision)
    float zl = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) zl += ((cand >> e) & 1u) ? pe[e] : 0.f;
    const float zw = wave_sum(zl);
    if (lane == 0) sm.red_f[wave] = zw;
  }
  SPOT_SEL_TS(2);

  // 2. the cut: survivors are the candidates with rank_key >= (kt, it)
  const bool thresh = cap > 0 && cap < n_res;
  uint32_t kt = cap <= 0 ? 0xffffffffu : 1u;     // threshold key
  int it = cap <= 0 ? -1 : 0x7fffffff;            // largest id kept at the threshold key
  float msum = 0.f;
  bool have_msum = false;
  bool crowded = thresh;
  bool by_bin = false;        // the survivors are exactly the candidates in bins <= b*
  uint32_t surv_bin = 0u;
  if (thresh) {
    const float vhi = M, vlo = order_key_inv(kmin);
    const float span = vhi - vlo;
    if (span > 0.f && span < INFINITY) {
      const float inv_w = (float)kValBins / span * 0.99999f;
      int bin[EPT];
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        // bins ascend as values descend; clamped in float first
        bin[e] = (int)fminf((vhi - sv[e]) * inv_w, (float)(kValBins - 1));
        if (key[e]) atomicAdd(&sm.hist[bin[e]], 1u);
      }
      __syncthreads();
      SPOT_SEL_TS(6);
      // Every wave finds the bin of the cap-th best candidate on its own: a
      // scan over the 64 coarse bins, then over the 32 fine bins of the
      // coarse bin that holds it (no barrier).
      // lane l sums fine bins [32 l, 32 l + 32): eight 16-byte reads, the
      // chunk order rotated by lane so a read spreads over the banks
      int cc = 0;
#pragma unroll
      for (int k = 0; k < kFine / 4; ++k) {
        const uint4 t = reinterpret_cast<const uint4*>(sm.hist)[lane * (kFine / 4) +
                                                              ((k + (lane >> 1)) & (kFine / 4 - 1))];
        cc += (int)(t.x + t.y + t.z + t.w);
      }
      const int c_incl = wave_incl_scan_i(cc);
      const int cb = min(__builtin_ctzll(__ballot(c_incl >= cap)), 63);
      const int c_before = __builtin_amdgcn_readlane(c_incl - cc, cb);
      const int fc = lane < kFine ? (int)sm.hist[cb * kFine + lane] : 0;
      const int f_incl = wave_incl_scan_i(fc) + c_before;
      const int fb = min(__builtin_ctzll(__ballot(lane < kFine && f_incl >= cap)), kFine - 1);
      const int b_star = cb * kFine + fb;
      const int need = cap - __builtin_amdgcn_readlane(f_incl - fc, fb);
      const int in_bin = __builtin_amdgcn_readlane(fc, fb);
      SPOT_SEL_TS(7);
      if (in_bin == need) {
        // The cap-th best candidate is the last of its bin: every candidate
        // of the bin and of the better bins survives, no ranking needed.
        crowded = false;
        by_bin = true;
#pragma unroll
        for (int e = 0; e < EPT; ++e) surv_bin |= (uint32_t)(key[e] && bin[e] <= b_star) << e;
      } else if (in_bin <= 64) {
        crowded = false;
        // each wave packs its members of the bin into its own run of s_K and
        // sums the mass of its candidates in better bins
        uint32_t mm = 0u;
        float ma = 0.f;
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
          mm |= (uint32_t)(key[e] && bin[e] == b_star) << e;
          ma += key[e] && bin[e] < b_star ? pe[e] : 0.f;
        }
        const int nm = __popc(mm);
        const int m_incl = wave_incl_scan_i(nm);
        int slot = wave * 64 + m_incl - nm;
#pragma unroll
        for (int e = 0; e < EPT; ++e)
          if ((mm >> e) & 1u) sm.s_K[slot++] = rank_key(key[e], j0 + e);
        const float mw = wave_sum(ma);
        if (lane == 63) sm.gc[wave] = m_incl;
        if (lane == 0) sm.red_m[wave] = mw;
        __syncthreads();
        SPOT_SEL_TS(8);
        // every wave ranks the members (member l in lane l) by counting the
        // better ones and derives the same cut and mass (no barrier)
        int w_of = 0, base = 0, run = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const int n_w = sm.gc[w];
          if (lane >= run) {
            w_of = w;
            base = run;
          }
          run += n_w;
        }
        const uint64_t mine = lane < in_bin ? sm.s_K[w_of * 64 + lane - base] : 0ull;
        int better = 0;
        for (int j = 0; j < in_bin; ++j) better += readlane_u64(mine, j) > mine ? 1 : 0;
        const bool top = lane < in_bin && better < need;
        const float x = top ? __builtin_amdgcn_exp2f(
                                  (order_key_inv((uint32_t)(mine >> 32)) - M) * kLog2e)
                            : 0.f;
        const float m_in = wave_sum(x);
        const int src = __builtin_ctzll(__ballot(lane < in_bin && better == need - 1));
        const uint64_t kc = readlane_u64(mine, src);
        kt = (uint32_t)(kc >> 32);
        it = (int)(0xffffffffu - (uint32_t)kc);
        msum = m_in;
#pragma unroll
        for (int w = 0; w < NW; ++w) msum += sm.red_m[w];
        have_msum = true;
      }
    }
  }
  if (crowded) {
    // 8-bit radix select by count on the keys, from the highest bit where
    // the candidates differ; equal keys at the threshold go to lower ids.
    __syncthreads();   // every wave is done reading the value histograms
    const uint32_t diff = kmin ^ kmax;
    int shift = diff ? 32 - __builtin_clz(diff) : 0;
    uint32_t prefix = shift >= 32 ? 0u : (kmax >> shift) << shift;
    uint32_t pmask = shift >= 32 ? 0u : ~0u << shift;
    int need = cap;
    while (shift > 0) {
      const int width = shift < 8 ? shift : 8;
      shift -= width;
      const uint32_t dmask = (1u << width) - 1u;
      sm.hist[tid] = 0u;
      __syncthreads();
#pragma unroll
      for (int e = 0; e < EPT; ++e)
        if (key[e] && (key[e] & pmask) == prefix) atomicAdd(&sm.hist[(key[e] >> shift) & dmask], 1u);
      __syncthreads();
      if (wave == 0) {
        int c[4], tot = 0;                   // lane l: digits 255-4l .. 252-4l
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          c[i] = (int)sm.hist[255 - 4 * lane - i];
          tot += c[i];
        }
        const int incl = wave_incl_scan_i(tot);
        int before = incl - tot;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (before < need && need <= before + c[i]) {
            sm.bc[0] = 255 - 4 * lane - i;
            sm.bc[1] = need - before;
          }
          before += c[i];
        }
      }
      __syncthreads();
      prefix |= (uint32_t)sm.bc[0] << shift;
      pmask |= dmask << shift;
      need = sm.bc[1];
    }
    // the need-th lowest id among the keys equal to the threshold
    int n_eq = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) n_eq += key[e] == prefix ? 1 : 0;
    int total;
    int eq_before = wg_excl_scan(n_eq, sm.red_i, total);
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if (key[e] == prefix) {
        if (++eq_before == need) sm.bc[2] = j0 + e;
      }
    }
    __syncthreads();
    kt = prefix;
    it = sm.bc[2];
  }
  // survivor bits (key > kt, or key == kt and id <= it; or by bin)
  uint32_t surv = surv_bin;
  if (!by_bin) {
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool sv_ = key[e] && (key[e] > kt || (key[e] == kt && j0 + e <= it));
      surv |= (uint32_t)sv_ << e;
    }
  }
  if (!have_msum) {
    float ms = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) ms += ((surv >> e) & 1u) ? pe[e] : 0.f;
    const float mw = wave_sum(ms);
    if (lane == 0) sm.red_m[wave] = mw;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < NW; ++w) msum += sm.red_m[w];
  }
  SPOT_SEL_TS(3);

  // 3. the nucleus (the same decision in every thread)
  float Z = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) Z += sm.red_f[w];
  const float pz = top_p * Z;
  int n;                                  // -1: the nucleus ends before the cap
  if (cap <= 0) n = 0;
  else if (top_p >= 1.f) n = cap;
  else if (top_p <= 0.f) n = 0;
  else if (msum < pz) n = cap;            // the cap binds before the nucleus reaches top_p
  else n = -1;
  if (n >= 0 && n_reserved + n < k_min) n = min(k_min - n_reserved, cap);
  uint32_t chosen = n == 0 ? 0u : surv;
  float mass = n > 0 && Z > 0.f ? msum / Z : 0.f;
  if ((n < 0 || (n > 0 && n < cap)) && cap <= 64) {
    // survivors (exactly cap <= 64 of them) ranked without a sort,
    // compacted in block order
    int run;
    int slot = wg_excl_scan(__popc(surv), sm.red_i, run);
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if ((surv >> e) & 1u) {
        sm.s_sk[slot] = rank_key(key[e], j0 + e);
        sm.s_pe[slot] = pe[e];
        ++slot;
      }
    }
    __syncthreads();
    SPOT_SEL_TS(5);
    // lane i holds survivor i
    const bool real = lane < run;
    const uint64_t mine = real ? sm.s_sk[lane] : 0ull;
    const float pmine = real ? sm.s_pe[lane] : 0.f;
    {
      // survivors [16 w, 16 w + 16) against survivor `lane`, in order, eight
      // per batch of LDS reads
      int rk = 0;
      float mb = 0.f;
#pragma unroll
      for (int jb = 16 * wave; jb < 16 * wave + 16; jb += 8) {
        uint64_t kk[8];
        float pp[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          kk[u] = sm.s_sk[jb + u];
          pp[u] = sm.s_pe[jb + u];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const bool better = jb + u < run && kk[u] > mine;
          rk += better ? 1 : 0;
          mb += better ? pp[u] : 0.f;
        }
      }
      sm.part_rk[wave][lane] = rk;
      sm.part_mb[wave][lane] = mb;
    }
    __syncthreads();
    SPOT_SEL_TS(9);
    int rk = 0;
    float mb = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      rk += sm.part_rk[w][lane];
      mb += sm.part_mb[w][lane];
    }
    int nn = n;
    if (nn < 0) {
      nn = __popcll(__ballot(real && mb < pz));
      if (n_reserved + nn < k_min) nn = min(k_min - n_reserved, cap);
    }
    nn = min(max(nn, 1), run);
    const uint64_t at = __ballot(real && rk == nn - 1);
    const int src = at ? __builtin_ctzll(at) : 0;
    const uint64_t kc = readlane_u64(mine, src);
    const float m_at = readlane_f(mb + pmine, src);
    mass = Z > 0.f ? m_at / Z : 0.f;
    const uint32_t ck = (uint32_t)(kc >> 32);
    const int ci = (int)(0xffffffffu - (uint32_t)kc);
    chosen = 0u;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool ch = ((surv >> e) & 1u) && (key[e] > ck || (key[e] == ck && j0 + e <= ci));
      chosen |= (uint32_t)ch << e;
    }
  } else if (n < 0 || (n > 0 && n < cap)) {
    // survivors (exactly cap of them) in rank order: compact, sort, cut
    int total;
    int pos = wg_excl_scan(__popc(surv), sm.red_i, total);
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if ((surv >> e) & 1u) sm.s_K[pos++] = rank_key(key[e], j0 + e);
    for (int i = total + tid; i < P; i += NT) sm.s_K[i] = 0ull;   // padding sorts last
    __syncthreads();
    if (wave == 0) {
      uint64_t K[SPL];
#pragma unroll
      for (int t = 0; t < SPL; ++t) K[t] = sm.s_K[lane * SPL + t];
      bitonic_desc<SPL>(K);
      float cum[SPL], run = 0.f;
#pragma unroll
      for (int t = 0; t < SPL; ++t) {
        const bool real = lane * SPL + t < cap;
        run += real ? __builtin_amdgcn_exp2f((order_key_inv((uint32_t)(K[t] >> 32)) - M) * kLog2e)
                    : 0.f;
        cum[t] = run;
      }
      const float offs = wave_incl_scan_f(run) - run;
#pragma unroll
      for (int t = 0; t < SPL; ++t) cum[t] += offs;
      int nn = n;
      if (nn < 0) {
        int below = 0;
#pragma unroll
        for (int t = 0; t < SPL; ++t) below += (lane * SPL + t < cap && cum[t] < pz) ? 1 : 0;
        nn = min(cap, wave_sum_i(below) + 1);
        if (n_reserved + nn < k_min) nn = min(k_min - n_reserved, cap);
      }
      const int ln = (nn - 1) / SPL, tn = (nn - 1) % SPL;
      uint64_t mk = 0ull;
      float mc = 0.f;
#pragma unroll
      for (int t = 0; t < SPL; ++t) {
        mk = t == tn ? K[t] : mk;
        mc = t == tn ? cum[t] : mc;
      }
      const uint64_t kc = readlane_u64(mk, ln);
      const float m_at = readlane_f(mc, ln);
      if (lane == 0) {
        sm.cut = kc;
        sm.cut_mass = Z > 0.f ? m_at / Z : 0.f;
      }
    }
    __syncthreads();
    const uint64_t kc = sm.cut;
    const uint32_t ck = (uint32_t)(kc >> 32);
    const int ci = (int)(0xffffffffu - (uint32_t)kc);
    mass = sm.cut_mass;
    chosen = 0u;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool ch = ((surv >> e) & 1u) && (key[e] > ck || (key[e] == ck && j0 + e <= ci));
      chosen |= (uint32_t)ch << e;
    }
  
  }
  SPOT_SEL_TS(4);

  return SelRow{resv | chosen, mass, true};
}

// Position (in ascending block id) of the calling thread's first id of S and
// |S| itself: a workgroup exclusive scan of the threads' counts (one barrier).
template <int EPT, int SPL>
__device__ __forceinline__ int sel_positions(SelWgSmem<EPT, SPL>& sm, uint32_t fin, int& total) {
  constexpr int NW = kSelWG / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int mine = __popc(fin);
  const int incl = wave_incl_scan_i(mine);
  if (lane == 63) sm.red_i[wave] = incl;
  __syncthreads();
  int pos = incl - mine;
  total = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int t = sm.red_i[w];
    pos += w < wave ? t : 0;
    total += t;
  }
  return pos;
}

// Writes the selection of one row: S in ascending block id into out[0,
// k_max) (-1 past |S|), |S| and the nucleus mass.  Every thread of the
// workgroup calls it with its own fin and position.
template <int EPT>
__device__ __forceinline__ void sel_write(int32_t* __restrict__ out, int32_t* __restrict__ count_out,
                                          float* __restrict__ mass_out, int k_max, uint32_t fin,
                                          int pos, int total, float mass) {
  const int tid = threadIdx.x, j0 = tid * EPT;
  const int n_out = min(total, k_max);
#pragma unroll
  for (int e = 0; e < EPT; ++e)
    if (((fin >> e) & 1u) && pos < n_out) out[pos++] = j0 + e;
  for (int i = n_out + tid; i < k_max; i += kSelWG) out[i] = -1;
  if (tid == 0) {
    *count_out = n_out;
    if (mass_out) *mass_out = mass;
  }
}

}  // namespace spot
