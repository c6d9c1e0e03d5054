// Dual top-p / top-K block selection (paper Section 2.3, Eqs. select-topk,
// select-nucleus and select-topp) with a cap k_max on the set size.
//
// Three kernels, chosen by row length and cap (one row per workgroup):
//  * rows of up to 512 blocks: one wavefront (select_wave_kernel);
//  * 513 .. 8192 blocks: one 256-thread workgroup (select_wg_kernel, its body
//    in select_core.h, shared with the fused decode step), for caps up to
//    1024 and, when top_p >= 1 (static top-K: no survivor sort), any cap;
//  * longer rows or larger caps: the 256-thread sort-based select_kernel.
// All follow the same steps per row:
//  1. reserved blocks (sink prefix, recency suffix) are set aside; the
//     residual candidates get an order-preserving 32-bit key of their score;
//  2. residual softmax statistics: max and Z = sum exp(s - max) with a fixed
//     reduction tree (deterministic);
//  3. only the best C = min(k_max - |R|, |B_res|) candidates can ever be
//     chosen; a radix select by count finds the C-th largest key, and equal
//     keys at the threshold are taken in ascending block id;
//  4. the C survivors are sorted by (score desc, id asc), their probabilities
//     prefix-summed in that order (fixed tree, FP32), and the nucleus length
//     n is the first prefix reaching top_p * Z, then capped and floored by
//     k_min (when the survivors' total mass stays below top_p * Z the cap
//     binds and no sort is needed);
//  5. reserved + the first n survivors are written in ascending block id.
#include "select_core.h"

namespace spot {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

struct Scratch {
  int wave_i[kWaves];
  float wave_f[kWaves];
  uint32_t wave_u[kWaves];
  uint32_t hist[256];
  int digit;
  int need;
};

// Block-wide exclusive prefix sum of one int per thread (thread order).
__device__ __forceinline__ int block_excl_scan(int v, int& total, Scratch& sc) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) sc.wave_i[wave] = incl;
  __syncthreads();
  int base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int t = sc.wave_i[w];
    base += (w < wave) ? t : 0;
    total += t;
  }
  __syncthreads();
  return base + incl - v;
}

// Block-wide exclusive prefix sum of one float per thread; fixed order.
__device__ __forceinline__ float block_excl_scan_f(float v, Scratch& sc) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) sc.wave_f[wave] = incl;
  __syncthreads();
  float base = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) base += (w < wave) ? sc.wave_f[w] : 0.f;
  __syncthreads();
  return base + (incl - v);
}

__device__ __forceinline__ float block_sum_f(float v, Scratch& sc) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) sc.wave_f[threadIdx.x >> 6] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t += sc.wave_f[w];
  __syncthreads();
  return t;
}

__device__ __forceinline__ int block_sum_i(int v, Scratch& sc) {
  int total;
  block_excl_scan(v, total, sc);
  return total;
}

__device__ __forceinline__ uint32_t block_max_u(uint32_t v, Scratch& sc) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, 64));
  if ((threadIdx.x & 63) == 0) sc.wave_u[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t = max(t, sc.wave_u[w]);
  __syncthreads();
  return t;
}

// "a ranks before b": higher key, then lower id.
__device__ __forceinline__ bool ranks_before(uint32_t ka, int ia, uint32_t kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

template <int EPT>
__global__ __launch_bounds__(kThreads) void select_kernel(
    const float* __restrict__ scores, int nblk, const int32_t* __restrict__ n_valid,
    float top_p, int k_max, int k_min, int n_sink, int n_recent, int P,
    int32_t* __restrict__ idx_out, int32_t* __restrict__ count_out,
    float* __restrict__ mass_out) {
  __shared__ Scratch sc;
  extern __shared__ uint32_t dyn[];  // [P] keys, [P] ids, [P] probs, [nblk/32+1] bitmap
  uint32_t* s_key = dyn;
  int* s_id = reinterpret_cast<int*>(dyn + P);
  float* s_p = reinterpret_cast<float*>(dyn + 2 * P);
  uint32_t* s_bits = dyn + 3 * P;

  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  int nv = n_valid ? n_valid[row] : nblk;
  nv = nv < 0 ? 0 : (nv > nblk ? nblk : nv);

  // Reserved tier (sink prefix + recency suffix of the valid blocks).
  const int sink_end = min(n_sink, nv);
  const int rec_start = max(0, nv - n_recent);
  const int n_reserved = sink_end + (nv - rec_start) - max(0, sink_end - rec_start);
  const int n_res = nv - n_reserved;
  const int cap = min(k_max - n_reserved, n_res);

  const float* srow = scores + (size_t)row * nblk;
  uint32_t key[EPT];
  float sv[EPT];
  bool cand[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = tid * EPT + e;
    cand[e] = j < nv && j >= sink_end && j < rec_start;
    sv[e] = cand[e] ? srow[j] : -INFINITY;
    key[e] = cand[e] ? order_key(sv[e]) : 0u;
  }
  for (int i = tid; i <= (nblk >> 5); i += kThreads) s_bits[i] = 0u;

  int n = 0;
  float mass = 0.f;
  if (cap > 0) {
    // ---- residual softmax statistics (Eq. select-nucleus) ----
    uint32_t kmax = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) kmax = max(kmax, key[e]);
    const float m = order_key_inv(block_max_u(kmax, sc));
    float pe[EPT];
    float zpart = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      pe[e] = cand[e] ? expf(sv[e] - m) : 0.f;
      zpart += pe[e];
    }
    const float Z = block_sum_f(zpart, sc);

    // ---- radix select of the cap-th largest key ----
    uint32_t prefix = 0, pmask = 0;
    int need = cap;
    if (cap < n_res) {
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        sc.hist[tid] = 0u;
        __syncthreads();
#pragma unroll
        for (int e = 0; e < EPT; ++e)
          if (cand[e] && (key[e] & pmask) == prefix)
            atomicAdd(&sc.hist[(key[e] >> shift) & 255u], 1u);
        __syncthreads();
        if (tid < 64) {
          // lane l holds digits 255-4l .. 252-4l (descending)
          int c[4], tot = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            c[i] = (int)sc.hist[255 - 4 * tid - i];
            tot += c[i];
          }
          int incl = tot;
#pragma unroll
          for (int off = 1; off < 64; off <<= 1) {
            const int o = __shfl_up(incl, off, 64);
            if (tid >= off) incl += o;
          }
          int before = incl - tot;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (before < need && need <= before + c[i]) {
              sc.digit = 255 - 4 * tid - i;
              sc.need = need - before;
            }
            before += c[i];
          }
        }
        __syncthreads();
        prefix |= (uint32_t)sc.digit << shift;
        pmask |= 255u << shift;
        need = sc.need;
        __syncthreads();
      }
    }
    const uint32_t thr = prefix;  // cap == n_res: every candidate passes (thr = 0)

    // ---- survivors: key > thr, or key == thr among the first `need` ids ----
    int n_eq = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) n_eq += (cand[e] && key[e] == thr) ? 1 : 0;
    int eq_total;
    int eq_rank = block_excl_scan(n_eq, eq_total, sc);
    bool sel[EPT];
    int n_sel = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool eq = cand[e] && key[e] == thr;
      sel[e] = cand[e] && (key[e] > thr || (eq && eq_rank < need));
      eq_rank += eq ? 1 : 0;
      n_sel += sel[e] ? 1 : 0;
    }
    int sel_total;
    int pos = block_excl_scan(n_sel, sel_total, sc);
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if (sel[e] && pos < P) {
        s_key[pos] = key[e];
        s_id[pos] = tid * EPT + e;
        s_p[pos] = pe[e];
        ++pos;
      }
    }
    for (int i = cap + tid; i < P; i += kThreads) {
      s_key[i] = 0u;
      s_id[i] = 0x7fffffff;
      s_p[i] = 0.f;
    }
    __syncthreads();

    // ---- bitonic sort of the P slots by (key desc, id asc) ----
    for (int kk = 2; kk <= P; kk <<= 1) {
      for (int jj = kk >> 1; jj > 0; jj >>= 1) {
        for (int i = tid; i < P; i += kThreads) {
          const int ixj = i ^ jj;
          if (ixj > i) {
            const uint32_t ka = s_key[i], kb = s_key[ixj];
            const int ia = s_id[i], ib = s_id[ixj];
            const bool a_first = ranks_before(ka, ia, kb, ib);
            const bool up = (i & kk) == 0;
            if (up != a_first) {
              s_key[i] = kb; s_key[ixj] = ka;
              s_id[i] = ib; s_id[ixj] = ia;
              const float pa = s_p[i];
              s_p[i] = s_p[ixj]; s_p[ixj] = pa;
            }
          }
        }
        __syncthreads();
      }
    }

    // ---- prefix mass in sorted order (thread t owns a contiguous run) ----
    const int per = (P + kThreads - 1) / kThreads;
    const int r0 = min(tid * per, P), r1 = min(r0 + per, P);
    float run = 0.f;
    for (int r = r0; r < r1; ++r) run += s_p[r];
    float acc = block_excl_scan_f(run, sc);
    const float pz = top_p * Z;
    int below = 0;
    for (int r = r0; r < r1; ++r) {
      acc += s_p[r];
      s_p[r] = acc;  // inclusive cumulative mass (unnormalised)
      below += (r < cap && acc < pz) ? 1 : 0;
    }
    const int n_below = block_sum_i(below, sc);  // also orders the s_p writes
    if (top_p >= 1.f)
      n = cap;
    else if (top_p <= 0.f)
      n = 0;
    else
      n = min(cap, n_below + 1);
    if (n_reserved + n < k_min) n = min(k_min - n_reserved, cap);
    mass = n > 0 ? s_p[n - 1] / Z : 0.f;
    for (int r = tid; r < n; r += kThreads) atomicOr(&s_bits[s_id[r] >> 5], 1u << (s_id[r] & 31));
  }
  __syncthreads();

  // ---- write S = reserved u nucleus in ascending block id ----
  bool fin[EPT];
  int n_fin = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = tid * EPT + e;
    const bool reserved = j < nv && (j < sink_end || j >= rec_start);
    fin[e] = reserved || (j < nv && ((s_bits[j >> 5] >> (j & 31)) & 1u));
    n_fin += fin[e] ? 1 : 0;
  }
  int total;
  int pos = block_excl_scan(n_fin, total, sc);
  int32_t* out = idx_out + (size_t)row * k_max;
#pragma unroll
  for (int e = 0; e < EPT; ++e)
    if (fin[e] && pos < k_max) out[pos++] = tid * EPT + e;
  for (int i = total + tid; i < k_max; i += kThreads) out[i] = -1;
  if (tid == 0) {
    count_out[row] = min(total, k_max);
    if (mass_out) mass_out[row] = mass;
  }
}

// ---------------------------------------------------------------------------
// Single-wavefront selection (rows of up to 4096 blocks, cap up to 512).
// Lane l owns the EPT consecutive block ids [l*EPT, (l+1)*EPT).  No workgroup
// barriers:
//  1. scores are loaded with coalesced loads (all issued before any use) and
//     transposed through LDS; candidates get order-preserving keys; residual
//     max m and Z = sum exp(s - m) with a fixed reduction tree;
//  2. if the cap C = min(k_max - |R|, |B_res|) binds, a radix select by count
//     (8-bit digits, LDS histogram, starting at the highest bit where the
//     candidate keys differ) finds the C-th largest key; equal keys at the
//     threshold go to the lowest block ids.  These C survivors are the only
//     blocks the rule can pick;
//  3. the survivors are bitonic-sorted in registers by (score desc, id asc),
//     packed as 64-bit keys, SPL = P / 64 slots per lane, lane exchanges via
//     DPP / swizzle / bpermute;
//  4. their probabilities are prefix-summed in that order; the nucleus is the
//     first prefix reaching top_p * Z, then capped and floored by k_min; the
//     chosen ids plus the reserved blocks are written in ascending order.

template <int EPT, int SPL>
__global__ __launch_bounds__(64) void select_wave_kernel(
    const float* __restrict__ scores, int nblk, const int32_t* __restrict__ n_valid,
    float top_p, int k_max, int k_min, int n_sink, int n_recent,
    int32_t* __restrict__ idx_out, int32_t* __restrict__ count_out,
    float* __restrict__ mass_out) {
  constexpr int kMaxBlocks = 64 * EPT;
  constexpr int P = 64 * SPL;
  constexpr float kLog2e = 1.4426950408889634f;
  __shared__ uint32_t hist[256];
  __shared__ uint32_t bits[(kMaxBlocks + 31) / 32];
  __shared__ float stage[kMaxBlocks];
  __shared__ uint64_t s_K[P];

  const int row = blockIdx.x;
  const int lane = threadIdx.x;
  int nv = n_valid ? n_valid[row] : nblk;
  nv = nv < 0 ? 0 : (nv > nblk ? nblk : nv);
  const int sink_end = min(n_sink, nv);
  const int rec_start = max(0, nv - n_recent);
  const int n_reserved = sink_end + (nv - rec_start) - max(0, sink_end - rec_start);
  const int n_res = nv - n_reserved;
  const int cap = min(k_max - n_reserved, n_res);

  // 1. Coalesced loads, all in flight at once, then transpose via LDS.
  const float* srow = scores + (size_t)row * nblk;
  float ld[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = e * 64 + lane;
    ld[e] = j < nv ? srow[j] : -INFINITY;
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) stage[e * 64 + lane] = ld[e];
  for (int i = lane; i < (kMaxBlocks + 31) / 32; i += 64) bits[i] = 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // Candidates get a non-zero order key; reserved blocks are remembered in a
  // per-lane bit word (VGPR) rather than as per-element lane masks.
  uint32_t key[EPT];
  float sv[EPT];
  uint64_t resv = 0;
  {
    const int j0 = lane * EPT;
    const int lo = max(sink_end - j0, 0), hi = min(rec_start - j0, EPT);  // candidate run
    const int vend = min(nv - j0, EPT);                                   // valid run
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool c = e >= lo && e < hi;
      sv[e] = stage[j0 + e];
      key[e] = c ? order_key(sv[e]) : 0u;  // 0 marks "not a candidate"
      resv |= (uint64_t)(e < vend && !c) << e;
    }
  }

  int n = 0;
  float mass = 0.f;
  if (cap > 0) {
    uint32_t kmax = 0u, kmin = 0xffffffffu;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      kmax = max(kmax, key[e]);
      if (key[e]) kmin = min(kmin, key[e]);
    }
    kmax = wave_max_u(kmax);
    kmin = wave_min_u(kmin);
    const float m = order_key_inv(kmax);
    float zl = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) zl += key[e] ? exp2f((sv[e] - m) * kLog2e) : 0.f;
    const float Z = wave_sum(zl);

    // ---- 2. radix select by count: the cap-th largest key ----
    uint32_t thr = 0u;  // cap == n_res: every candidate survives (keys > 0)
    int need = cap;
    if (cap < n_res) {
      const uint32_t diff = kmin ^ kmax;
      int shift = diff ? 32 - __builtin_clz(diff) : 0;  // low bits still to resolve
      uint32_t prefix = shift >= 32 ? 0u : (kmax >> shift) << shift;
      uint32_t pmask = shift >= 32 ? 0u : ~0u << shift;
      while (shift > 0) {
        const int width = shift < 8 ? shift : 8;
        shift -= width;
        const uint32_t dmask = (1u << width) - 1u;
        for (int i = lane; i < 256; i += 64) hist[i] = 0u;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int e = 0; e < EPT; ++e)
          if (key[e] && (key[e] & pmask) == prefix) atomicAdd(&hist[(key[e] >> shift) & dmask], 1u);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // lane l holds digits 255-4l .. 252-4l (descending)
        int c[4], tot = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          c[i] = (int)hist[255 - 4 * lane - i];
          tot += c[i];
        }
        const int incl = wave_incl_scan_i(tot);
        int before = incl - tot, digit = -1, left = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (before < need && need <= before + c[i]) {
            digit = 255 - 4 * lane - i;
            left = need - before;
          }
          before += c[i];
        }
        const unsigned long long who = __ballot(digit >= 0);
        const int src = __ffsll((long long)who) - 1;
        digit = __builtin_amdgcn_readlane(digit, src);
        need = __builtin_amdgcn_readlane(left, src);
        prefix |= (uint32_t)digit << shift;
        pmask |= dmask << shift;
      }
      thr = prefix;
    }

    // survivors (id order): key > thr, or key == thr among the first `need`
    int n_eq = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) n_eq += (key[e] && key[e] == thr) ? 1 : 0;
    int eq_rank = wave_incl_scan_i(n_eq) - n_eq;
    // Per-lane flag words live in VGPRs (bool arrays would become SGPR lane
    // masks and spill).
    uint64_t surv = 0;
    int n_sv = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool eq = key[e] && key[e] == thr;
      const bool sv_e = key[e] && (key[e] > thr || (eq && eq_rank < need));
      eq_rank += eq ? 1 : 0;
      n_sv += sv_e ? 1 : 0;
      surv |= (uint64_t)sv_e << e;
    }
    int pos = wave_incl_scan_i(n_sv) - n_sv;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if (((surv >> e) & 1u) && pos < P) {
        // (key desc, id asc) == packed value desc
        s_K[pos] = ((uint64_t)key[e] << 32) | (uint64_t)(0xffffffffu - (uint32_t)(lane * EPT + e));
        ++pos;
      }
    }
    for (int i = cap + lane; i < P; i += 64) s_K[i] = 0ull;  // padding sorts last
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- 3. sort the survivors ----
    uint64_t K[SPL];
#pragma unroll
    for (int t = 0; t < SPL; ++t) K[t] = s_K[lane * SPL + t];
    bitonic_desc<SPL>(K);

    // ---- 4. prefix mass in sorted order ----
    float cum[SPL];
    float run = 0.f;
#pragma unroll
    for (int t = 0; t < SPL; ++t) {
      const bool real = lane * SPL + t < cap;
      const float s = order_key_inv((uint32_t)(K[t] >> 32));
      run += real ? exp2f((s - m) * kLog2e) : 0.f;
      cum[t] = run;
    }
    const float base = wave_incl_scan_f(run) - run;
    const float pz = top_p * Z;
    int below = 0;
#pragma unroll
    for (int t = 0; t < SPL; ++t) {
      cum[t] += base;
      below += (lane * SPL + t < cap && cum[t] < pz) ? 1 : 0;
    }
    if (top_p >= 1.f)
      n = cap;
    else if (top_p <= 0.f)
      n = 0;
    else
      n = min(cap, wave_sum_i(below) + 1);
    if (n_reserved + n < k_min) n = min(k_min - n_reserved, cap);
#pragma unroll
    for (int t = 0; t < SPL; ++t) {
      if (lane * SPL + t < n) {
        const int id = (int)(0xffffffffu - (uint32_t)K[t]);
        atomicOr(&bits[id >> 5], 1u << (id & 31));
      }
    }
    if (n > 0) {
      const int ln = (n - 1) / SPL, tn = (n - 1) % SPL;
      float mine = 0.f;
#pragma unroll
      for (int t = 0; t < SPL; ++t) mine = t == tn ? cum[t] : mine;
      mass = readlane_f(mine, ln) / Z;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // ---- write S = reserved u chosen, ascending ----
  // chosen bits of this lane's run [lane*EPT, lane*EPT + EPT) (EPT <= 64)
  uint64_t fin = resv;
  {
    const int j0 = lane * EPT;
    if (EPT >= 32) {
#pragma unroll
      for (int w = 0; w < EPT / 32; ++w) fin |= (uint64_t)bits[j0 / 32 + w] << (32 * w);
    } else {
      fin |= (uint64_t)((bits[j0 >> 5] >> (j0 & 31)) & ((1u << EPT) - 1u));
    }
  }
  const int n_fin = __popcll(fin);
  const int incl = wave_incl_scan_i(n_fin);
  const int total = __builtin_amdgcn_readlane(incl, 63);
  int pos = incl - n_fin;
  int32_t* out = idx_out + (size_t)row * k_max;
#pragma unroll
  for (int e = 0; e < EPT; ++e)
    if (((fin >> e) & 1u) && pos < k_max) out[pos++] = lane * EPT + e;
  for (int i = total + lane; i < k_max; i += 64) out[i] = -1;
  if (lane == 0) {
    count_out[row] = min(total, k_max);
    if (mass_out) mass_out[row] = mass;
  }
}

// Workgroup selection kernel: one 256-thread workgroup per row (rows of
// 513 .. 8192 blocks, cap <= 512).
template <int EPT, int SPL>
__global__ __launch_bounds__(kSelWG) void select_wg_kernel(
    const float* __restrict__ scores, int nblk, const int32_t* __restrict__ n_valid,
    float top_p, int k_max, int k_min, int n_sink, int n_recent,
    int32_t* __restrict__ idx_out, int32_t* __restrict__ count_out,
    float* __restrict__ mass_out) {
  __shared__ SelWgSmem<EPT, SPL> sm;
  const int row = blockIdx.x;
  int nv = n_valid ? n_valid[row] : nblk;
  nv = nv < 0 ? 0 : (nv > nblk ? nblk : nv);
  SelRow r;
  if constexpr (EPT >= 16) {
    __shared__ alignas(16) float stage[kSelWG * EPT];
    r = select_row_core<EPT, SPL>(sm, StagedRowScores{scores + (size_t)row * nblk, stage}, nv,
                                  top_p, k_max, k_min, n_sink, n_recent);
  } else {
    r = select_row_core<EPT, SPL>(sm, RowScores{scores + (size_t)row * nblk}, nv, top_p, k_max,
                                  k_min, n_sink, n_recent);
  }
  int total;
  const int pos = sel_positions(sm, r.fin, total);
  sel_write<EPT>(idx_out + (size_t)row * k_max, count_out + row,
                 mass_out ? mass_out + row : nullptr, k_max, r.fin, pos, total, r.mass);
}

}  // namespace

hipError_t launch_select_blocks(const float* scores, int rows, int nblk, const int32_t* n_valid,
                                float top_p, int k_max, int k_min, int n_sink, int n_recent,
                                int32_t* idx, int32_t* count, float* nuc_mass, hipStream_t s) {
  int P = 1;
  const int cap = min(k_max, nblk);
  while (P < cap) P <<= 1;
  dim3 grid(rows);
  const int ept = nblk <= 64 ? 1 : nblk <= 128 ? 2 : nblk <= 256 ? 4 : nblk <= 512 ? 8
                : nblk <= 1024 ? 16 : nblk <= 2048 ? 32 : 64;
  const int spl = P <= 64 ? 1 : P / 64;
  // With top_p >= 1 every candidate up to the cap is kept, so the survivors
  // are never sorted and the survivor buffer (64 * SPL keys) does not bound
  // the cap: static top-K at any budget runs on the 512-key instantiation.
  const int spl_wg = top_p >= 1.f && spl > 8 ? 8 : spl;
  if (nblk > 512 && nblk <= 8192 && spl_wg <= 16) {
    const int e2 = nblk <= 1024 ? 4 : nblk <= 2048 ? 8 : nblk <= 4096 ? 16 : 32;
#define SPOT_SELECT_WG(E, S)                                                                    \
    if (e2 == E && spl_wg == S) {                                                             \
      hipLaunchKernelGGL((select_wg_kernel<E, S>), grid, dim3(kSelWG), 0, s, scores, nblk,    \
                         n_valid, top_p, k_max, k_min, n_sink, n_recent, idx, count,          \
                         nuc_mass);                                                           \
      return hipGetLastError();                                                                \
    }
#define SPOT_SELECT_WG_E(E)                                                      \
    SPOT_SELECT_WG(E, 1) SPOT_SELECT_WG(E, 2) SPOT_SELECT_WG(E, 4) SPOT_SELECT_WG(E, 8) \
    SPOT_SELECT_WG(E, 16)
    SPOT_SELECT_WG_E(4)
    SPOT_SELECT_WG_E(8)
    SPOT_SELECT_WG_E(16)
    SPOT_SELECT_WG_E(32)
#undef SPOT_SELECT_WG_E
#undef SPOT_SELECT_WG
  }
  if (nblk <= 4096 && spl <= 8) {
#define SPOT_SELECT_WAVE(E, S)                                                                  \
    if (ept == E && spl == S) {                                                               \
      hipLaunchKernelGGL((select_wave_kernel<E, S>), grid, dim3(64), 0, s, scores, nblk,      \
                         n_valid, top_p, k_max, k_min, n_sink, n_recent, idx, count,          \
                         nuc_mass);                                                           \
      return hipGetLastError();                                                                \
    }
#define SPOT_SELECT_WAVE_E(E) \
    SPOT_SELECT_WAVE(E, 1) SPOT_SELECT_WAVE(E, 2) SPOT_SELECT_WAVE(E, 4) SPOT_SELECT_WAVE(E, 8)
    SPOT_SELECT_WAVE_E(1)
    SPOT_SELECT_WAVE_E(2)
    SPOT_SELECT_WAVE_E(4)
    SPOT_SELECT_WAVE_E(8)
    SPOT_SELECT_WAVE_E(16)
    SPOT_SELECT_WAVE_E(32)
    SPOT_SELECT_WAVE_E(64)
#undef SPOT_SELECT_WAVE_E
#undef SPOT_SELECT_WAVE
  }
  const size_t shm = (size_t)(3 * P + (nblk >> 5) + 1) * 4;
  const int ept_needed = (nblk + kThreads - 1) / kThreads;
  dim3 block(kThreads);
#define SPOT_SELECT_CASE(E)                                                                   \
  if (ept_needed <= E) {                                                                    \
    hipLaunchKernelGGL((select_kernel<E>), grid, block, shm, s, scores, nblk, n_valid, top_p, \
                       k_max, k_min, n_sink, n_recent, P, idx, count, nuc_mass);            \
    return hipGetLastError();                                                                \
  }
  SPOT_SELECT_CASE(1)
  SPOT_SELECT_CASE(2)
  SPOT_SELECT_CASE(4)
  SPOT_SELECT_CASE(8)
  SPOT_SELECT_CASE(16)
  SPOT_SELECT_CASE(32)
  SPOT_SELECT_CASE(64)
#undef SPOT_SELECT_CASE
  return hipErrorInvalidValue;
}

}  // namespace spot
