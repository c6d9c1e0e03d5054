// Dual top-p / top-K block selection (paper Section 2.3, Eqs. select-topk,
// select-nucleus and select-topp) with a cap k_max on the set size.
//
// Rows of up to 4096 blocks use the single-wavefront kernel further down.
// Larger rows use one workgroup (256 threads) per row; thread t owns the EPT
// consecutive block ids [t*EPT, (t+1)*EPT) in registers.  Per row:
//  1. reserved blocks (sink prefix, recency suffix) are set aside; the
//     residual candidates get an order-preserving 32-bit key of their score;
//  2. residual softmax statistics: max and Z = sum exp(s - max) with a fixed
//     reduction tree (deterministic);
//  3. only the best C = min(k_max - |R|, |B_res|) candidates can ever be
//     chosen, so a fixed 4-pass 8-bit radix select finds the C-th largest key;
//     equal keys at the threshold are taken in ascending block id;
//  4. the C survivors are bitonic-sorted in LDS by (score desc, id asc), their
//     probabilities prefix-summed in that order (fixed tree, FP32), and the
//     nucleus length n is the first prefix reaching top_p * Z, then capped
//     and floored by k_min;
//  5. reserved + the first n survivors are written in ascending block id.
#include "spot_internal.h"

namespace spot {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float order_key_inv(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

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
// One wavefront per row (rows of up to 4096 blocks).  Lane l owns the EPT
// consecutive block ids [l*EPT, (l+1)*EPT).  No workgroup barriers and no sort:
//  1. candidates' order keys, residual max m and Z = sum exp(s - m);
//  2. if the cap C = min(k_max - |R|, |B_res|) binds, a radix select by count
//     (8-bit digits, LDS histogram, starting at the highest bit where the
//     candidate keys differ) finds the C-th largest key; equal keys at the
//     threshold are taken in ascending block id.  These C survivors are the
//     only blocks the rule can pick;
//  3. the survivors are compacted (id order) and the nucleus length is found
//     by bisection on the key: the largest threshold T whose mass
//     sum_{key >= T} exp(s - m) still reaches top_p * Z, plus as many blocks
//     tied at T (lowest ids first) as are needed to reach it;
//  4. the k_min floor and the cap give the final n; the top-n survivors (by
//     count bisection, ties by id) plus the reserved blocks are written in
//     ascending block id.
template <int EPT>
__global__ __launch_bounds__(64) void select_wave_kernel(
    const float* __restrict__ scores, int nblk, const int32_t* __restrict__ n_valid,
    float top_p, int k_max, int k_min, int n_sink, int n_recent, int P,
    int32_t* __restrict__ idx_out, int32_t* __restrict__ count_out,
    float* __restrict__ mass_out) {
  constexpr int kMaxBlocks = 64 * EPT;
  __shared__ uint32_t hist[256];
  __shared__ uint32_t bits[kMaxBlocks / 32];
  extern __shared__ uint32_t dyn[];  // staging [kMaxBlocks] | surv key [P] | id [P] | e [P]
  float* stage = reinterpret_cast<float*>(dyn);
  uint32_t* s_key = dyn + kMaxBlocks;
  int* s_id = reinterpret_cast<int*>(s_key + P);
  float* s_e = reinterpret_cast<float*>(s_id + P);

  const int row = blockIdx.x;
  const int lane = threadIdx.x;
  int nv = n_valid ? n_valid[row] : nblk;
  nv = nv < 0 ? 0 : (nv > nblk ? nblk : nv);
  const int sink_end = min(n_sink, nv);
  const int rec_start = max(0, nv - n_recent);
  const int n_reserved = sink_end + (nv - rec_start) - max(0, sink_end - rec_start);
  const int n_res = nv - n_reserved;
  const int cap = min(k_max - n_reserved, n_res);

  // Coalesced load into LDS, then each lane takes its consecutive run.
  const float* srow = scores + (size_t)row * nblk;
  for (int j = lane; j < nv; j += 64) stage[j] = srow[j];
  for (int i = lane; i < kMaxBlocks / 32; i += 64) bits[i] = 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  uint32_t key[EPT];
  float sv[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = lane * EPT + e;
    const bool c = j < nv && j >= sink_end && j < rec_start;
    sv[e] = c ? stage[j] : -INFINITY;
    key[e] = c ? order_key(sv[e]) : 0u;  // 0 marks "not a candidate"
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
    float pe[EPT];
    float zl = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      pe[e] = key[e] ? exp2f((sv[e] - m) * 1.4426950408889634f) : 0.f;
      zl += pe[e];
    }
    const float Z = wave_sum(zl);

    // ---- 2. radix select by count: the cap-th largest key ----
    uint32_t thr = 0u;  // cap == n_res: every candidate survives (keys > 0)
    int need = cap;
    if (cap < n_res) {
      const uint32_t diff = kmin ^ kmax;
      int shift = diff ? 32 - __builtin_clz(diff) : 0;   // bits still to resolve
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

    // survivors in id order: key > thr, or key == thr among the first `need`
    int n_eq = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) n_eq += (key[e] && key[e] == thr) ? 1 : 0;
    int eq_rank = wave_incl_scan_i(n_eq) - n_eq;
    bool surv[EPT];
    int n_sv = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const bool eq = key[e] && key[e] == thr;
      surv[e] = key[e] && (key[e] > thr || (eq && eq_rank < need));
      eq_rank += eq ? 1 : 0;
      n_sv += surv[e] ? 1 : 0;
    }
    int pos = wave_incl_scan_i(n_sv) - n_sv;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      if (surv[e] && pos < P) {
        s_key[pos] = key[e];
        s_id[pos] = lane * EPT + e;
        s_e[pos] = pe[e];
        ++pos;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- 3. work on the cap survivors, SP consecutive ones per lane ----
    const int SP = (cap + 63) / 64;
    const int i0 = min(lane * SP, cap), i1 = min(i0 + SP, cap);
    auto mass_ge = [&](uint32_t T) {
      float part = 0.f;
      for (int i = i0; i < i1; ++i) part += s_key[i] >= T ? s_e[i] : 0.f;
      return wave_sum(part);
    };
    auto count_ge = [&](uint32_t T) {
      int part = 0;
      for (int i = i0; i < i1; ++i) part += s_key[i] >= T ? 1 : 0;
      return wave_sum_i(part);
    };
    // Largest T with f(T) >= target, for f non-increasing in T (bisection).
    const float pz = top_p * Z;
    int n_target;
    if (top_p >= 1.f) {
      n_target = cap;
    } else if (top_p <= 0.f) {
      n_target = 0;
    } else if (mass_ge(0u) < pz) {
      n_target = cap;  // the nucleus would need more than the cap allows
    } else {
      uint32_t T = 0u;
      for (int bit = 31; bit >= 0; --bit) {
        const uint32_t Tc = T | (1u << bit);
        if (mass_ge(Tc) >= pz) T = Tc;
      }
      const float mass_gt = T == 0xffffffffu ? 0.f : mass_ge(T + 1u);
      const int n_gt = T == 0xffffffffu ? 0 : count_ge(T + 1u);
      const int n_eqT = count_ge(T) - n_gt;
      float eT = 0.f;
      for (int i = i0; i < i1; ++i) eT = s_key[i] == T ? s_e[i] : eT;
      eT = wave_max(eT);
      int t = 1;
      while (t < n_eqT && mass_gt + (float)t * eT < pz) ++t;
      n_target = n_gt + t;
    }
    n = min(n_target, cap);
    if (n_reserved + n < k_min) n = min(k_min - n_reserved, cap);

    // ---- 4. the top-n survivors (count bisection, ties by lowest id) ----
    uint32_t T2 = 0u;
    int need2 = n;
    if (n < cap) {
      for (int bit = 31; bit >= 0; --bit) {
        const uint32_t Tc = T2 | (1u << bit);
        if (count_ge(Tc) >= n) T2 = Tc;
      }
      need2 = n - (T2 == 0xffffffffu ? 0 : count_ge(T2 + 1u));
    }
    int q_eq = 0;
    for (int i = i0; i < i1; ++i) q_eq += s_key[i] == T2 ? 1 : 0;
    int r = wave_incl_scan_i(q_eq) - q_eq;
    float ml = 0.f;
    for (int i = i0; i < i1; ++i) {
      const bool eq = s_key[i] == T2;
      const bool take = n > 0 && (s_key[i] > T2 || (eq && r < need2));
      r += eq ? 1 : 0;
      if (take) {
        atomicOr(&bits[s_id[i] >> 5], 1u << (s_id[i] & 31));
        ml += s_e[i];
      }
    }
    mass = n > 0 ? wave_sum(ml) / Z : 0.f;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // ---- write S = reserved u chosen, ascending ----
  bool fin[EPT];
  int n_fin = 0;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = lane * EPT + e;
    const bool reserved = j < nv && (j < sink_end || j >= rec_start);
    fin[e] = reserved || (j < nv && ((bits[j >> 5] >> (j & 31)) & 1u));
    n_fin += fin[e] ? 1 : 0;
  }
  const int incl = wave_incl_scan_i(n_fin);
  const int total = __builtin_amdgcn_readlane(incl, 63);
  int pos = incl - n_fin;
  int32_t* out = idx_out + (size_t)row * k_max;
#pragma unroll
  for (int e = 0; e < EPT; ++e)
    if (fin[e] && pos < k_max) out[pos++] = lane * EPT + e;
  for (int i = total + lane; i < k_max; i += 64) out[i] = -1;
  if (lane == 0) {
    count_out[row] = min(total, k_max);
    if (mass_out) mass_out[row] = mass;
  }
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
  const size_t shm_w = (size_t)(64 * ept + 3 * P) * 4;
  if (nblk <= 4096 && shm_w <= 56 * 1024) {
#define SPOT_SELECT_WAVE(E)                                                                     \
    if (ept == E) {                                                                           \
      hipLaunchKernelGGL((select_wave_kernel<E>), grid, dim3(64), shm_w, s, scores, nblk,     \
                         n_valid, top_p, k_max, k_min, n_sink, n_recent, P, idx, count,       \
                         nuc_mass);                                                           \
      return hipGetLastError();                                                                \
    }
    SPOT_SELECT_WAVE(1)
    SPOT_SELECT_WAVE(2)
    SPOT_SELECT_WAVE(4)
    SPOT_SELECT_WAVE(8)
    SPOT_SELECT_WAVE(16)
    SPOT_SELECT_WAVE(32)
    SPOT_SELECT_WAVE(64)
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
