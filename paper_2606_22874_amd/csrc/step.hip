// Fused decode step: selector scoring, block selection and block-sparse
// attention of every sequence in one launch (paper Section 2: score every KV
// block, pick blocks by the dual top-p / top-K rule with sink and recency
// reserved, attend to the chosen blocks only).
//
// Separate launches pay a kernel boundary (completion, cache maintenance and
// dispatch of the next grid, a few microseconds each) twice per step, and the
// attention grid only starts fetching once its dispatch is done.  Here one
// grid of n_pairs * n_slot workgroups runs
//   1. scoring: the first kMaxScorers workgroups of each row (workgroup i
//      serves row i % batch) score a contiguous run of its blocks; each
//      score also goes out as a self-flagging record word;
//   2. selection: workgroup r (a scorer of row r) polls the row's score
//      records (each thread its own ids, as they land), clears them, selects
//      the row (the workgroup core shared with the stand-alone kernel) and
//      publishes the block list as record words, one copy per KV head;
//   3. attention: every workgroup polls the list records of its (sequence,
//      KV head) share, clears them and runs its (pair, slot) of the split-KV
//      decode (shared core).
// A record word is nonzero once written and its reader sets it back to zero,
// so a hand-off costs one round trip to the device coherence point, there
// are no flags or contended atomics, and the workspace is all zero again
// when the launch ends.
//
// The waits need every workgroup of the grid to be resident at once: the
// launcher sizes the grid to the occupancy-derived capacity of the device
// (workgroups that cannot start right away because other work holds CUs
// start when it drains, since nothing else depends on this grid).  Each wait
// is also bounded in time (kWaitTicks of the 100 MHz real-time counter), so
// a wait can never hang the device; an expired wait lets the workgroup
// finish with whatever the records held.
#include "decode_core.h"
#include "score_core.h"
#include "select_core.h"

namespace spot {
namespace {

using namespace dec;

constexpr int kStepG = 4;                 // GQA group of the fused path (256 threads)
constexpr int kScoreRun = 8;              // blocks per scoring call of one wave (the
                                          // stand-alone kernel's run: same code, same bits)
constexpr int kMaxScorers = 64;           // scoring workgroups per row
constexpr int kRecRow = 4096;             // score record words per row (the fused maximum)
constexpr uint64_t kWaitTicks = 20000000; // 0.2 s of the 100 MHz real-time counter

struct StepArgs {
  const uint16_t* q_sel;
  const float* w;
  const uint8_t* k_sel;
  const uint8_t* k_scale;
  const int32_t* n_valid;
  int kfmt, lph;
  float top_p;
  int k_max, k_min, n_sink, n_recent;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* seq_len;
  int batch, h_q, h_kv, l_cap, nblk, n_slot;
  float scale_log2;
  float* scores;
  int32_t* idx;
  int32_t* count;
  float* mass;
  uint16_t* out;
  float* lse;
  float* ws_o;
  float* ws_ml;
  unsigned* pair_cnt;   // [batch * h_kv] split completion (decode merge)
  uint32_t* srec;       // [batch, kRecRow] score records
  uint32_t* irec;       // [batch, h_kv, rec_len] block list records
  int rec_len;          // min(k_max, nblk)
};

__device__ __forceinline__ uint64_t now() { return __builtin_amdgcn_s_memrealtime(); }

template <typename W>
__device__ __forceinline__ W load_rec(const W* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename W>
__device__ __forceinline__ void store_rec(W* p, W v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Score source of the selector: thread t polls the records of its own ids
// [j0, j0 + EPT) until every valid one is written (two words per load; the
// words past nv stay zero all launch).  clear_scores() zeroes them again
// once the selection is done: a store issued here would hold up the
// selection's next barrier until it completed.
struct PolledScores {
  uint32_t* rec;   // the row's kRecRow record words
  template <int EPT>
  __device__ __forceinline__ void operator()(float (&sv)[EPT], int j0, int nv) const {
    uint32_t wd[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) wd[e] = 0u;
    const uint64_t deadline = now() + kWaitTicks;
    for (;;) {
      bool all = true;
      if constexpr (EPT % 2 == 0) {
#pragma unroll
        for (int e = 0; e < EPT; e += 2) {
          const bool need = (j0 + e < nv && wd[e] == 0u) || (j0 + e + 1 < nv && wd[e + 1] == 0u);
          if (need) {
            const uint64_t x = load_rec(reinterpret_cast<const uint64_t*>(rec + j0 + e));
            wd[e] = (uint32_t)x;
            wd[e + 1] = (uint32_t)(x >> 32);
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < EPT; ++e)
          if (j0 + e < nv && wd[e] == 0u) wd[e] = load_rec(rec + j0 + e);
      }
#pragma unroll
      for (int e = 0; e < EPT; ++e) all = all && (j0 + e >= nv || wd[e] != 0u);
      if (all || now() > deadline) break;
      __builtin_amdgcn_s_sleep(1);
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) sv[e] = j0 + e < nv ? rec_value(wd[e]) : -INFINITY;
  }
};

// Clears thread t's score records [j0, j0 + EPT) below nv (see PolledScores).
template <int EPT>
__device__ __forceinline__ void clear_scores(uint32_t* rec, int j0, int nv) {
  if constexpr (EPT % 2 == 0) {
#pragma unroll
    for (int e = 0; e < EPT; e += 2)
      if (j0 + e < nv) store_rec(reinterpret_cast<uint64_t*>(rec + j0 + e), (uint64_t)0);
  } else {
#pragma unroll
    for (int e = 0; e < EPT; ++e)
      if (j0 + e < nv) store_rec(rec + j0 + e, 0u);
  }
}

// Block list source of an attention workgroup: entries slot, slot + n_slot,
// ... of its (sequence, KV head) copy of the list records (the stand-alone
// decode's share of the same list, in the same order), polled until written.
// Called by wave 0; clear_list() zeroes the same words after the attention
// (a store here would hold up the next workgroup barrier).
struct PolledList {
  const uint32_t* irec;
  int h_kv, rec_len;
  __device__ __forceinline__ int operator()(int* ids, int b, int g, int slot, int n_slot,
                                            int nb_valid) const {
    const int lane = __lane_id();
    uint32_t* rec = const_cast<uint32_t*>(irec) + ((size_t)b * h_kv + g) * rec_len;
    const uint64_t deadline = now() + kWaitTicks;
    int cnt = 0;
    for (int base = slot; base < rec_len; base += 64 * n_slot) {
      const int e = base + lane * n_slot;
      uint32_t wd = e < rec_len ? 0u : 0xffffffffu;
      for (;;) {
        if (wd == 0u) wd = load_rec(rec + e);
        if (__ballot(wd == 0u) == 0ull || now() > deadline) break;
        __builtin_amdgcn_s_sleep(1);
      }
      const int j = wd == 0u || wd == 0xffffffffu ? -1 : (int)(wd - 1u);
      cnt = append_ids(ids, cnt, j, nb_valid);
    }
    return min(cnt, kMaxIds);
  }
};

__device__ __forceinline__ void clear_list(uint32_t* irec, int h_kv, int rec_len, int b, int g,
                                           int slot, int n_slot) {
  uint32_t* rec = irec + ((size_t)b * h_kv + g) * rec_len;
  for (int e = slot + __lane_id() * n_slot; e < rec_len; e += 64 * n_slot) store_rec(rec + e, 0u);
}

template <int KFMT, int LPH>
__device__ __forceinline__ void score_run(const StepArgs& a, int row, int nv, int j0, int jend,
                                          int lane) {
  score_blocks<KFMT, LPH, kScoreRun>(a.q_sel, a.w, a.k_sel, a.k_scale, row, row, a.nblk, nv, j0,
                                     jend, a.scores, a.srec + (size_t)row * kRecRow, lane);
}

__device__ __forceinline__ void score_run_rt(const StepArgs& a, int row, int nv, int j0, int jend,
                                             int lane) {
  if (a.lph == 8) {
    switch (a.kfmt) {
      case SPOT_KFMT_BF16: score_run<SPOT_KFMT_BF16, 8>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_INT4_G32: score_run<SPOT_KFMT_INT4_G32, 8>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_INT8_G32: score_run<SPOT_KFMT_INT8_G32, 8>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_MXFP8_G32:
        score_run<SPOT_KFMT_MXFP8_G32, 8>(a, row, nv, j0, jend, lane);
        break;
      default: score_run<SPOT_KFMT_MXFP4_G32, 8>(a, row, nv, j0, jend, lane); break;
    }
  } else {
    switch (a.kfmt) {
      case SPOT_KFMT_BF16: score_run<SPOT_KFMT_BF16, 16>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_INT4_G32: score_run<SPOT_KFMT_INT4_G32, 16>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_INT8_G32: score_run<SPOT_KFMT_INT8_G32, 16>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_MXFP8_G32:
        score_run<SPOT_KFMT_MXFP8_G32, 16>(a, row, nv, j0, jend, lane);
        break;
      default: score_run<SPOT_KFMT_MXFP4_G32, 16>(a, row, nv, j0, jend, lane); break;
    }
  }
}

template <int EPT, int SPL>
__global__ __launch_bounds__(64 * kStepG, 2) void step_kernel(StepArgs a) {
  __shared__ union {
    SelWgSmem<EPT, SPL> sel;
    DecodeSmem<kStepG> dec;
  } sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wg = blockIdx.x, nwg = gridDim.x;

  // ---- 1. scoring: row r = wg % B, by its first n_sc workgroups
  const int B = a.batch;
  const int r = wg % B, c = wg / B;
  const int n_sc = min(kMaxScorers, (nwg - r + B - 1) / B);   // scorers of row r
  int nv = a.n_valid ? a.n_valid[r] : a.nblk;
  nv = nv < 0 ? 0 : (nv > a.nblk ? a.nblk : nv);
  if (c < n_sc) {
    const int per = (a.nblk + n_sc - 1) / n_sc;
    const int jb = c * per, je = min(jb + per, a.nblk);
    for (int j0 = jb + wave * kScoreRun; j0 < je; j0 += kStepG * kScoreRun)
      score_run_rt(a, r, nv, j0, je, lane);
  }

  // ---- 2. selection of row wg by workgroup wg (wg < B is scorer 0 of it)
  if (wg < B) {
    select_row_wg<EPT, SPL>(sm.sel, PolledScores{a.srec + (size_t)wg * kRecRow}, a.nblk, nv,
                            a.top_p, a.k_max, a.k_min, a.n_sink, a.n_recent,
                            a.idx + (size_t)wg * a.k_max, a.count + wg,
                            a.mass ? a.mass + wg : nullptr,
                            IdRecords{a.irec + (size_t)wg * a.h_kv * a.rec_len, a.rec_len,
                                      a.h_kv});
    clear_scores<EPT>(a.srec + (size_t)wg * kRecRow, tid * EPT, nv);
    // The selection's LDS is reused below: every wave's LDS accesses are
    // done; no wait for the stores in flight.
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
  }

  // ---- 3. attention for (pair, slot) on the published block list
  const int pair = wg / a.n_slot, slot = wg % a.n_slot;
  decode_body<kStepG, false>(sm.dec, PolledList{a.irec, a.h_kv, a.rec_len}, pair, slot, a.q, a.k,
                             a.v, a.seq_len, a.h_q, a.h_kv, a.l_cap, a.scale_log2, a.n_slot,
                             a.ws_o, a.ws_ml, a.pair_cnt, a.out, a.lse);
  if (wave == 0) clear_list(a.irec, a.h_kv, a.rec_len, pair / a.h_kv, pair % a.h_kv, slot, a.n_slot);
}

// Workgroups of one step kernel that can be resident at once (per CU times
// the CU count), queried once per device and instantiation and cached.
template <int EPT, int SPL>
int step_capacity() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cached[dev] > 0) return cached[dev];
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(&step_kernel<EPT, SPL>), 64 * kStepG, 0) !=
      hipSuccess)
    return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  cached[dev] = per_cu * cus;
  return cached[dev];
}

template <int EPT, int SPL>
hipError_t launch_step_t(StepArgs& a, int n_pairs, int n_slot_max, hipStream_t s) {
  const int cap = step_capacity<EPT, SPL>();
  if (cap < n_pairs) return hipErrorCooperativeLaunchTooLarge;
  a.n_slot = n_slot_max < cap / n_pairs ? n_slot_max : cap / n_pairs;
  hipLaunchKernelGGL((step_kernel<EPT, SPL>), dim3(n_pairs * a.n_slot), dim3(64 * kStepG), 0, s,
                     a);
  return hipGetLastError();
}

}  // namespace

// Workspace: the split-decode partials and pair counters, then (16-byte
// aligned) the score records [batch, kRecRow] and the list records
// [batch, h_kv, min(k_max, nblk)] (sized for k_max).
static size_t step_records_offset(int batch, int h_q, int h_kv, int d, int k_max) {
  return (decode_workspace_bytes(batch, h_q, h_kv, d, k_max) + 15) & ~(size_t)15;
}
size_t step_workspace_bytes(int batch, int h_q, int h_kv, int d, int k_max) {
  return step_records_offset(batch, h_q, h_kv, d, k_max) +
         (size_t)batch * (kRecRow + (size_t)h_kv * k_max) * sizeof(uint32_t);
}

bool step_fusable(int h_q, int h_kv, int nblk, int k_max) {
  if (h_q != kStepG * h_kv || nblk < 1 || nblk > kRecRow) return false;
  int P = 1;
  const int cap = k_max < nblk ? k_max : nblk;
  while (P < cap) P <<= 1;
  return P <= 512;
}

hipError_t launch_decode_step(const void* q_sel, const float* w, const void* k_sel,
                              const void* k_scale, int kfmt, int d_s, const int32_t* n_valid,
                              float top_p, int k_max, int k_min, int n_sink, int n_recent,
                              const void* q, const void* k, const void* v,
                              const int32_t* seq_len, int batch, int h_q, int h_kv, int l_cap,
                              float sm_scale, float* scores, int32_t* idx, int32_t* count,
                              float* nuc_mass, void* out, float* lse, void* ws, hipStream_t s) {
  StepArgs a;
  a.q_sel = static_cast<const uint16_t*>(q_sel);
  a.w = w;
  a.k_sel = static_cast<const uint8_t*>(k_sel);
  a.k_scale = static_cast<const uint8_t*>(k_scale);
  a.n_valid = n_valid;
  a.kfmt = kfmt;
  a.lph = d_s / 8;
  a.top_p = top_p;
  a.k_max = k_max;
  a.k_min = k_min;
  a.n_sink = n_sink;
  a.n_recent = n_recent;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.seq_len = seq_len;
  a.batch = batch;
  a.h_q = h_q;
  a.h_kv = h_kv;
  a.l_cap = l_cap;
  a.nblk = l_cap / kBlk;
  a.scale_log2 = sm_scale * kLog2e;
  a.scores = scores;
  a.idx = idx;
  a.count = count;
  a.mass = nuc_mass;
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse;
  const int n_pairs = batch * h_kv;
  const int n_slot_max = decode_num_splits(batch, h_kv, k_max, kStepG);
  a.ws_o = static_cast<float*>(ws);
  a.ws_ml = a.ws_o + (size_t)batch * h_q * n_slot_max * kD;
  a.pair_cnt = reinterpret_cast<unsigned*>(a.ws_ml + (size_t)batch * h_q * n_slot_max * 2);
  a.srec = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) +
                                       step_records_offset(batch, h_q, h_kv, kD, k_max));
  a.irec = a.srec + (size_t)batch * kRecRow;
  a.rec_len = k_max < a.nblk ? k_max : a.nblk;
  // The partial buffers are laid out for n_slot_max; a smaller n_slot (when
  // fewer workgroups fit) uses a prefix of each head's run, indexed with the
  // actual n_slot -- the layout is [B, h_q, n_slot] either way.
  int P = 1;
  const int cap = k_max < a.nblk ? k_max : a.nblk;
  while (P < cap) P <<= 1;
  const int spl = P <= 64 ? 1 : P / 64;
  const int ept = a.nblk <= 256 ? 1 : a.nblk <= 512 ? 2 : a.nblk <= 1024 ? 4
                : a.nblk <= 2048 ? 8 : 16;
#define SPOT_STEP_CASE(E, S) \
  if (ept == E && spl == S) return launch_step_t<E, S>(a, n_pairs, n_slot_max, s);
#define SPOT_STEP_E(E) SPOT_STEP_CASE(E, 1) SPOT_STEP_CASE(E, 2) SPOT_STEP_CASE(E, 4) \
  SPOT_STEP_CASE(E, 8)
  SPOT_STEP_E(1)
  SPOT_STEP_E(2)
  SPOT_STEP_E(4)
  SPOT_STEP_E(8)
  SPOT_STEP_E(16)
#undef SPOT_STEP_E
#undef SPOT_STEP_CASE
  return hipErrorInvalidValue;
}

}  // namespace spot
