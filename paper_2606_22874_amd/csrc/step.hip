// Fused decode step: selector scoring, block selection and block-sparse
// attention of every sequence in one cooperative launch (paper Section 2:
// score every KV block, pick blocks by the dual top-p / top-K rule with sink
// and recency reserved, attend to the chosen blocks only).
//
// Separate launches pay a kernel boundary (completion, cache maintenance and
// dispatch of the next grid, a few microseconds each) twice per step, and the
// attention grid only starts fetching once its dispatch is done.  Here one
// grid of n_pairs * n_slot workgroups runs
//   1. scoring: the first kMaxScorers workgroups of each row (workgroup i
//      serves row i % batch) score a contiguous run of its blocks with
//      device-scope stores, then raise their own done flag;
//   2. selection: workgroup r (a scorer of row r) waits for the row's done
//      flags, clears them, selects the row (the workgroup core shared with
//      the stand-alone kernel, device-scope loads and stores) and raises the
//      row's ready flag;
//   3. attention: every workgroup takes its (pair, slot) of the split-KV
//      decode (shared core) once its sequence's ready flag is up.
// One flag per writer keeps the hand-offs free of contended atomics (a
// counter bumped by every scorer serialises at the memory).  The last
// workgroup of each sequence clears the ready flag, so all flags and counters
// are zero again when the launch ends.
//
// The waits need every workgroup of the grid to be resident at once: the
// launcher sizes the grid to the occupancy-derived capacity of the device
// (workgroups that cannot start right away because other work holds CUs
// start when it drains, since nothing else depends on this grid).  Each wait
// is also bounded in time (kWaitTicks of the 100 MHz real-time counter), so
// a wait can never hang the device; an expired wait lets the workgroup
// finish with whatever the flag guarded.
#include "decode_core.h"
#include "score_core.h"
#include "select_core.h"

namespace spot {
namespace {

using namespace dec;

constexpr int kStepG = 4;                 // GQA group of the fused path (256 threads)
constexpr int kScoreRun = 8;              // blocks per scoring call of one wave (the
                                          // stand-alone kernel's run: same code, same bits)
constexpr int kMaxScorers = 64;           // scoring workgroups per row (<= 64: one wave polls)
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
  unsigned* done;       // [batch, kMaxScorers] scorer finished
  unsigned* ready;      // [batch] selection published
  unsigned* row_done;   // [batch] pairs merged
};

__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

template <int KFMT, int LPH>
__device__ __forceinline__ void score_run(const StepArgs& a, int row, int nv, int j0, int jend,
                                          int lane) {
  score_blocks<KFMT, LPH, kScoreRun, true>(a.q_sel, a.w, a.k_sel, a.k_scale, row, row, a.nblk,
                                           nv, j0, jend, a.scores, lane);
}

__device__ __forceinline__ void score_run_rt(const StepArgs& a, int row, int nv, int j0, int jend,
                                             int lane) {
  if (a.lph == 8) {
    switch (a.kfmt) {
      case SPOT_KFMT_BF16: score_run<SPOT_KFMT_BF16, 8>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_INT4_G32: score_run<SPOT_KFMT_INT4_G32, 8>(a, row, nv, j0, jend, lane); break;
      default: score_run<SPOT_KFMT_MXFP4_G32, 8>(a, row, nv, j0, jend, lane); break;
    }
  } else {
    switch (a.kfmt) {
      case SPOT_KFMT_BF16: score_run<SPOT_KFMT_BF16, 16>(a, row, nv, j0, jend, lane); break;
      case SPOT_KFMT_INT4_G32: score_run<SPOT_KFMT_INT4_G32, 16>(a, row, nv, j0, jend, lane); break;
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
    wait_vm();  // this thread's score stores are visible device-wide
    __syncthreads();
    if (tid == 0)
      __hip_atomic_store(&a.done[r * kMaxScorers + c], 1u, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }

  // ---- 2. selection of row wg by workgroup wg (wg < B is scorer 0 of it)
  if (wg < B) {
    if (wave == 0) {
      const uint64_t deadline = __builtin_amdgcn_s_memrealtime() + kWaitTicks;
      unsigned* flag = &a.done[wg * kMaxScorers + lane];
      for (;;) {
        const bool up = lane >= n_sc ||
                        __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
        if (__ballot(!up) == 0 || __builtin_amdgcn_s_memrealtime() > deadline) break;
        __builtin_amdgcn_s_sleep(2);
      }
      if (lane < n_sc) __hip_atomic_store(flag, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    select_row_wg<EPT, SPL, true>(sm.sel, a.scores + (size_t)wg * a.nblk, a.nblk, nv, a.top_p,
                                  a.k_max, a.k_min, a.n_sink, a.n_recent,
                                  a.idx + (size_t)wg * a.k_max, a.count + wg,
                                  a.mass ? a.mass + wg : nullptr);
    wait_vm();
    __syncthreads();
    if (tid == 0) __hip_atomic_store(&a.ready[wg], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // ---- 3. attention for (pair, slot) once the sequence's selection is out
  const int pair = wg / a.n_slot, slot = wg % a.n_slot;
  const int b = pair / a.h_kv;
  if (tid == 0) {
    const uint64_t deadline = __builtin_amdgcn_s_memrealtime() + kWaitTicks;
    while (__hip_atomic_load(&a.ready[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u &&
           __builtin_amdgcn_s_memrealtime() <= deadline)
      __builtin_amdgcn_s_sleep(8);
  }
  __syncthreads();
  const bool merged = decode_body<kStepG, false, true>(
      sm.dec, pair, slot, a.q, a.k, a.v, a.seq_len, a.idx, a.count, a.k_max, a.h_q, a.h_kv,
      a.l_cap, a.scale_log2, a.n_slot, a.ws_o, a.ws_ml, a.pair_cnt, a.out, a.lse);
  if (merged && tid == 0) {
    const unsigned prev =
        __hip_atomic_fetch_add(&a.row_done[b], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == (unsigned)(a.h_kv - 1)) {
      __hip_atomic_store(&a.row_done[b], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ready[b], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
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

size_t step_workspace_bytes(int batch, int h_q, int h_kv, int d, int k_max) {
  return decode_workspace_bytes(batch, h_q, h_kv, d, k_max) +
         (size_t)batch * (kMaxScorers + 2) * sizeof(unsigned);
}

bool step_fusable(int h_q, int h_kv, int nblk, int k_max) {
  if (h_q != kStepG * h_kv || nblk < 1 || nblk > 4096) return false;
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
  a.done = a.pair_cnt + n_pairs;
  a.ready = a.done + (size_t)batch * kMaxScorers;
  a.row_done = a.ready + batch;
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
