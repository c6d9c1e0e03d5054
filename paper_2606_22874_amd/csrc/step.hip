// Fused decode step: selector scoring, block selection and block-sparse
// attention of every sequence in one launch (paper Section 2: score every KV
// block, pick blocks by the dual top-p / top-K rule with sink and recency
// reserved, attend to the chosen blocks only).
//
// Separate launches pay a kernel boundary (completion, cache maintenance and
// dispatch of the next grid, a few microseconds each) twice per step, and
// the attention grid only starts fetching once its dispatch is done.  Here
// one grid of n_pairs * n_slot workgroups (pair = (sequence b, KV head g),
// slot s) runs
//   1. scoring: the first kMaxScorers workgroups of each row (workgroup i
//      serves row i % batch) score a contiguous run of its blocks; each
//      score also goes out as a self-flagging record word;
//   2. selection: workgroup r (a scorer of row r) polls the row's score
//      records (each thread its own ids, as they land), selects the row (the
//      workgroup core shared with the stand-alone kernel), publishes the
//      selected set as a bitmap (16 block bits and a flag bit per word, one
//      copy per KV head), then writes idx / count / nuc_mass and clears the
//      score records;
//   3. attention: every workgroup polls its pair's bitmap copy, takes its
//      share of the set (entries s, s + n_slot, ... in ascending block id:
//      the stand-alone decode's share of the same list) and runs its part of
//      the split-KV decode (shared core).  The partials go to the workspace;
//      the last workgroup of the pair to finish (device-scope counter)
//      merges them in slot order (deterministic), resets the counter and
//      clears the bitmap, which every workgroup of the pair has read by then.
// A record word is nonzero once written and its reader sets it back to zero,
// so a hand-off needs no flag or fence, only polling readers; the records,
// bitmaps and counters are all zero again when a launch ends.
//
// Residency: a row's selector waits for the row's scorers, and every
// workgroup waits for its row's selector; the merge waits for nothing (the
// last finisher reads partials that are already written).  The launcher
// sizes the grid to the occupancy-derived capacity of the device, so on an
// otherwise idle device all workgroups are resident together; the scorers
// and selectors are the lowest workgroup ids and start first.  A kernel
// holding compute units on another stream can delay some of them; each wait
// is therefore bounded (wait_ticks of the 100 MHz real-time counter).  An
// expired wait computes nothing on unwritten records: that workgroup attends
// to no block (an expired selector publishes an empty set), sets
// count[b] = -1 and a sticky error word in the workspace.  A launch that
// finds the sticky word set does not wait at all (count = -1 for every row,
// outputs zero) until spot_decode_step_status() reports the expiry and
// zero-fills the workspace.
#include <atomic>
#include <mutex>

#include "decode_core.h"
#include "score_core.h"
#include "select_core.h"

// Measurement hook: SPOT_STEP_TS(i) marks phase i of a workgroup (a
// timeline build defines it; empty otherwise).
#ifndef SPOT_STEP_TS
#define SPOT_STEP_TS(i) ((void)0)
#endif

namespace spot {
namespace {

using namespace dec;

constexpr int kScoreRun = 8;              // blocks per scoring call of one wave (the
                                          // stand-alone kernel's run: same code, same bits)
constexpr int kMaxScorers = 64;           // scoring workgroups per row
constexpr int kRecRow = 4096;             // score record words per row (the fused maximum)
constexpr int kMaxSlots = 16;             // attention workgroups per pair (merge_small)
constexpr uint64_t kWaitTicks = 20000000; // 0.2 s of the 100 MHz real-time counter

struct StepArgs {
  const void* q_sel;       // BF16, or codes of the key cache's format (qfmt)
  const uint8_t* q_scale;  // the query codes' scales (qfmt != BF16)
  int qfmt;
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
  int slot_div;        // ceil(2^18 / n_slot): x / n_slot == (x * slot_div) >> 18 below 2^14
  float scale_log2;
  float* scores;
  int32_t* idx;
  int32_t* count;
  float* mass;
  uint16_t* out;
  float* lse;
  float* part_o;       // [batch * h_q, n_slot, 128] partial o
  float* part_ml;      // [batch * h_q, n_slot, 2] partial (m, l)
  unsigned* pair_cnt;  // [batch * h_kv] split completion counters
  uint32_t* sticky;    // expiry word (one per workspace)
  uint32_t* srec;      // [batch, kRecRow] score records
  uint32_t* brec;      // [batch * h_kv, kBitWords] selected-set bitmap copies, one per pair
  uint64_t wait_ticks;
  int force_expire;    // test hook: every score wait gives up at once
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

// Score source of the selection: thread t polls the records of its own ids
// [j0, j0 + EPT) of the row until every valid one is written (two
// words per load; the words past nv stay zero all launch).  Fails when the
// wait expires, or at once when give_up is set.
struct PolledScores {
  const uint32_t* rec;
  uint64_t ticks;
  bool give_up;
  template <int EPT>
  __device__ __forceinline__ bool operator()(float (&sv)[EPT], int j0, int nv) const {
    uint32_t wd[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) wd[e] = 0u;
    bool all = false;
    if (!give_up) {
      const uint64_t deadline = now() + ticks;
      for (;;) {
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
        all = true;
#pragma unroll
        for (int e = 0; e < EPT; ++e) all = all && (j0 + e >= nv || wd[e] != 0u);
        if (all || now() > deadline) break;
      }
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) sv[e] = j0 + e < nv && wd[e] != 0u ? rec_value(wd[e]) : -INFINITY;
    return all;
  }
};

// The selected set of a row travels as a bitmap: record word w holds the
// bits of ids [16w, 16w + 16) in its low half and kBitFlag (so that every
// written word is nonzero).  An attention workgroup's wave 0 polls its pair's
// copy, scans the bit counts over the lanes and takes the entries slot, slot
// + n_slot, ... of the ascending list whose ids lie below nb_valid (the
// stand-alone decode's share of the same list, in the same order).  Returns
// the share's length, or -1 when the wait expired.
constexpr uint32_t kBitFlag = 0x10000u;
constexpr int kBitWords = kRecRow / 16;   // bitmap words per copy

// Position of the r-th (from 0) set bit of x; r < popcount(x).
__device__ __forceinline__ int nth_set_bit(uint64_t x, int r) {
  int base = 0;
  uint32_t w = (uint32_t)x;
  int c = __popc(w);
  if (r >= c) {
    r -= c;
    w = (uint32_t)(x >> 32);
    base = 32;
  }
#pragma unroll
  for (int half = 16; half >= 1; half >>= 1) {
    c = __popc(w & ((1u << half) - 1u));
    if (r >= c) {
      r -= c;
      w >>= half;
      base += half;
    }
  }
  return base;
}

__device__ __forceinline__ int poll_bitmap(int* ids, const uint32_t* rec, int nwords, int k_max,
                                           int slot, int n_slot, int slot_div, int nb_valid,
                                           uint64_t ticks, bool give_up) {
  const int lane = __lane_id();
  // lane l: words [4l, 4l + 4), ids [64l, 64l + 64)
  uint32_t wd[4];
#pragma unroll
  for (int x = 0; x < 4; ++x) wd[x] = 4 * lane + x < nwords ? 0u : kBitFlag;
  bool expired = give_up;
  if (!give_up) {
    const uint64_t deadline = now() + ticks;
    for (;;) {
#pragma unroll
      for (int x = 0; x < 4; x += 2) {
        if (wd[x] == 0u || wd[x + 1] == 0u) {
          const uint64_t v = load_rec(reinterpret_cast<const uint64_t*>(rec + 4 * lane + x));
          if (wd[x] == 0u) wd[x] = (uint32_t)v;
          if (wd[x + 1] == 0u) wd[x + 1] = (uint32_t)(v >> 32);
        }
      }
      const bool mine = wd[0] && wd[1] && wd[2] && wd[3];
      if (__ballot(!mine) == 0ull) break;
      if (now() > deadline) {
        expired = true;
        break;
      }
    }
  }
  if (expired) return -1;
  uint64_t bits = 0;
#pragma unroll
  for (int x = 0; x < 4; ++x) bits |= (uint64_t)(wd[x] & 0xffffu) << (16 * x);
  const int base_id = 64 * lane;
  // entries below k_max and below nb_valid only (the list ascends, so the
  // valid ids are a prefix of it)
  const uint64_t valid = base_id >= nb_valid ? 0ull
                         : nb_valid - base_id >= 64 ? ~0ull
                                                    : (1ull << (nb_valid - base_id)) - 1ull;
  const int cnt = __popcll(bits);
  const int incl = wave_incl_scan_i(cnt);
  const int pos = incl - cnt;             // list position of this lane's first id
  const int total = min(__builtin_amdgcn_readlane(incl, 63), k_max);
  // set bits below nb_valid: the list position of id nb_valid (the lane that
  // holds it adds its own bits below it)
  const int lv = min(nb_valid >> 6, 63);
  const int n_ok = min(__builtin_amdgcn_readlane(incl - cnt + __popcll(bits & valid), lv), total);
  // This lane's entries of the share: positions slot + kk * n_slot in
  // [pos, min(pos + cnt, n_ok)), each the (position - pos)-th set bit.
  // Divisions by n_slot are a multiply and a shift (positions stay below
  // 2^14, where that is exact).
  const int end = min(pos + cnt, n_ok);
  for (int kk = pos > slot ? ((pos - slot + n_slot - 1) * slot_div) >> 18 : 0;; ++kk) {
    const int p = slot + kk * n_slot;
    if (p >= end || kk >= kMaxIds) break;
    ids[kk] = base_id + nth_set_bit(bits, p - pos);
  }
  return n_ok > slot ? min(((n_ok - slot + n_slot - 1) * slot_div) >> 18, kMaxIds) : 0;
}

// Queries in BF16 or, when qfmt is not BF16, in the key cache's own format.
template <int KFMT, int LPH>
__device__ __forceinline__ void score_run(const StepArgs& a, int row, int nv, int j0, int jend,
                                          int lane) {
  uint32_t* rec = a.srec + (size_t)row * kRecRow;
  if (KFMT == SPOT_KFMT_BF16 || a.qfmt == SPOT_KFMT_BF16)
    score_blocks<KFMT, LPH, kScoreRun>(a.q_sel, a.w, a.k_sel, a.k_scale, row, row, a.nblk, nv,
                                       j0, jend, a.scores, rec, lane);
  else
    score_blocks<KFMT, LPH, kScoreRun, KFMT>(a.q_sel, a.w, a.k_sel, a.k_scale, row, row, a.nblk,
                                             nv, j0, jend, a.scores, rec, lane, a.q_scale);
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

template <int EPT, int SPL, int G>
union StepSmem {
  SelWgSmem<EPT, SPL> sel;
  DecodeSmem<G> dec;
};

// G: query heads per KV head (4 or 8), a compile-time constant of the
// attention core; 4 waves (256 threads) either way.
template <int EPT, int SPL, int G>
__global__ __launch_bounds__(64 * kDecWaves, 2) void step_kernel(StepArgs a) {
  __shared__ StepSmem<EPT, SPL, G> sm;
  // The block list and the per-workgroup flags of the decode layout lie past
  // every field of the selection.
  static_assert(offsetof(DecodeSmem<G>, ids) >= sizeof(SelWgSmem<EPT, SPL>),
                "decode list overlaps the selection storage");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wg = blockIdx.x, nwg = gridDim.x;
  const int n_slot = a.n_slot;
  const int pair = wg / n_slot, slot = wg % n_slot;
  const int b = pair / a.h_kv, g = pair % a.h_kv;
  const bool failed_before = load_rec(a.sticky) != 0u;
  const int sl = min(a.seq_len[b], a.l_cap);
  SPOT_STEP_TS(0);

  // ---- 1. scoring: row r = wg % B, by its first n_sc workgroups
  const int B = a.batch;
  {
    const int r = wg % B, c = wg / B;
    const int n_sc = min(kMaxScorers, (nwg - r + B - 1) / B);   // scorers of row r
    if (c < n_sc) {
      int nv = a.n_valid ? a.n_valid[r] : a.nblk;
      nv = nv < 0 ? 0 : (nv > a.nblk ? a.nblk : nv);
      const int per = (a.nblk + n_sc - 1) / n_sc;
      const int jb = c * per, je = min(jb + per, a.nblk);
      for (int j0 = jb + wave * kScoreRun; j0 < je; j0 += kDecWaves * kScoreRun)
        score_run_rt(a, r, nv, j0, je, lane);
    }
  }
  SPOT_STEP_TS(1);

  // ---- 2. selection of row wg by workgroup wg (wg < B is scorer 0 of it)
  if (wg < B) {
    int nv = a.n_valid ? a.n_valid[wg] : a.nblk;
    nv = nv < 0 ? 0 : (nv > a.nblk ? a.nblk : nv);
    uint32_t* srec = a.srec + (size_t)wg * kRecRow;
    const SelRow r = select_row_core<EPT, SPL>(
        sm.sel, PolledScores{srec, a.wait_ticks, failed_before || a.force_expire != 0}, nv,
        a.top_p, a.k_max, a.k_min, a.n_sink, a.n_recent);
    SPOT_STEP_TS(2);
    // Publish the set as a bitmap right away (the lanes of a 16-id word
    // combine their bits with shuffles), then write idx / count / nuc_mass.
    {
      constexpr int K = 16 / EPT;   // threads per bitmap word
      uint32_t wb = r.ok ? r.fin : 0u;
#pragma unroll
      for (int d = 1; d < K; d <<= 1) wb |= (uint32_t)__shfl_down((int)wb, d, 64) << (d * EPT);
      const int nwords = (a.nblk + 15) / 16;
      const int w = tid * EPT / 16;
      if (tid % K == 0 && w < nwords) {
        uint32_t* bm = a.brec + (size_t)wg * a.h_kv * kBitWords + w;
        const uint32_t word = (wb & 0xffffu) | kBitFlag;
        for (int c = 0; c < a.h_kv; ++c) store_rec(bm + (size_t)c * kBitWords, word);
      }
    }
    int total;
    const int pos = sel_positions(sm.sel, r.fin, total);
    if (r.ok) {
      sel_write<EPT>(a.idx + (size_t)wg * a.k_max, a.count + wg, a.mass ? a.mass + wg : nullptr,
                     a.k_max, r.fin, pos, total, r.mass);
    } else if (tid == 0) {
      // The wait expired (or an earlier one did): an empty set was published.
      if (!failed_before) store_rec(a.sticky, 1u);
      store_rec(a.count + wg, -1);
    }
    // The selector is the score records' only reader.
    for (int j = 2 * tid; j < nv; j += 2 * kSelWG)
      store_rec(reinterpret_cast<uint64_t*>(srec + j), (uint64_t)0);
    SPOT_STEP_TS(3);
    __syncthreads();   // the selection's LDS is reused below
  }

  // ---- 3. attention on this workgroup's share of the published set
  uint32_t* bmap = a.brec + (size_t)pair * kBitWords;
  const int nb_valid = (sl + kBlk - 1) / kBlk;
  if (wave == 0) {
    const int n = poll_bitmap(sm.dec.ids, bmap, (a.nblk + 15) / 16, a.k_max, slot, n_slot,
                              a.slot_div, nb_valid, a.wait_ticks, false);
    if (lane == 0) sm.dec.n_local = n;
  }
  __syncthreads();
  int n_local = sm.dec.n_local;
  if (n_local < 0) {
    n_local = 0;
    if (tid == 0) {
      store_rec(a.sticky, 1u);
      store_rec(a.count + b, -1);
    }
  }
  SPOT_STEP_TS(4);

  const QueryFrag qf = load_query_heads<G>(a.q, b, g, a.h_q);
  const size_t head_base = ((size_t)b * a.h_kv + g) * (size_t)a.l_cap * kD;
  auto blk_of = [&](int n) { return sm.dec.ids[n]; };
  const Partials<G> hp = attend_blocks<G>(sm.dec, qf, a.k + head_base, a.v + head_base, sl,
                                           n_local, blk_of, a.scale_log2, NoHook{});
  SPOT_STEP_TS(5);
  // wave w holds heads w, w + 4, ... of the group
#pragma unroll
  for (int jh = 0; jh < Partials<G>::HPW; ++jh) {
    const size_t bh = (size_t)b * a.h_q + g * G + wave + kDecWaves * jh;
    store_coherent(&a.part_o[(bh * n_slot + slot) * kD + 2 * lane],
                   make_float2(hp.h[jh].o0, hp.h[jh].o1));
    if (lane == 0)
      store_coherent(&a.part_ml[(bh * n_slot + slot) * 2], make_float2(hp.h[jh].M, hp.h[jh].L));
  }

  // ---- the last workgroup of the pair to finish merges all slots
  wait_stores();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&a.pair_cnt[pair], 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    sm.dec.last = prev == (unsigned)(n_slot - 1);
  }
  __syncthreads();
  SPOT_STEP_TS(6);
  if (!sm.dec.last) return;
  if (tid == 0) store_rec(&a.pair_cnt[pair], 0u);
  for (int w = 2 * tid; w < (a.nblk + 15) / 16; w += 2 * kSelWG)
    store_rec(reinterpret_cast<uint64_t*>(bmap + w), (uint64_t)0);
#pragma unroll
  for (int jh = 0; jh < Partials<G>::HPW; ++jh)
    merge_head(a.part_o, a.part_ml, n_slot, (size_t)b * a.h_q + g * G + wave + kDecWaves * jh,
               a.out, a.lse, lane);
  SPOT_STEP_TS(7);
}

// ---- Short rows: a step whose rows have at most kSmallBlocks blocks.  The
// two hand-offs of step_kernel (scores to the selector, the set to the
// attention workgroups) cost ~1.5 us each, more than scoring a short row
// takes, so here every workgroup of a sequence scores the whole row itself
// (the row's selector cache is at most 128 KiB and stays in L2), keeps the
// scores in LDS, runs the same selection core on them and takes its share
// of the ascending list directly; only workgroup (KV head 0, slot 0) of the
// sequence writes the scores, idx, count and nucleus mass.  Scores and set
// are those of step_kernel (same scoring code, same selection core) and the
// split is the stand-alone decode's (at most 16 workgroups per pair, with no
// residency cap, since nothing waits), so the results are the same bits as
// step_kernel's wherever its own split is not capped.  No workgroup waits
// for another (the last finisher of a pair merges, as in step_kernel); the
// expiry word keeps its meaning: a launch that finds it set (or the forced
// expiry of the tests) selects nothing and reports count = -1.
constexpr int kSmallBlocks = 128;
constexpr int kSmallRun = 16;   // blocks per scoring call of one wave

// Score source of the short-row kernel: the row's scores in LDS; fails at
// once (no ids) when give_up is set.
struct LdsRowScores {
  const float* s;
  bool give_up;
  template <int EPT>
  __device__ __forceinline__ bool operator()(float (&sv)[EPT], int j0, int nv) const {
#pragma unroll
    for (int e = 0; e < EPT; ++e) sv[e] = !give_up && j0 + e < nv ? s[j0 + e] : -INFINITY;
    return !give_up;
  }
};

template <int KFMT, int LPH>
__device__ __forceinline__ float score_small(const StepArgs& a, int row, int nv, int j0,
                                             float* scores, int lane) {
  if (KFMT == SPOT_KFMT_BF16 || a.qfmt == SPOT_KFMT_BF16)
    return score_blocks<KFMT, LPH, kSmallRun>(a.q_sel, a.w, a.k_sel, a.k_scale, row, row,
                                              a.nblk, nv, j0, a.nblk, scores, nullptr, lane);
  return score_blocks<KFMT, LPH, kSmallRun, KFMT>(a.q_sel, a.w, a.k_sel, a.k_scale, row, row,
                                                  a.nblk, nv, j0, a.nblk, scores, nullptr, lane,
                                                  a.q_scale);
}

__device__ __forceinline__ float score_small_rt(const StepArgs& a, int row, int nv, int j0,
                                                float* scores, int lane) {
  if (a.lph == 8) {
    switch (a.kfmt) {
      case SPOT_KFMT_BF16: return score_small<SPOT_KFMT_BF16, 8>(a, row, nv, j0, scores, lane);
      case SPOT_KFMT_INT4_G32:
        return score_small<SPOT_KFMT_INT4_G32, 8>(a, row, nv, j0, scores, lane);
      case SPOT_KFMT_INT8_G32:
        return score_small<SPOT_KFMT_INT8_G32, 8>(a, row, nv, j0, scores, lane);
      case SPOT_KFMT_MXFP8_G32:
        return score_small<SPOT_KFMT_MXFP8_G32, 8>(a, row, nv, j0, scores, lane);
      default: return score_small<SPOT_KFMT_MXFP4_G32, 8>(a, row, nv, j0, scores, lane);
    }
  }
  switch (a.kfmt) {
    case SPOT_KFMT_BF16: return score_small<SPOT_KFMT_BF16, 16>(a, row, nv, j0, scores, lane);
    case SPOT_KFMT_INT4_G32:
      return score_small<SPOT_KFMT_INT4_G32, 16>(a, row, nv, j0, scores, lane);
    case SPOT_KFMT_INT8_G32:
      return score_small<SPOT_KFMT_INT8_G32, 16>(a, row, nv, j0, scores, lane);
    case SPOT_KFMT_MXFP8_G32:
      return score_small<SPOT_KFMT_MXFP8_G32, 16>(a, row, nv, j0, scores, lane);
    default: return score_small<SPOT_KFMT_MXFP4_G32, 16>(a, row, nv, j0, scores, lane);
  }
}

// One id per thread (EPT = 1: nblk <= kSmallBlocks < 256).
template <int SPL, int G>
__global__ __launch_bounds__(64 * kDecWaves, 2) void step_small_kernel(StepArgs a) {
  constexpr int EPT = 1;
  __shared__ StepSmem<EPT, SPL, G> sm;
  __shared__ float sc[kSmallBlocks];
  static_assert(offsetof(DecodeSmem<G>, ids) >= sizeof(SelWgSmem<EPT, SPL>),
                "decode list overlaps the selection storage");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_slot = a.n_slot;
  const int pair = blockIdx.x / n_slot, slot = blockIdx.x % n_slot;
  const int b = pair / a.h_kv, g = pair % a.h_kv;
  const bool failed_before = load_rec(a.sticky) != 0u;
  const int sl = min(a.seq_len[b], a.l_cap);
  const bool writer = g == 0 && slot == 0;
  int nv = a.n_valid ? a.n_valid[b] : a.nblk;
  nv = nv < 0 ? 0 : (nv > a.nblk ? a.nblk : nv);
  SPOT_STEP_TS(0);

  // The attention's query fragment goes out first; it waits in registers.
  const QueryFrag qf = load_query_heads<G>(a.q, b, g, a.h_q);

  // ---- 1. scoring: the whole row, runs of kSmallRun blocks per wave.  The
  // key loads do not wait for n_valid (every block of the row is in the
  // cache); scores past it become -inf here, as score_blocks makes them.
  for (int j0 = wave * kSmallRun; j0 < a.nblk; j0 += kDecWaves * kSmallRun) {
    const float v = score_small_rt(a, b, a.nblk, j0, nullptr, lane);
    const int j = j0 + lane;
    if (lane < kSmallRun && j < a.nblk) sc[j] = j < nv ? v : -INFINITY;
  }
  __syncthreads();
  if (writer)
    for (int j = tid; j < a.nblk; j += kSelWG) a.scores[(size_t)b * a.nblk + j] = sc[j];
  SPOT_STEP_TS(1);

  // ---- 2. selection, then this workgroup's share of the list
  const SelRow r = select_row_core<EPT, SPL>(
      sm.sel, LdsRowScores{sc, failed_before || a.force_expire != 0}, nv, a.top_p, a.k_max,
      a.k_min, a.n_sink, a.n_recent);
  SPOT_STEP_TS(2);
  int total;
  const int pos = sel_positions(sm.sel, r.fin, total);
  if (writer) {
    if (r.ok) {
      sel_write<EPT>(a.idx + (size_t)b * a.k_max, a.count + b, a.mass ? a.mass + b : nullptr,
                     a.k_max, r.fin, pos, total, r.mass);
    } else if (tid == 0) {
      if (!failed_before) store_rec(a.sticky, 1u);
      store_rec(a.count + b, -1);
    }
  }
  // The list is S in ascending id, cut at k_max entries; the ids below
  // nb_valid are a prefix of it, [0, n_ok), n_ok read off thread nb_valid's
  // position (nb_valid <= nblk < 256).  Entries slot, slot + n_slot, ...
  // of that prefix are the share (as the stand-alone decode takes them).
  const int nb_valid = (sl + kBlk - 1) / kBlk;
  const int n_entries = min(total, a.k_max);
  if (tid == nb_valid) {
    const int n_ok = min(pos, n_entries);
    sm.dec.n_local = n_ok > slot ? min((n_ok - slot + n_slot - 1) / n_slot, kMaxIds) : 0;
  }
  if ((r.fin & 1u) && tid < nb_valid && pos < n_entries && pos >= slot &&
      (pos - slot) % n_slot == 0 && (pos - slot) / n_slot < kMaxIds)
    sm.dec.ids[(pos - slot) / n_slot] = tid;
  __syncthreads();
  const int n_local = sm.dec.n_local;
  SPOT_STEP_TS(3);
  SPOT_STEP_TS(4);

  // ---- 3. attention on the share, partials, the last finisher merges
  const size_t head_base = ((size_t)b * a.h_kv + g) * (size_t)a.l_cap * kD;
  auto blk_of = [&](int n) { return sm.dec.ids[n]; };
  const Partials<G> hp = attend_blocks<G>(sm.dec, qf, a.k + head_base, a.v + head_base, sl,
                                           n_local, blk_of, a.scale_log2, NoHook{});
  SPOT_STEP_TS(5);
#pragma unroll
  for (int jh = 0; jh < Partials<G>::HPW; ++jh) {
    const size_t bh = (size_t)b * a.h_q + g * G + wave + kDecWaves * jh;
    store_coherent(&a.part_o[(bh * n_slot + slot) * kD + 2 * lane],
                   make_float2(hp.h[jh].o0, hp.h[jh].o1));
    if (lane == 0)
      store_coherent(&a.part_ml[(bh * n_slot + slot) * 2], make_float2(hp.h[jh].M, hp.h[jh].L));
  }
  wait_stores();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&a.pair_cnt[pair], 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    sm.dec.last = prev == (unsigned)(n_slot - 1);
  }
  __syncthreads();
  SPOT_STEP_TS(6);
  if (!sm.dec.last) return;
  if (tid == 0) store_rec(&a.pair_cnt[pair], 0u);
#pragma unroll
  for (int jh = 0; jh < Partials<G>::HPW; ++jh)
    merge_head(a.part_o, a.part_ml, n_slot, (size_t)b * a.h_q + g * G + wave + kDecWaves * jh,
               a.out, a.lse, lane);
  SPOT_STEP_TS(7);
}

template <int SPL, int G>
hipError_t launch_small_t(StepArgs& a, int n_pairs, int n_slot_max, hipStream_t s) {
  a.n_slot = n_slot_max;
  a.slot_div = ((1 << 18) + a.n_slot - 1) / a.n_slot;
  hipLaunchKernelGGL((step_small_kernel<SPL, G>), dim3(n_pairs * a.n_slot), dim3(64 * kDecWaves),
                     0, s, a);
  return hipGetLastError();
}

// Workgroups of one step kernel that can be resident at once (per CU times
// the CU count), queried once per device and instantiation.  The value only
// depends on the device, so concurrent first calls store the same number.
template <int EPT, int SPL, int G>
int step_capacity() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  const int c = cached[dev].load(std::memory_order_relaxed);
  if (c > 0) return c;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(&step_kernel<EPT, SPL, G>), 64 * kDecWaves, 0) !=
      hipSuccess)
    return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  cached[dev].store(per_cu * cus, std::memory_order_relaxed);
  return per_cu * cus;
}

template <int EPT, int SPL, int G>
hipError_t launch_step_t(StepArgs& a, int n_pairs, int n_slot_max, hipStream_t s) {
  const int cap = step_capacity<EPT, SPL, G>();
  if (cap < n_pairs) return hipErrorCooperativeLaunchTooLarge;
  a.n_slot = n_slot_max < cap / n_pairs ? n_slot_max : cap / n_pairs;
  a.slot_div = ((1 << 18) + a.n_slot - 1) / a.n_slot;
  hipLaunchKernelGGL((step_kernel<EPT, SPL, G>), dim3(n_pairs * a.n_slot), dim3(64 * kDecWaves), 0, s,
                     a);
  return hipGetLastError();
}

std::atomic<int> g_force_expire{0};

__global__ __launch_bounds__(256) void zero_fill_kernel(uint4* __restrict__ p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

}  // namespace

// Workspace of spot_decode_step_static: one array per device, kept until the
// process ends.  Host code never passes `scratch` itself to a kernel (in host
// code the name is only a stand-in); it uses the device address that
// hipGetSymbolAddress returns for the current device.
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;
constexpr size_t kStaticCtrlBytes = (size_t)1 << 20;   // control region of every shape
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
std::atomic<void*> g_scratch_ptr[64];
}  // namespace

// Workspace of a decode step (both paths).  The control region comes first:
// the split completion counters (one per pair, used by the fused launch and
// by the separate decode alike), the expiry word (16 bytes), the score
// records [batch, kRecRow] and the bitmap copies [batch * h_kv, kBitWords];
// every call leaves it all zero.  The partials follow at `part`: o
// [batch * h_q, ns, 128] then (m, l) [batch * h_q, ns, 2], ns being the
// separate decode's split count (the fused launch indexes them with its own
// n_slot <= ns); they hold data between calls.  ctrl_cap > 0 fixes where the
// partials start, so that calls of any shape find zeros in their control
// words; 0 puts them right after the control words.
StepWs step_layout(int batch, int h_q, int h_kv, int k_max, size_t ctrl_cap) {
  StepWs L;
  L.cnt = 0;
  L.sticky = ((size_t)batch * h_kv * 4 + 15) & ~(size_t)15;
  L.srec = L.sticky + 16;
  L.brec = L.srec + (size_t)batch * kRecRow * 4;
  L.ctrl = (L.brec + (size_t)batch * h_kv * kBitWords * 4 + 255) & ~(size_t)255;
  L.part = ctrl_cap > 0 ? ctrl_cap : L.ctrl;
  const size_t ns = (size_t)decode_num_splits(batch, h_kv, k_max, h_q / h_kv);
  L.total = L.part + (size_t)batch * h_q * ns * (kD + 2) * 4;
  return L;
}

size_t static_scratch_bytes() { return kStaticScratchBytes; }

hipError_t static_scratch(void** out, bool setup, hipStream_t s) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p || !setup) {
    *out = p;
    return hipSuccess;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    // Zero-filled once (a fill kernel, also safe inside a captured graph);
    // every call leaves the array zeroed again.
    hipLaunchKernelGGL(zero_fill_kernel, dim3(1024), dim3(256), 0, s, static_cast<uint4*>(p),
                       kStaticScratchBytes / 16);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return hipSuccess;
}

size_t step_workspace_bytes(int batch, int h_q, int h_kv, int d, int k_max) {
  (void)d;
  return step_layout(batch, h_q, h_kv, k_max, 0).total;
}

StepWs step_static_layout(int batch, int h_q, int h_kv, int k_max) {
  return step_layout(batch, h_q, h_kv, k_max, kStaticCtrlBytes);
}

bool step_static_fits(int batch, int h_q, int h_kv, int k_max) {
  const StepWs L = step_static_layout(batch, h_q, h_kv, k_max);
  return L.ctrl <= kStaticCtrlBytes && L.total <= kStaticScratchBytes;
}

void step_force_expiry(int on) { g_force_expire.store(on ? 1 : 0, std::memory_order_relaxed); }

// Groups the fused kernel is compiled for: 4 and 8 query heads per KV head
// (a build that defines SPOT_STEP_GROUP4_ONLY, the phase-stamping timeline
// build, only 4); other groups run the three stages as separate launches.
#ifdef SPOT_STEP_GROUP4_ONLY
constexpr bool kStepGroup8 = false;
#else
constexpr bool kStepGroup8 = true;
#endif

bool step_fusable(int h_q, int h_kv, int nblk, int k_max) {
  if (h_kv < 1 || (h_q != 4 * h_kv && !(kStepGroup8 && h_q == 8 * h_kv)) || nblk < 1 ||
      nblk > kRecRow)
    return false;
  int P = 1;
  const int cap = k_max < nblk ? k_max : nblk;
  while (P < cap) P <<= 1;
  return P <= 512;
}

hipError_t launch_decode_step(const void* q_sel, const void* q_scale, int qfmt, const float* w,
                              const void* k_sel, const void* k_scale, int kfmt, int d_s,
                              const int32_t* n_valid,
                              float top_p, int k_max, int k_min, int n_sink, int n_recent,
                              const void* q, const void* k, const void* v,
                              const int32_t* seq_len, int batch, int h_q, int h_kv, int l_cap,
                              float sm_scale, float* scores, int32_t* idx, int32_t* count,
                              float* nuc_mass, void* out, float* lse, void* ws, bool static_ws,
                              hipStream_t s) {
  StepArgs a;
  a.q_sel = q_sel;
  a.q_scale = static_cast<const uint8_t*>(q_scale);
  a.qfmt = qfmt;
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
  const StepWs L = static_ws ? step_static_layout(batch, h_q, h_kv, k_max)
                            : step_layout(batch, h_q, h_kv, k_max, 0);
  const int ns = decode_num_splits(batch, h_kv, k_max, h_q / h_kv);
  const int n_slot_max = ns < kMaxSlots ? ns : kMaxSlots;
  char* base = static_cast<char*>(ws);
  a.part_o = reinterpret_cast<float*>(base + L.part);
  a.part_ml = a.part_o + (size_t)batch * h_q * ns * kD;
  a.pair_cnt = reinterpret_cast<unsigned*>(base + L.cnt);
  a.sticky = reinterpret_cast<uint32_t*>(base + L.sticky);
  a.srec = reinterpret_cast<uint32_t*>(base + L.srec);
  a.brec = reinterpret_cast<uint32_t*>(base + L.brec);
  a.wait_ticks = kWaitTicks;
  a.force_expire = g_force_expire.load(std::memory_order_relaxed);
  const int n_pairs = batch * h_kv;
  // The partials are laid out for ns splits; the launch's n_slot (at most
  // n_slot_max, fewer when fewer workgroups fit) uses a prefix of each
  // head's run, indexed with the actual n_slot -- [B, h_q, n_slot] either way.
  int P = 1;
  const int cap = k_max < a.nblk ? k_max : a.nblk;
  while (P < cap) P <<= 1;
  const int spl = P <= 64 ? 1 : P / 64;
  if (a.nblk <= kSmallBlocks) {   // P <= 128
#ifdef SPOT_STEP_GROUP4_ONLY
    return spl == 1 ? launch_small_t<1, 4>(a, n_pairs, n_slot_max, s)
                    : launch_small_t<2, 4>(a, n_pairs, n_slot_max, s);
#else
    if (h_q == 8 * h_kv)
      return spl == 1 ? launch_small_t<1, 8>(a, n_pairs, n_slot_max, s)
                      : launch_small_t<2, 8>(a, n_pairs, n_slot_max, s);
    return spl == 1 ? launch_small_t<1, 4>(a, n_pairs, n_slot_max, s)
                    : launch_small_t<2, 4>(a, n_pairs, n_slot_max, s);
#endif
  }
  const int ept = a.nblk <= 256 ? 1 : a.nblk <= 512 ? 2 : a.nblk <= 1024 ? 4
                : a.nblk <= 2048 ? 8 : 16;
#ifdef SPOT_STEP_GROUP4_ONLY
#define SPOT_STEP_CASE(E, S) \
  if (ept == E && spl == S) return launch_step_t<E, S, 4>(a, n_pairs, n_slot_max, s);
#else
#define SPOT_STEP_CASE(E, S)                                                         \
  if (ept == E && spl == S)                                                          \
    return h_q == 8 * h_kv ? launch_step_t<E, S, 8>(a, n_pairs, n_slot_max, s)       \
                           : launch_step_t<E, S, 4>(a, n_pairs, n_slot_max, s);
#endif
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
