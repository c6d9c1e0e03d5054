// C ABI of libspot: argument validation, then kernel launches.  Nothing is
// enqueued unless every argument check passes.
#include "spot_internal.h"

#define SPOT_VERSION_STR "spot-mi355x 0.1 (gfx950)"

using namespace spot;

namespace {

spot_status from_hip(hipError_t e) { return e == hipSuccess ? SPOT_OK : SPOT_ERR_HIP; }

// Decode: any group up to 16 query heads per KV head (the group is the
// columns of a 16-wide matrix tile).
bool supported_group(int h_q, int h_kv) {
  if (h_kv < 1 || h_q < h_kv || h_q % h_kv) return false;
  return h_q / h_kv <= kMaxGroupSize;
}

// Prefill: a workgroup takes up to four heads of a group, so groups of
// 1, 2, 4 or 8.
bool supported_prefill_group(int h_q, int h_kv) {
  if (h_kv < 1 || h_q < h_kv || h_q % h_kv) return false;
  const int g = h_q / h_kv;
  return g == 1 || g == 2 || g == 4 || g == 8;
}

}  // namespace

extern "C" {

const char* spot_status_str(spot_status s) {
  switch (s) {
    case SPOT_OK: return "ok";
    case SPOT_ERR_NULL: return "null pointer";
    case SPOT_ERR_SHAPE: return "invalid shape";
    case SPOT_ERR_UNSUPPORTED: return "unsupported size or format";
    case SPOT_ERR_RULE: return "invalid selection rule";
    case SPOT_ERR_WORKSPACE: return "workspace missing or too small";
    case SPOT_ERR_HIP: return "HIP launch error";
    case SPOT_ERR_EXPIRED: return "a bounded wait of the fused decode step expired";
    default: return "unknown status";
  }
}

const char* spot_version(void) { return SPOT_VERSION_STR; }

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

static bool valid_kfmt(int kfmt) {
  return kfmt == SPOT_KFMT_BF16 || kfmt == SPOT_KFMT_INT4_G32 || kfmt == SPOT_KFMT_MXFP4_G32 ||
         kfmt == SPOT_KFMT_INT8_G32 || kfmt == SPOT_KFMT_MXFP8_G32;
}

spot_status spot_selector_project(const void* h, const void* w_q, const void* w_k,
                                  const void* w_w, const int32_t* pos, int rows, int d_model,
                                  int h_s, int d_s, int rope_dim, float rope_base, void* q_out,
                                  float* w_out, void* k_cache, int rows_per_seq, int l_cap,
                                  void* stream) {
  if (!h || !w_q || !w_k || !w_w || !pos || !q_out || !w_out || !k_cache) return SPOT_ERR_NULL;
  if (rows < 0 || d_model < 8 || d_model % 8 || h_s < 1 || d_s < 1 || rows_per_seq < 1 ||
      rows % rows_per_seq || l_cap < 0)
    return SPOT_ERR_SHAPE;
  if (!aligned16(h) || !aligned16(w_q) || !aligned16(w_k) || !aligned16(w_w))
    return SPOT_ERR_SHAPE;
  if (h_s * d_s != 512 || (d_s != 64 && d_s != 128)) return SPOT_ERR_UNSUPPORTED;
  if (rope_dim < 0 || rope_dim > d_s || rope_dim % 2 || !(rope_base > 0.f) ||
      rope_base > 3.0e38f)
    return SPOT_ERR_UNSUPPORTED;
  if (rows == 0) return SPOT_OK;
  return from_hip(launch_selector_project(h, w_q, w_k, w_w, pos, rows, d_model, h_s, d_s,
                                          rope_dim, rope_base, q_out, w_out, k_cache,
                                          rows_per_seq, l_cap, nullptr, nullptr,
                                          static_cast<hipStream_t>(stream)));
}

spot_status spot_selector_project_pooled(const void* h, const void* w_q, const void* w_k,
                                         const void* w_w, const int32_t* pos,
                                         const int32_t* seq_len, int n_seq, int d_model,
                                         int h_s, int d_s, int rope_dim, float rope_base,
                                         void* q_out, float* w_out, void* k_cache, void* k_pool,
                                         int l_cap, void* stream) {
  if (!k_pool) return SPOT_ERR_NULL;
  if (l_cap % kBlk) return SPOT_ERR_SHAPE;
  if (!aligned16(k_pool)) return SPOT_ERR_SHAPE;
  const spot_status st = spot_selector_project(h, w_q, w_k, w_w, pos, 0, d_model, h_s, d_s,
                                               rope_dim, rope_base, q_out, w_out, k_cache, 1,
                                               l_cap, stream);   // validation only
  if (st != SPOT_OK || n_seq == 0) return st;
  if (n_seq < 0) return SPOT_ERR_SHAPE;
  return from_hip(launch_selector_project(h, w_q, w_k, w_w, pos, n_seq, d_model, h_s, d_s,
                                          rope_dim, rope_base, q_out, w_out, k_cache, 1, l_cap,
                                          k_pool, seq_len, static_cast<hipStream_t>(stream)));
}

spot_status spot_selector_pool(const void* k_tok, void* k_pool, int n_seq, int l_cap, int h_s,
                               int d_s, const int32_t* seq_len, const int32_t* first_block,
                               int max_blocks, void* stream) {
  if (!k_tok || !k_pool) return SPOT_ERR_NULL;
  if (n_seq < 0 || l_cap < 0 || l_cap % kBlk || max_blocks < 0 || h_s < 1 || d_s < 1)
    return SPOT_ERR_SHAPE;
  if (!aligned16(k_tok) || !aligned16(k_pool)) return SPOT_ERR_SHAPE;
  if (h_s * d_s != 512) return SPOT_ERR_UNSUPPORTED;
  if (max_blocks > 65535) return SPOT_ERR_UNSUPPORTED;
  if (n_seq == 0 || l_cap == 0 || max_blocks == 0) return SPOT_OK;
  return from_hip(launch_selector_pool(k_tok, k_pool, n_seq, l_cap, seq_len, first_block,
                                       max_blocks, static_cast<hipStream_t>(stream)));
}

spot_status spot_selector_score(const void* q_sel, const float* w, const void* k_sel,
                                const void* k_scale, int kfmt, int n_seq, int rows_per_seq,
                                int nblk, int h_s, int d_s, const int32_t* n_valid,
                                float* scores, void* stream) {
  if (!q_sel || !w || !k_sel || !scores) return SPOT_ERR_NULL;
  if (n_seq < 0 || rows_per_seq < 1 || nblk < 0 || h_s < 1 || d_s < 1) return SPOT_ERR_SHAPE;
  if (!valid_kfmt(kfmt)) return SPOT_ERR_UNSUPPORTED;
  if (kfmt != SPOT_KFMT_BF16 && !k_scale) return SPOT_ERR_NULL;
  if (h_s * d_s != 512 || (d_s != 64 && d_s != 128)) return SPOT_ERR_UNSUPPORTED;
  if ((long long)n_seq * rows_per_seq > 0x7fffffffLL) return SPOT_ERR_SHAPE;
  if (n_seq == 0 || nblk == 0) return SPOT_OK;
  return from_hip(launch_selector_score(q_sel, w, k_sel, k_scale, kfmt, n_seq, rows_per_seq,
                                        nblk, h_s, d_s, n_valid, scores,
                                        static_cast<hipStream_t>(stream)));
}

spot_status spot_selector_score_q(const void* q_sel, const void* q_scale, int qfmt,
                                  const float* w, const void* k_sel, const void* k_scale,
                                  int kfmt, int n_seq, int rows_per_seq, int nblk, int h_s,
                                  int d_s, const int32_t* n_valid, float* scores, void* stream) {
  if (qfmt == SPOT_KFMT_BF16)
    return spot_selector_score(q_sel, w, k_sel, k_scale, kfmt, n_seq, rows_per_seq, nblk, h_s,
                               d_s, n_valid, scores, stream);
  if (!q_sel || !w || !k_sel || !scores) return SPOT_ERR_NULL;
  if (n_seq < 0 || rows_per_seq < 1 || nblk < 0 || h_s < 1 || d_s < 1) return SPOT_ERR_SHAPE;
  if (!valid_kfmt(qfmt) || !valid_kfmt(kfmt)) return SPOT_ERR_UNSUPPORTED;
  if (!q_scale || (kfmt != SPOT_KFMT_BF16 && !k_scale)) return SPOT_ERR_NULL;
  if (h_s * d_s != 512 || (d_s != 64 && d_s != 128)) return SPOT_ERR_UNSUPPORTED;
  if ((long long)n_seq * rows_per_seq > 0x7fffffffLL) return SPOT_ERR_SHAPE;
  if (n_seq == 0 || nblk == 0) return SPOT_OK;
  return from_hip(launch_selector_score_q(q_sel, q_scale, qfmt, w, k_sel, k_scale, kfmt, n_seq,
                                          rows_per_seq, nblk, d_s, n_valid, scores,
                                          static_cast<hipStream_t>(stream)));
}

spot_status spot_selector_score_tokens_blk(const void* q_sel, const float* w, const void* k_tok,
                                           const void* k_scale, int kfmt, int n_seq,
                                           int rows_per_seq, int l_cap, int blk, int h_s, int d_s,
                                           const int32_t* seq_len, float* scores, void* stream) {
  if (!q_sel || !w || !k_tok || !scores) return SPOT_ERR_NULL;
  if (n_seq < 0 || rows_per_seq < 1 || l_cap < 0 || l_cap % kBlk || h_s < 1 || d_s < 1)
    return SPOT_ERR_SHAPE;
  if (!valid_kfmt(kfmt) || (blk != 16 && blk != kBlk)) return SPOT_ERR_UNSUPPORTED;
  if (kfmt != SPOT_KFMT_BF16 && !k_scale) return SPOT_ERR_NULL;
  if (h_s * d_s != 512 || (d_s != 64 && d_s != 128)) return SPOT_ERR_UNSUPPORTED;
  // Launch size: at most one workgroup per (row, block), padded to 8 blocks.
  if (((long long)n_seq * (l_cap / kBlk) + 7) / 8 * 8 * rows_per_seq > 0x7fffffffLL)
    return SPOT_ERR_SHAPE;
  if (n_seq == 0 || l_cap == 0) return SPOT_OK;
  return from_hip(launch_selector_score_tokens(q_sel, w, k_tok, k_scale, kfmt, n_seq,
                                               rows_per_seq, l_cap, blk, d_s, seq_len, scores,
                                               static_cast<hipStream_t>(stream)));
}

spot_status spot_selector_score_tokens(const void* q_sel, const float* w, const void* k_tok,
                                       const void* k_scale, int kfmt, int n_seq,
                                       int rows_per_seq, int l_cap, int h_s, int d_s,
                                       const int32_t* seq_len, float* scores, void* stream) {
  return spot_selector_score_tokens_blk(q_sel, w, k_tok, k_scale, kfmt, n_seq, rows_per_seq,
                                        l_cap, kBlk, h_s, d_s, seq_len, scores, stream);
}

spot_status spot_select_blocks(const float* scores, int rows, int nblk, const int32_t* n_valid,
                               float top_p, int k_max, int k_min, int n_sink, int n_recent,
                               int32_t* idx, int32_t* count, float* nuc_mass, void* stream) {
  if (!scores || !idx || !count) return SPOT_ERR_NULL;
  if (rows < 0 || nblk < 0) return SPOT_ERR_SHAPE;
  if (top_p != top_p || k_max < 1 || k_min > k_max || n_sink < 0 || n_recent < 0 ||
      k_max < n_sink + n_recent)
    return SPOT_ERR_RULE;
  if (nblk > 16384 || k_max > 4096) return SPOT_ERR_UNSUPPORTED;
  if (rows == 0) return SPOT_OK;
  return from_hip(launch_select_blocks(scores, rows, nblk, n_valid, top_p, k_max, k_min, n_sink,
                                       n_recent, idx, count, nuc_mass,
                                       static_cast<hipStream_t>(stream)));
}

size_t spot_decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks) {
  if (batch < 1 || h_q < 1 || h_kv < 1 || d < 1 || max_blocks < 1) return 0;
  return decode_workspace_bytes(batch, h_q, h_kv, d, max_blocks);
}

// Workspaces hold 8-byte device-scope words; 16-byte alignment is required
// (every hipMalloc allocation has it).
static bool misaligned(const void* ws) { return (reinterpret_cast<uintptr_t>(ws) & 15u) != 0; }

static spot_status check_decode(const void* q, const void* k, const void* v,
                                const int32_t* seq_len, const void* out, int batch, int h_q,
                                int h_kv, int d, int l_cap) {
  if (!q || !k || !v || !seq_len || !out) return SPOT_ERR_NULL;
  if (batch < 0 || h_q < 1 || h_kv < 1 || l_cap < 0 || l_cap % kBlk) return SPOT_ERR_SHAPE;
  if (d != 128 || !supported_group(h_q, h_kv)) return SPOT_ERR_UNSUPPORTED;
  return SPOT_OK;
}

spot_status spot_sparse_decode_blk(const void* q, const void* k, const void* v,
                                   const int32_t* seq_len, const int32_t* idx,
                                   const int32_t* count, int k_max, int blk, int batch, int h_q,
                                   int h_kv, int d, int l_cap, float sm_scale, void* out,
                                   float* lse, void* ws, size_t ws_bytes, void* stream) {
  spot_status st = check_decode(q, k, v, seq_len, out, batch, h_q, h_kv, d, l_cap);
  if (st != SPOT_OK) return st;
  if (!idx || !count) return SPOT_ERR_NULL;
  if (k_max < 1) return SPOT_ERR_SHAPE;
  if (blk != 16 && blk != kBlk) return SPOT_ERR_UNSUPPORTED;
  if (batch == 0) return SPOT_OK;
  if (!ws || ws_bytes < decode_workspace_bytes(batch, h_q, h_kv, d, k_max) || misaligned(ws))
    return SPOT_ERR_WORKSPACE;
  return from_hip(launch_decode(false, q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv,
                                l_cap, blk, sm_scale, out, lse, ws, nullptr,
                                static_cast<hipStream_t>(stream)));
}

spot_status spot_sparse_decode(const void* q, const void* k, const void* v,
                               const int32_t* seq_len, const int32_t* idx, const int32_t* count,
                               int k_max, int batch, int h_q, int h_kv, int d, int l_cap,
                               float sm_scale, void* out, float* lse, void* ws, size_t ws_bytes,
                               void* stream) {
  return spot_sparse_decode_blk(q, k, v, seq_len, idx, count, k_max, kBlk, batch, h_q, h_kv, d,
                                l_cap, sm_scale, out, lse, ws, ws_bytes, stream);
}

spot_status spot_dense_decode(const void* q, const void* k, const void* v,
                              const int32_t* seq_len, int batch, int h_q, int h_kv, int d,
                              int l_cap, float sm_scale, void* out, float* lse, void* ws,
                              size_t ws_bytes, void* stream) {
  spot_status st = check_decode(q, k, v, seq_len, out, batch, h_q, h_kv, d, l_cap);
  if (st != SPOT_OK) return st;
  if (l_cap == 0) return SPOT_ERR_SHAPE;
  if (batch == 0) return SPOT_OK;
  if (!ws || ws_bytes < decode_workspace_bytes(batch, h_q, h_kv, d, l_cap / kBlk) ||
      misaligned(ws))
    return SPOT_ERR_WORKSPACE;
  return from_hip(launch_decode(true, q, k, v, seq_len, nullptr, nullptr, 0, batch, h_q, h_kv,
                                l_cap, kBlk, sm_scale, out, lse, ws, nullptr,
                                static_cast<hipStream_t>(stream)));
}

size_t spot_decode_step_workspace_bytes(int batch, int h_q, int h_kv, int d, int k_max) {
  if (batch < 1 || h_q < 1 || h_kv < 1 || d < 1 || k_max < 1) return 0;
  return step_workspace_bytes(batch, h_q, h_kv, d, k_max);
}

}  // extern "C"

static spot_status decode_step_impl(const void* q_sel, const void* q_scale, int qfmt,
                             const float* w, const void* k_sel,
                             const void* k_scale, int kfmt, int h_s, int d_s,
                             const int32_t* n_valid, float top_p, int k_max, int k_min,
                             int n_sink, int n_recent, const void* q, const void* k,
                             const void* v, const int32_t* seq_len, int batch, int h_q,
                             int h_kv, int d, int l_cap, float sm_scale, float* scores,
                             int32_t* idx, int32_t* count, float* nuc_mass, void* out,
                             float* lse, void* ws, size_t ws_bytes, bool static_ws,
                             void* stream) {
  spot_status st = check_decode(q, k, v, seq_len, out, batch, h_q, h_kv, d, l_cap);
  if (st != SPOT_OK) return st;
  if (!q_sel || !w || !k_sel || !scores || !idx || !count) return SPOT_ERR_NULL;
  if (!valid_kfmt(kfmt)) return SPOT_ERR_UNSUPPORTED;
  if (qfmt != SPOT_KFMT_BF16 && qfmt != kfmt) return SPOT_ERR_UNSUPPORTED;
  if (kfmt != SPOT_KFMT_BF16 && !k_scale) return SPOT_ERR_NULL;
  if (qfmt != SPOT_KFMT_BF16 && !q_scale) return SPOT_ERR_NULL;
  if (h_s < 1 || d_s < 1) return SPOT_ERR_SHAPE;
  if (h_s * d_s != 512 || (d_s != 64 && d_s != 128)) return SPOT_ERR_UNSUPPORTED;
  if (l_cap == 0) return SPOT_ERR_SHAPE;
  if (top_p != top_p || k_max < 1 || k_min > k_max || n_sink < 0 || n_recent < 0 ||
      k_max < n_sink + n_recent)
    return SPOT_ERR_RULE;
  const int nblk = l_cap / kBlk;
  if (nblk > 16384 || k_max > 4096) return SPOT_ERR_UNSUPPORTED;
  if (batch == 0) return SPOT_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (static_ws) {
    // the device's static scratch: no allocation, a size limit instead
    if (!step_static_fits(batch, h_q, h_kv, k_max)) return SPOT_ERR_WORKSPACE;
    if (static_scratch(&ws, true, s) != hipSuccess) return SPOT_ERR_HIP;
  } else if (!ws || ws_bytes < step_workspace_bytes(batch, h_q, h_kv, d, k_max) ||
             misaligned(ws)) {
    return SPOT_ERR_WORKSPACE;
  }
  if (step_fusable(h_q, h_kv, nblk, k_max)) {
    const hipError_t e = launch_decode_step(q_sel, q_scale, qfmt, w, k_sel, k_scale, kfmt, d_s,
                                            n_valid, top_p,
                                            k_max, k_min, n_sink, n_recent, q, k, v, seq_len,
                                            batch, h_q, h_kv, l_cap, sm_scale, scores, idx,
                                            count, nuc_mass, out, lse, ws, static_ws, s);
    if (e == hipSuccess) return SPOT_OK;
    if (e != hipErrorCooperativeLaunchTooLarge) return SPOT_ERR_HIP;
    (void)hipGetLastError();  // clear the refused launch; run the stages separately
  }
  hipError_t e = qfmt == SPOT_KFMT_BF16
                     ? launch_selector_score(q_sel, w, k_sel, k_scale, kfmt, batch, 1, nblk, h_s,
                                             d_s, n_valid, scores, s)
                     : launch_selector_score_q(q_sel, q_scale, qfmt, w, k_sel, k_scale, kfmt,
                                               batch, 1, nblk, d_s, n_valid, scores, s);
  if (e == hipSuccess)
    e = launch_select_blocks(scores, batch, nblk, n_valid, top_p, k_max, k_min, n_sink,
                             n_recent, idx, count, nuc_mass, s);
  if (e == hipSuccess) {
    // the partials after the control region, the counters inside it
    const StepWs L = static_ws ? step_static_layout(batch, h_q, h_kv, k_max)
                               : step_layout(batch, h_q, h_kv, k_max, 0);
    char* base = static_cast<char*>(ws);
    e = launch_decode(false, q, k, v, seq_len, idx, count, k_max, batch, h_q, h_kv, l_cap, kBlk,
                      sm_scale, out, lse, base + L.part, reinterpret_cast<unsigned*>(base + L.cnt),
                      s);
  }
  return from_hip(e);
}

extern "C" {

spot_status spot_decode_step(const void* q_sel, const float* w, const void* k_sel,
                             const void* k_scale, int kfmt, int h_s, int d_s,
                             const int32_t* n_valid, float top_p, int k_max, int k_min,
                             int n_sink, int n_recent, const void* q, const void* k,
                             const void* v, const int32_t* seq_len, int batch, int h_q,
                             int h_kv, int d, int l_cap, float sm_scale, float* scores,
                             int32_t* idx, int32_t* count, float* nuc_mass, void* out,
                             float* lse, void* ws, size_t ws_bytes, void* stream) {
  return decode_step_impl(q_sel, nullptr, SPOT_KFMT_BF16, w, k_sel, k_scale, kfmt, h_s, d_s,
                          n_valid, top_p, k_max, k_min, n_sink, n_recent, q, k, v, seq_len, batch,
                          h_q, h_kv, d, l_cap, sm_scale, scores, idx, count, nuc_mass, out, lse,
                          ws, ws_bytes, false, stream);
}

spot_status spot_decode_step_q(const void* q_sel, const void* q_scale, int qfmt, const float* w,
                               const void* k_sel, const void* k_scale, int kfmt, int h_s,
                               int d_s, const int32_t* n_valid, float top_p, int k_max,
                               int k_min, int n_sink, int n_recent, const void* q, const void* k,
                               const void* v, const int32_t* seq_len, int batch, int h_q,
                               int h_kv, int d, int l_cap, float sm_scale, float* scores,
                               int32_t* idx, int32_t* count, float* nuc_mass, void* out,
                               float* lse, void* ws, size_t ws_bytes, void* stream) {
  return decode_step_impl(q_sel, q_scale, qfmt, w, k_sel, k_scale, kfmt, h_s, d_s, n_valid,
                          top_p, k_max, k_min, n_sink, n_recent, q, k, v, seq_len, batch, h_q,
                          h_kv, d, l_cap, sm_scale, scores, idx, count, nuc_mass, out, lse, ws,
                          ws_bytes, false, stream);
}

spot_status spot_decode_step_static(const void* q_sel, const float* w, const void* k_sel,
                                    const void* k_scale, int kfmt, int h_s, int d_s,
                                    const int32_t* n_valid, float top_p, int k_max, int k_min,
                                    int n_sink, int n_recent, const void* q, const void* k,
                                    const void* v, const int32_t* seq_len, int batch, int h_q,
                                    int h_kv, int d, int l_cap, float sm_scale, float* scores,
                                    int32_t* idx, int32_t* count, float* nuc_mass, void* out,
                                    float* lse, void* stream) {
  return decode_step_impl(q_sel, nullptr, SPOT_KFMT_BF16, w, k_sel, k_scale, kfmt, h_s, d_s,
                          n_valid, top_p, k_max, k_min, n_sink, n_recent, q, k, v, seq_len, batch,
                          h_q, h_kv, d, l_cap, sm_scale, scores, idx, count, nuc_mass, out, lse,
                          nullptr, 0, true, stream);
}

spot_status spot_decode_step_status(void* ws, size_t ws_bytes, int batch, int h_q, int h_kv,
                                    int d, int k_max, void* stream) {
  if (batch < 1 || h_q < 1 || h_kv < 1 || d < 1 || k_max < 1) return SPOT_ERR_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  StepWs L = step_layout(batch, h_q, h_kv, k_max, 0);
  if (!ws) {
    // the static scratch of spot_decode_step_static on the current device
    if (!step_static_fits(batch, h_q, h_kv, k_max)) return SPOT_ERR_WORKSPACE;
    if (static_scratch(&ws, false, s) != hipSuccess) return SPOT_ERR_HIP;
    if (!ws) return SPOT_OK;   // never used on this device
    L = step_static_layout(batch, h_q, h_kv, k_max);
    ws_bytes = L.total;
  }
  const size_t need = L.total;
  if (ws_bytes < need || misaligned(ws)) return SPOT_ERR_WORKSPACE;
  uint32_t word = 0;
  const char* w = static_cast<const char*>(ws) + L.sticky;
  if (hipMemcpyAsync(&word, w, sizeof(word), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return SPOT_ERR_HIP;
  if (word == 0u) return SPOT_OK;
  if (hipMemsetAsync(ws, 0, need, s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
    return SPOT_ERR_HIP;
  return SPOT_ERR_EXPIRED;
}

void spot_test_force_expiry(int on) { step_force_expiry(on); }

spot_status spot_sparse_prefill(const void* q, const void* k, const void* v, int L,
                                const int32_t* idx, const int32_t* count, int k_max, int batch,
                                int h_q, int h_kv, int d, float sm_scale, void* out, float* lse,
                                void* stream) {
  if (!q || !k || !v || !idx || !count || !out) return SPOT_ERR_NULL;
  if (L < 0 || L % kBlk || batch < 0 || k_max < 1 || h_q < 1 || h_kv < 1) return SPOT_ERR_SHAPE;
  if (d != 128 || !supported_prefill_group(h_q, h_kv) || k_max > 4096)
    return SPOT_ERR_UNSUPPORTED;
  if (!(sm_scale > 0.f) || sm_scale > 3.0e38f) return SPOT_ERR_UNSUPPORTED;
  if ((long long)batch * (L / kBlk) * h_kv > 0x0fffffffLL) return SPOT_ERR_SHAPE;
  if (batch == 0 || L == 0) return SPOT_OK;
  return from_hip(launch_sparse_prefill(q, k, v, L, idx, count, k_max, batch, h_q, h_kv,
                                        sm_scale, out, lse, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
