// Host side of the C ABI: argument validation, workspace sizing and launch
// dispatch.  Every check here runs before any HIP call, so invalid calls
// return without touching the device.
#include <math.h>
#include <stdlib.h>

#include "compact_internal.h"
#include "lethe_internal.h"

using namespace lethe;

namespace {

size_t elem_bytes(lethe_dtype dt) { return dt == LETHE_BF16 ? 2 : 4; }

// Host-checkable validity of the sizes of a cache description.
lethe_status check_desc(const lethe_cache* c) {
  if (!c) return LETHE_ERR_INVALID;
  if (c->num_layers < 1 || c->num_seqs < 1 || c->num_q_heads < 1 || c->num_kv_heads < 1)
    return LETHE_ERR_INVALID;
  if (c->rows_per_layer < 1) return LETHE_ERR_INVALID;
  if (c->num_q_heads % c->num_kv_heads != 0) return LETHE_ERR_INVALID;
  if (c->dtype != LETHE_BF16 && c->dtype != LETHE_F32) return LETHE_ERR_INVALID;
  if (c->head_dim != 64 && c->head_dim != 128) return LETHE_ERR_UNSUPPORTED;
  int G = c->num_q_heads / c->num_kv_heads;
  if (G > 8) return LETHE_ERR_UNSUPPORTED;
  if (c->num_seqs > kMaxSeqs) return LETHE_ERR_UNSUPPORTED;
  if (c->num_layers > kMaxLayers) return LETHE_ERR_UNSUPPORTED;
  // Element offsets must stay within int64 and row indices within 2^40.
  if (c->rows_per_layer > ((int64_t)1 << 40) / c->num_layers) return LETHE_ERR_UNSUPPORTED;
  return LETHE_OK;
}

// Sizes plus the device pointers every call needs.
lethe_status check_cache(const lethe_cache* c) {
  lethe_status st = check_desc(c);
  if (st != LETHE_OK) return st;
  if (!c->k || !c->v || !c->score || !c->len || !c->seq_base || !c->cap || !c->dev_status || !c->state)
    return LETHE_ERR_INVALID;
  return LETHE_OK;
}

int group_size(const lethe_cache* c) { return c->num_q_heads / c->num_kv_heads; }

StateLayout state_of(const lethe_cache* c) {
  return state_layout(c->num_layers, c->num_seqs, c->num_kv_heads, group_size(c), c->head_dim, elem_bytes(c->dtype));
}

// Applies every pending decode step (no-op kernel blocks where none is).
// Applies the pending decode step of layers l0 .. l0 + nl - 1 (all of them by
// default) and refreshes their tiling hints.
lethe_status flush_pending(const lethe_cache* c, hipStream_t stream, int l0 = 0, int nl = -1) {
  const StateLayout sl = state_of(c);
  char* st = (char*)c->state;
  FlushArgs a;
  a.k = c->k;
  a.score = c->score;
  a.len = c->len;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.l0 = l0;
  a.L = nl < 0 ? c->num_layers : nl;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  if ((long long)a.L * a.B * a.HK == 0) return LETHE_OK;
  a.pend_len = (int32_t*)(st + sl.len_off);
  a.pend_par = (const int32_t*)(st + sl.par_off);
  a.pend_gamma = (const float*)(st + sl.gamma_off);
  a.pend_scale = (const float*)(st + sl.scale_off);
  a.segstat = (const float*)(st + sl.stat_off);
  a.qprev = st + sl.q_off;
  a.flush_cnt = (int32_t*)(st + sl.flush_cnt_off);
  a.hint = (int32_t*)(st + sl.hint_off);
  return launch_flush(a, c->dtype, c->head_dim, group_size(c), stream);
}

}  // namespace

extern "C" {

const char* lethe_status_string(lethe_status s) {
  switch (s) {
    case LETHE_OK: return "ok";
    case LETHE_ERR_INVALID: return "invalid argument";
    case LETHE_ERR_UNSUPPORTED: return "unsupported configuration";
    case LETHE_ERR_WORKSPACE: return "workspace too small";
    case LETHE_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

size_t lethe_workspace_bytes(const lethe_cache* c, int op) {
  if (check_desc(c) != LETHE_OK) return 0;
  switch (op) {
    case LETHE_OP_DECODE:
      return decode_ws_bytes(c->num_seqs, c->num_kv_heads, group_size(c), c->head_dim);
    case LETHE_OP_DECODE_FINAL:
      return decode_final_ws_bytes(c->num_seqs, c->num_kv_heads, group_size(c), c->head_dim, c->rows_per_layer);
    case LETHE_OP_SPARSITY:
      return 0;
    case LETHE_OP_SELECT:
      return 0;
    case LETHE_OP_COMPACT:
      return compact_ws_bytes(c->rows_per_layer, c->num_layers, c->num_seqs, c->num_kv_heads);
    case LETHE_OP_COMPACT_PLAN:
      return plan_ws_bytes(c->rows_per_layer, c->num_layers, c->num_seqs, c->num_kv_heads);
  }
  return 0;
}

size_t lethe_state_bytes(const lethe_cache* c) {
  if (check_desc(c) != LETHE_OK) return 0;
  return state_of(c).total;
}

lethe_status lethe_score_flush(const lethe_cache* c, hipStream_t stream) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  return flush_pending(c, stream);
}

}  // extern "C"

namespace {

// Host checks of a decode call's arguments (before any HIP call).
lethe_status check_decode(const lethe_cache* c, int32_t layer, const void* q, const void* k_new,
                          const void* v_new, float gamma, float softmax_scale, const float* out) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (layer < 0 || layer >= c->num_layers) return LETHE_ERR_INVALID;
  if (!q || !out) return LETHE_ERR_INVALID;
  if ((k_new == nullptr) != (v_new == nullptr)) return LETHE_ERR_INVALID;
  if (!(gamma > 0.0f && gamma <= 1.0f)) return LETHE_ERR_INVALID;  // also rejects NaN
  if (isnan(softmax_scale) || isinf(softmax_scale)) return LETHE_ERR_INVALID;
  return LETHE_OK;
}

// Launch arguments of a decode call whose arguments passed check_decode; ws
// holds at least one chunk partial per segment (and, settling, the logits
// after the partials of a full workspace).
DecodeArgs decode_args(const lethe_cache* c, int32_t layer, const void* q, const void* k_new, const void* v_new,
                       float gamma, float softmax_scale, float* out, void* ws, size_t ws_bytes, bool settle) {
  const int G = group_size(c);
  const int D = c->head_dim;
  float scale = softmax_scale > 0.0f ? softmax_scale : 1.0f / sqrtf((float)D);

  const size_t eb = elem_bytes(c->dtype);
  const size_t layer_off = (size_t)layer * (size_t)c->rows_per_layer * (size_t)D * eb;
  DecodeArgs a;
  a.k = (const char*)c->k + layer_off;
  a.v = (const char*)c->v + layer_off;
  a.k_w = (char*)c->k + layer_off;
  a.v_w = (char*)c->v + layer_off;
  a.score = c->score + (size_t)layer * (size_t)c->rows_per_layer;
  a.len = c->len + (size_t)layer * c->num_seqs;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.gamma = gamma;
  a.out = out;
  const StateLayout sl = state_of(c);
  char* st_base = (char*)c->state;
  const size_t lb = (size_t)layer * c->num_seqs;
  a.pend_len = (int32_t*)(st_base + sl.len_off) + lb;
  a.pend_par = (int32_t*)(st_base + sl.par_off) + lb;
  a.pend_gamma = (float*)(st_base + sl.gamma_off) + lb;
  a.pend_scale = (float*)(st_base + sl.scale_off) + lb;
  a.segstat = (float*)(st_base + sl.stat_off) + lb * c->num_kv_heads * 2 * G;
  a.qprev = st_base + sl.q_off + lb * 2 * (size_t)c->num_q_heads * D * eb;
  a.seg_cnt = (int32_t*)(st_base + sl.seg_cnt_off);
  a.seq_cnt = (int32_t*)(st_base + sl.seq_cnt_off);
  a.hint = (const int32_t*)(st_base + sl.hint_off) + lb;
  a.part = (float*)ws;
  const size_t part_bytes = settle ? decode_final_rows_off(c->num_seqs, c->num_kv_heads, G, D) : ws_bytes;
  a.part_cap = (int64_t)(part_bytes / ((size_t)part_stride(G, D) * sizeof(float)));
  a.dev_status = c->dev_status;
  a.nbt = a.nch_flat = 0;  // chosen by the launcher
  a.adaptive = a.steps_per_chunk = a.min_chunks = 0;  // chosen by the launcher
  a.deterministic = 0;
  a.logit = settle ? (float*)((char*)ws + decode_final_logit_off(c->num_seqs, c->num_kv_heads, G, D)) : nullptr;
  a.apply_rows = settle ? (int32_t*)((char*)ws + decode_final_rows_off(c->num_seqs, c->num_kv_heads, G, D)) : nullptr;
  a.seg_plan = nullptr;
  a.step_plan = nullptr;
  a.step_flag = nullptr;
  a.plan_steps = 0;
  a.spin_limit = 0;
  return a;
}

lethe_status decode_call(const lethe_cache* c, int32_t layer, const void* q, const void* k_new,
                         const void* v_new, float gamma, float softmax_scale, float* out, void* ws,
                         size_t ws_bytes, bool settle, hipStream_t stream) {
  const DecodeArgs a = decode_args(c, layer, q, k_new, v_new, gamma, softmax_scale, out, ws, ws_bytes, settle);
  return launch_decode(a, c->dtype, c->head_dim, group_size(c), stream);
}

// Where the parts of a compaction plan sit in its buffer.
struct PlanParts {
  int32_t* seg;
  int32_t* step;
  int32_t* flag;
  int64_t steps_per_layer;
};

PlanParts plan_parts(const lethe_cache* c, void* plan) {
  PlanParts p;
  char* w = (char*)plan;
  p.seg = (int32_t*)w;
  w += plan_seg_bytes(c->num_layers, c->num_seqs, c->num_kv_heads);
  p.step = (int32_t*)w;
  w += plan_step_bytes(c->rows_per_layer, c->num_layers, c->num_seqs, c->num_kv_heads);
  p.flag = (int32_t*)w;
  p.steps_per_layer = plan_steps_per_layer(c->rows_per_layer, c->num_seqs, c->num_kv_heads);
  return p;
}

// Bounded waits of the compacting decode: 2^20 flag polls per wavefront
// (about a second); LETHE_COMPACT_SPIN_LIMIT lowers it (tests).
int decode_spin_limit() {
  const char* e = getenv("LETHE_COMPACT_SPIN_LIMIT");
  const int v = e ? atoi(e) : 0;
  return (v > 0 && v < (1 << 20)) ? v : (1 << 20);
}

// Host limits of a plan: step indices are int32, and a block counts the
// heads of a (layer, sequence) in shared memory.
lethe_status check_plan_size(const lethe_cache* c) {
  const int64_t steps = plan_steps_per_layer(c->rows_per_layer, c->num_seqs, c->num_kv_heads) * c->num_layers;
  if (steps > 0x7fffffffLL || c->num_kv_heads > 64) return LETHE_ERR_UNSUPPORTED;
  return LETHE_OK;
}

}  // namespace

extern "C" {

lethe_status lethe_decode_attn_score(const lethe_cache* c, int32_t layer, const void* q,
                                     const void* k_new, const void* v_new, float gamma,
                                     float softmax_scale, float* out, void* ws, size_t ws_bytes,
                                     hipStream_t stream) {
  lethe_status st = check_decode(c, layer, q, k_new, v_new, gamma, softmax_scale, out);
  if (st != LETHE_OK) return st;
  if (!ws) return LETHE_ERR_INVALID;
  if (ws_bytes < decode_ws_bytes(c->num_seqs, c->num_kv_heads, group_size(c), c->head_dim))
    return LETHE_ERR_WORKSPACE;
  return decode_call(c, layer, q, k_new, v_new, gamma, softmax_scale, out, ws, ws_bytes, false, stream);
}

lethe_status lethe_decode_attn_score_final(const lethe_cache* c, int32_t layer, const void* q,
                                           const void* k_new, const void* v_new, float gamma,
                                           float softmax_scale, float* out, void* ws, size_t ws_bytes,
                                           hipStream_t stream) {
  lethe_status st = check_decode(c, layer, q, k_new, v_new, gamma, softmax_scale, out);
  if (st != LETHE_OK) return st;
  if (!ws) return LETHE_ERR_INVALID;
  if (ws_bytes < decode_final_ws_bytes(c->num_seqs, c->num_kv_heads, group_size(c), c->head_dim,
                                       c->rows_per_layer))
    return LETHE_ERR_WORKSPACE;
  return decode_call(c, layer, q, k_new, v_new, gamma, softmax_scale, out, ws, ws_bytes, true, stream);
}

lethe_status lethe_decode_attn_score_noalloc(const lethe_cache* c, int32_t layer, const void* q,
                                             const void* k_new, const void* v_new, float gamma,
                                             float softmax_scale, float* out, hipStream_t stream) {
  lethe_status st = check_decode(c, layer, q, k_new, v_new, gamma, softmax_scale, out);
  if (st != LETHE_OK) return st;
  // One chunk partial per segment must fit the static scratch.
  const size_t per_chunk = (size_t)part_stride(group_size(c), c->head_dim) * sizeof(float);
  if ((size_t)c->num_seqs * (size_t)c->num_kv_heads * per_chunk > kDecodeScratchBytes) return LETHE_ERR_UNSUPPORTED;
  void* scratch_ptr = nullptr;
  st = decode_scratch(&scratch_ptr);
  if (st != LETHE_OK) return st;
  return decode_call(c, layer, q, k_new, v_new, gamma, softmax_scale, out, scratch_ptr, kDecodeScratchBytes, false,
                     stream);
}

lethe_status lethe_layer_sparsity(const lethe_cache* c, const int64_t* global_budget,
                                  int32_t recent, int32_t sink, const float* sparsity_in,
                                  float* sparsity_out, int32_t* budget_out, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (!global_budget || !sparsity_out || !budget_out) return LETHE_ERR_INVALID;
  if (recent < 0 || sink < 0) return LETHE_ERR_INVALID;
  st = flush_pending(c, stream);
  if (st != LETHE_OK) return st;
  SparsityArgs a;
  a.score = c->score;
  a.len = c->len;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.L = c->num_layers;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  a.global_budget = global_budget;
  a.recent = recent;
  a.sink = sink;
  a.sparsity_in = sparsity_in;
  a.sparsity_out = sparsity_out;
  a.budget_out = budget_out;
  a.dev_status = c->dev_status;
  return launch_sparsity(a, stream);
}

namespace {

lethe::SelectArgs select_args(const lethe_cache* c, int32_t mode, uint8_t* keep) {
  lethe::SelectArgs a;
  a.score = c->score;
  a.len = c->len;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.L = c->num_layers;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  a.mode = mode;
  a.budget = nullptr;
  a.recent = 0;
  a.sink = 0;
  a.segments = 0;
  a.tau = 0.0f;
  a.evict = nullptr;
  a.breakpoint = nullptr;
  a.keep = keep;
  a.dev_status = c->dev_status;
  return a;
}

lethe_status rasr_select_mode(const lethe_cache* c, const int32_t* budget, int32_t recent,
                              int32_t sink, uint8_t* keep, int32_t mode, hipStream_t stream) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (!budget || !keep) return LETHE_ERR_INVALID;
  if (recent < 0 || sink < 0) return LETHE_ERR_INVALID;
  st = flush_pending(c, stream);
  if (st != LETHE_OK) return st;
  lethe::SelectArgs a = select_args(c, mode, keep);
  a.budget = budget;
  a.recent = recent;
  a.sink = sink;
  return lethe::launch_select(a, stream);
}

}  // namespace

lethe_status lethe_rasr_select(const lethe_cache* c, const int32_t* budget, int32_t recent,
                               int32_t sink, uint8_t* keep, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  return rasr_select_mode(c, budget, recent, sink, keep, lethe::kSelectRasr, stream);
}

lethe_status lethe_rasr_select_shared(const lethe_cache* c, const int32_t* budget, int32_t recent,
                                      int32_t sink, uint8_t* keep, void* ws, size_t ws_bytes,
                                      hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  return rasr_select_mode(c, budget, recent, sink, keep, lethe::kSelectRasrShared, stream);
}

lethe_status lethe_segmented_shrink(const lethe_cache* c, int32_t segments, float tau,
                                    int32_t recent, int32_t sink, int32_t* evict_threshold,
                                    int32_t* breakpoint, uint8_t* keep, void* ws, size_t ws_bytes,
                                    hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (!evict_threshold || !keep) return LETHE_ERR_INVALID;
  if (recent < 0 || sink < 0 || segments < 1) return LETHE_ERR_INVALID;
  if (!(tau > 1.0f) || !isfinite(tau)) return LETHE_ERR_INVALID;
  st = flush_pending(c, stream);
  if (st != LETHE_OK) return st;
  lethe::SelectArgs a = select_args(c, lethe::kSelectShrink, keep);
  a.recent = recent;
  a.sink = sink;
  a.segments = segments;
  a.tau = tau;
  a.evict = evict_threshold;
  a.breakpoint = breakpoint;
  return lethe::launch_select(a, stream);
}

size_t lethe_prefill_workspace_bytes(const lethe_cache* c, int64_t q_rows) {
  if (!c || q_rows <= 0 || c->num_q_heads <= 0) return 0;
  // (max, 1 / sum) per query row and head, plus slack for reads in pairs.
  return align_up((size_t)q_rows * (size_t)c->num_q_heads * 2 * sizeof(float) + 16, 256);
}

lethe_status lethe_prefill_attn_score(const lethe_cache* c, int32_t layer, const void* q,
                                      const int64_t* q_start, const int32_t* q_len, int64_t q_rows,
                                      int32_t max_q_len, int32_t max_kv_len, float softmax_scale,
                                      float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (c->dtype != LETHE_BF16) return LETHE_ERR_UNSUPPORTED;
  if (layer < 0 || layer >= c->num_layers) return LETHE_ERR_INVALID;
  if (!q_start || !q_len || q_rows < 0 || max_q_len < 0 || max_kv_len < 0) return LETHE_ERR_INVALID;
  if (q_rows > 0 && (!q || !out)) return LETHE_ERR_INVALID;
  if (isnan(softmax_scale) || isinf(softmax_scale)) return LETHE_ERR_INVALID;
  const size_t need = lethe_prefill_workspace_bytes(c, q_rows);
  if (need > 0 && (!ws || ws_bytes < need)) return LETHE_ERR_WORKSPACE;
  st = flush_pending(c, stream);
  if (st != LETHE_OK) return st;
  const int D = c->head_dim;
  const int G = c->num_q_heads / c->num_kv_heads;
  const float scale = softmax_scale > 0.0f ? softmax_scale : 1.0f / sqrtf((float)D);
  const size_t rowb = (size_t)D * 2;
  const size_t lrow = (size_t)layer * (size_t)c->rows_per_layer;
  PrefillArgs a;
  a.k = (const char*)c->k + lrow * rowb;
  a.v = (const char*)c->v + lrow * rowb;
  a.score = c->score + lrow;
  a.len = c->len;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.layer = layer;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  a.q = q;
  a.q_start = q_start;
  a.q_len = q_len;
  a.q_rows = q_rows;
  a.max_q = max_q_len;
  a.max_kv = max_kv_len;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.out = out;
  a.stat = (float*)ws;
  a.dev_status = c->dev_status;
  if (max_q_len == 0) return LETHE_OK;
  return launch_prefill(a, D, G, stream);
}

lethe_status lethe_kv_compact_layers(const lethe_cache* c, int32_t layer_begin, int32_t layer_count,
                                     const uint8_t* keep, void* ws, size_t ws_bytes, hipStream_t stream) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (!keep || !ws) return LETHE_ERR_INVALID;
  if (layer_begin < 0 || layer_count < 0 || layer_begin > c->num_layers - layer_count) return LETHE_ERR_INVALID;
  if (ws_bytes < lethe_workspace_bytes(c, LETHE_OP_COMPACT)) return LETHE_ERR_WORKSPACE;
  if (layer_count == 0) return LETHE_OK;
  st = flush_pending(c, stream, layer_begin, layer_count);
  if (st != LETHE_OK) return st;
  CompactArgs a;
  a.k = c->k;
  a.v = c->v;
  a.score = c->score;
  a.len = c->len;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.l0 = layer_begin;
  a.L = layer_count;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  a.row_bytes = c->head_dim * (int32_t)elem_bytes(c->dtype);
  a.keep = keep;
  const int64_t qcap = compact_queue_cap(c->rows_per_layer, a.L, a.B, a.HK);
  if (qcap > 0x3fffffffLL) return LETHE_ERR_UNSUPPORTED;
  char* w = (char*)ws;
  a.counts = (int32_t*)w;
  w += compact_counts_bytes(a.L, a.B, a.HK);
  a.items = (CompactItem*)w;
  w += align_up((size_t)qcap * sizeof(CompactItem), 256);
  a.flags = (int32_t*)w;
  a.qcap = (int32_t)qcap;
  const StateLayout sl = state_of(c);
  int32_t* cmp = (int32_t*)((char*)c->state + sl.cmp_off);
  a.qctl = (unsigned long long*)cmp;
  a.ticket = cmp + kCntStride;
  a.hint = (int32_t*)((char*)c->state + sl.hint_off);
  a.dev_status = c->dev_status;
  return launch_compact(a, stream);
}

lethe_status lethe_kv_compact(const lethe_cache* c, const uint8_t* keep, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  return lethe_kv_compact_layers(c, 0, c->num_layers, keep, ws, ws_bytes, stream);
}

lethe_status lethe_kv_compact_plan(const lethe_cache* c, const uint8_t* keep, void* plan, size_t plan_bytes,
                                   hipStream_t stream) {
  lethe_status st = check_cache(c);
  if (st != LETHE_OK) return st;
  if (!keep || !plan) return LETHE_ERR_INVALID;
  st = check_plan_size(c);
  if (st != LETHE_OK) return st;
  if (plan_bytes < plan_ws_bytes(c->rows_per_layer, c->num_layers, c->num_seqs, c->num_kv_heads))
    return LETHE_ERR_WORKSPACE;
  const PlanParts pp = plan_parts(c, plan);
  PlanArgs a;
  a.keep = keep;
  a.len = c->len;
  a.seq_base = c->seq_base;
  a.cap = c->cap;
  a.rows_per_layer = c->rows_per_layer;
  a.L = c->num_layers;
  a.B = c->num_seqs;
  a.HK = c->num_kv_heads;
  a.steps_per_layer = (int32_t)pp.steps_per_layer;
  a.seg_plan = pp.seg;
  a.step_plan = pp.step;
  a.step_flag = pp.flag;
  a.hint = (int32_t*)((char*)c->state + state_of(c).hint_off);
  a.dev_status = c->dev_status;
  return launch_plan(a, stream);
}

lethe_status lethe_decode_attn_score_compact(const lethe_cache* c, int32_t layer, const void* q,
                                             const void* k_new, const void* v_new, float gamma,
                                             float softmax_scale, float* out, void* plan, size_t plan_bytes,
                                             void* ws, size_t ws_bytes, hipStream_t stream) {
  lethe_status st = check_decode(c, layer, q, k_new, v_new, gamma, softmax_scale, out);
  if (st != LETHE_OK) return st;
  if (c->dtype != LETHE_BF16) return LETHE_ERR_UNSUPPORTED;
  st = check_plan_size(c);
  if (st != LETHE_OK) return st;
  if (!plan || !ws) return LETHE_ERR_INVALID;
  if (plan_bytes < plan_ws_bytes(c->rows_per_layer, c->num_layers, c->num_seqs, c->num_kv_heads))
    return LETHE_ERR_WORKSPACE;
  if (ws_bytes < decode_ws_bytes(c->num_seqs, c->num_kv_heads, group_size(c), c->head_dim))
    return LETHE_ERR_WORKSPACE;
  DecodeArgs a = decode_args(c, layer, q, k_new, v_new, gamma, softmax_scale, out, ws, ws_bytes, false);
  const PlanParts pp = plan_parts(c, plan);
  a.seg_plan = pp.seg + (size_t)layer * c->num_seqs * c->num_kv_heads * kSegPlanWords;
  a.step_plan = pp.step;
  a.step_flag = pp.flag;
  a.plan_steps = (int32_t)(pp.steps_per_layer * c->num_layers);
  a.spin_limit = decode_spin_limit();
  return launch_decode_compact(a, c->head_dim, group_size(c), stream);
}

}  // extern "C"
