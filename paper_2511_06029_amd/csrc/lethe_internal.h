// Internal declarations shared by the host entry points and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lethe.h"

namespace lethe {

// Largest batch (the budget kernel and the tests size arrays by it).
constexpr int kMaxSeqs = 1024;
// Largest number of layers the budget split handles.
constexpr int kMaxLayers = 256;
// Most chunks one (sequence, KV head) segment is split into per decode call.
constexpr int kMaxChunksPerSeg = 64;
// Most blocks a decode launch aims for beyond one per segment (the partial
// buffer holds one partial per block: this many plus one per segment).
constexpr int kMaxDecodeTarget = 4096;

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Per-cache decode state (lethe_cache::state), zero-filled once before first
// use; the calls keep it consistent afterwards.
//
// The score update of a decode step needs the step's final softmax max and
// sum per head, which exist only once every chunk of the segment is done.  A
// decode call therefore leaves its step pending: it keeps the step's query
// and scale and, per segment and head, (M, 1/L).  The next decode call on the
// layer recomputes the pending step's logits from the K rows it streams
// anyway and applies the update; a flush does the same on its own.
//   pend_len   [L][B]               rows with a pending contribution (0: none)
//   pend_par   [L][B]               which half of qprev holds the pending query
//   pend_gamma [L][B]               decay of the pending step
//   pend_scale [L][B]               softmax scale * log2(e) of the pending step
//   seg_cnt    [B*HK] x kCntStride  blocks of a segment done, and the
//                                   segment's next step (0 between calls)
//   seq_cnt    [B] x kCntStride     segments of a sequence done (0 between calls)
//   segstat    [L][B*HK][2G]        per head: M (max scaled logit), then 1 / L
//   qprev      [L][2][B][HQ][D]     queries (storage type), double buffered
//   hint       [L][B]               lengths the decode tiling balances by
//                                   (written by flush and compaction only,
//                                   so a decode launch sees one value)
// Counters sit kCntStride words apart so the atomics of different segments
// meet in different cache lines and memory channels.  A segment's slot also
// holds, kStepCounter words in, the counter its wavefronts take decode steps
// from.
constexpr int kCntStride = 64;
constexpr int kStepCounter = 32;

struct StateLayout {
  size_t len_off, par_off, gamma_off, scale_off, seg_cnt_off, seq_cnt_off, flush_cnt_off, cmp_off, stat_off, q_off,
      hint_off, total;
};

inline StateLayout state_layout(int L, int B, int HK, int G, int D, size_t elem_bytes) {
  StateLayout s;
  const size_t lb = (size_t)L * B;
  s.len_off = 0;
  s.par_off = align_up(lb * sizeof(int32_t), 256);
  s.gamma_off = s.par_off + align_up(lb * sizeof(int32_t), 256);
  s.scale_off = s.gamma_off + align_up(lb * sizeof(float), 256);
  s.seg_cnt_off = s.scale_off + align_up(lb * sizeof(float), 256);
  s.seq_cnt_off = s.seg_cnt_off + align_up((size_t)B * HK * kCntStride * sizeof(int32_t), 256);
  s.flush_cnt_off = s.seq_cnt_off + align_up((size_t)B * kCntStride * sizeof(int32_t), 256);
  s.cmp_off = s.flush_cnt_off + align_up(lb * sizeof(int32_t), 256);
  s.stat_off = s.cmp_off + align_up(2 * kCntStride * sizeof(int32_t), 256);
  s.q_off = s.stat_off + align_up(lb * HK * 2 * G * sizeof(float), 256);
  s.hint_off = s.q_off + align_up(lb * 2 * (size_t)HK * G * D * elem_bytes, 256);
  s.total = s.hint_off + align_up(lb * sizeof(int32_t), 256);
  return s;
}

// Floats per chunk partial (m, l, o[D] per head), padded to 128 bytes so no
// two chunks share a cache line.
__host__ __device__ inline int part_stride(int G, int D) { return (int)align_up((size_t)G * (D + 2), 32); }

// Chunks the partial buffer of a decode workspace holds.
inline int64_t decode_max_chunks(int B, int HK) { return (int64_t)B * HK + kMaxDecodeTarget; }

// Decode workspace: the chunk partials, scratch between calls.
inline size_t decode_ws_bytes(int B, int HK, int G, int D) {
  return align_up((size_t)decode_max_chunks(B, HK) * part_stride(G, D) * sizeof(float), 256);
}

// A decode call that settles its own score update also keeps, after the
// partials, the rows to update per sequence and every row's logits of the
// step: 8 floats per row of the layer (query heads of the group, padded).
constexpr int kLogitStride = 8;
inline size_t decode_final_rows_off(int B, int HK, int G, int D) { return decode_ws_bytes(B, HK, G, D); }
inline size_t decode_final_logit_off(int B, int HK, int G, int D) {
  return decode_final_rows_off(B, HK, G, D) + align_up((size_t)B * sizeof(int32_t), 256);
}
inline size_t decode_final_ws_bytes(int B, int HK, int G, int D, int64_t rows_per_layer) {
  return decode_final_logit_off(B, HK, G, D) + align_up((size_t)rows_per_layer * kLogitStride * sizeof(float), 256);
}

struct DecodeArgs {
  const void* k;         // layer base, rows x D of the storage type
  const void* v;
  void* k_w;             // same as k, writable (append)
  void* v_w;
  float* score;          // layer base
  int32_t* len;          // [B] of this layer
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t B, HK;
  const void* q;         // [B][HQ][D]
  const void* k_new;     // [B][HK][D] or null
  const void* v_new;
  float scale_log2;      // softmax scale * log2(e)
  float gamma;
  float* out;            // [B][HQ][D]
  int32_t* pend_len;     // state of this layer: [B]
  int32_t* pend_par;     // [B]
  float* pend_gamma;     // [B]
  float* pend_scale;     // [B]
  float* segstat;        // [B*HK][2G]
  void* qprev;           // [2][B][HQ][D]
  int32_t* seg_cnt;      // [B*HK] x kCntStride
  int32_t* seq_cnt;      // [B] x kCntStride
  const int32_t* hint;   // state [B] of this layer: tiling lengths
  float* part;           // workspace: one partial per block
  int64_t part_cap;      // chunk partials `part` holds (at least B * HK)
  int32_t* dev_status;
  int32_t nbt;           // blocks the tiling aims for (at most)
  int32_t adaptive;      // fewer chunks for small hinted totals
  int32_t steps_per_chunk; // adaptive split: hinted steps a chunk aims for
  int32_t min_chunks;    // adaptive split: fewest chunks (at most nbt)
  int32_t nch_flat;      // chunks per segment when every hint is 0
  int32_t deterministic; // fixed step schedule instead of the per-segment step counter
  // Compacting call only (else null): the plan lethe_kv_compact_plan wrote.
  const int32_t* seg_plan;  // this layer's [B*HK] x kSegPlanWords
  const int32_t* step_plan; // [steps] x 2: kept rows before the step, keep mask of its 32 rows
  int32_t* step_flag;       // [steps]: the step's rows have been read (set by this call)
  int32_t plan_steps;       // steps the plan's arrays hold
  int32_t spin_limit;       // flag polls a wavefront may spend in all
  // Settling call only (else null): the step's logits [rows_per_layer][8]
  // (raw q.k for bf16, scaled to log2 units for fp32) and the rows to
  // update per sequence (0: skipped), both in the workspace.
  float* logit;
  int32_t* apply_rows;
};

// Compaction that the next decode step carries out (lethe_kv_compact_plan,
// lethe_decode_attn_score_compact).  Per (layer, sequence, KV head) segment
// the plan keeps kSegPlanWords words: the live rows it was made for, the rows
// kept (-1: no valid plan), the first 32-row step holding an evicted row, and
// the index of the segment's step 0 in the per-step arrays.  Per step: the
// kept rows before it, the keep mask of its 32 rows, and a flag the decode
// sets once the step's rows have been read.  Steps of layer l start at
// l * plan_steps_per_layer; those of sequence b after the steps of every
// earlier sequence (ceil(cap / 32) per KV head).
constexpr int kSegPlanWords = 4;
inline int64_t plan_steps_per_layer(int64_t rows_per_layer, int B, int HK) {
  return (rows_per_layer + 31) / 32 + (int64_t)B * HK;
}
inline size_t plan_seg_bytes(int L, int B, int HK) {
  return align_up((size_t)L * B * HK * kSegPlanWords * sizeof(int32_t), 256);
}
inline size_t plan_step_bytes(int64_t rows_per_layer, int L, int B, int HK) {
  return align_up((size_t)L * plan_steps_per_layer(rows_per_layer, B, HK) * 2 * sizeof(int32_t), 256);
}
inline size_t plan_ws_bytes(int64_t rows_per_layer, int L, int B, int HK) {
  return plan_seg_bytes(L, B, HK) + plan_step_bytes(rows_per_layer, L, B, HK) +
         align_up((size_t)L * plan_steps_per_layer(rows_per_layer, B, HK) * sizeof(int32_t), 256);
}

struct PlanArgs {
  const uint8_t* keep;
  const int32_t* len;
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t L, B, HK;
  int32_t steps_per_layer;
  int32_t* seg_plan;
  int32_t* step_plan;
  int32_t* step_flag;
  int32_t* hint;          // decode state [L][B]: set to the rows kept
  int32_t* dev_status;
};

lethe_status launch_plan(const PlanArgs& a, hipStream_t s);

struct FlushArgs {
  const void* k;         // all layers
  float* score;
  const int32_t* len;    // [L][B]
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t l0;            // first layer of the launch
  int32_t L, B, HK;      // L: layers of the launch (l0 .. l0 + L - 1)
  int32_t* pend_len;     // state, all layers
  const int32_t* pend_par;
  const float* pend_gamma;
  const float* pend_scale;
  const float* segstat;
  const void* qprev;
  int32_t* flush_cnt;    // state [L][B]: flush blocks done with the pending state
  int32_t* hint;         // state [L][B]: tiling lengths, refreshed from len
};

lethe_status launch_flush(const FlushArgs& a, lethe_dtype dt, int D, int G, hipStream_t s);

lethe_status launch_decode(const DecodeArgs& a, lethe_dtype dt, int D, int G, hipStream_t s);
// The decode step that also carries out the plan's compaction (bf16 only).
lethe_status launch_decode_compact(const DecodeArgs& a, int D, int G, hipStream_t s);

// Device scratch of lethe_decode_attn_score_noalloc: a static array of this
// many bytes per device, holding the chunk partials of one call.
constexpr size_t kDecodeScratchBytes = (size_t)32 << 20;
// This device's address of that array (looked up once per device).
lethe_status decode_scratch(void** ptr);

struct SparsityArgs {
  const float* score;     // all layers
  const int32_t* len;     // [L][B]
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t L, B, HK;
  const int64_t* global_budget;
  int32_t recent, sink;
  const float* sparsity_in;
  float* sparsity_out;
  int32_t* budget_out;
  int32_t* dev_status;
};

lethe_status launch_sparsity(const SparsityArgs& a, hipStream_t s);

struct PrefillArgs {
  const void* k;          // the layer's first row
  const void* v;
  float* score;           // the layer's first row
  const int32_t* len;     // [L][B]
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t layer, B, HK;
  const void* q;          // [q_rows][H_Q][D]
  const int64_t* q_start; // [B]
  const int32_t* q_len;   // [B]
  int64_t q_rows;
  int32_t max_q, max_kv;
  float scale_log2;       // softmax scale * log2(e)
  float* out;             // fp32 [q_rows][H_Q][D]
  float* stat;            // fp32 [q_rows][H_Q][2]: max (base 2), 1 / sum
  int32_t* dev_status;
};

lethe_status launch_prefill(const PrefillArgs& a, int D, int G, hipStream_t s);

// Selection rules of launch_select.
enum SelectMode : int32_t {
  kSelectRasr = 0,        // RASR per (layer, sequence, KV head)
  kSelectRasrShared = 1,  // RASR on the head-summed score, one mask per (layer, sequence)
  kSelectShrink = 2,      // Algorithm 1 with the size trigger, head-summed score
};
constexpr int32_t kShrinkNoBreakpoint = -1;
constexpr int32_t kShrinkNotTriggered = -2;

struct SelectArgs {
  const float* score;
  const int32_t* len;
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t L, B, HK;
  int32_t mode;           // SelectMode
  const int32_t* budget;  // [B][L], RASR modes
  int32_t recent, sink;
  int32_t segments;       // cut points of Algorithm 1: segments - 1
  float tau;              // Algorithm 1 ratio threshold (> 1)
  int32_t* evict;         // [L][B] eviction thresholds, in/out (shrink)
  int32_t* breakpoint;    // [L][B] or null (shrink)
  uint8_t* keep;
  int32_t* dev_status;
};

lethe_status launch_select(const SelectArgs& a, hipStream_t s);

}  // namespace lethe
