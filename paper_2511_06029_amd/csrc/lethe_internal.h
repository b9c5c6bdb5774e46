// Internal declarations shared by the host entry points and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lethe.h"

namespace lethe {

// Largest batch the decode planner keeps in LDS.
constexpr int kMaxSeqs = 1024;
// Largest number of layers the budget split handles.
constexpr int kMaxLayers = 256;
// Upper bounds on decode blocks and on the chunk target of one launch; the
// workspace is sized for kMaxDecodeTasks + num_seqs * num_kv_heads chunks.
constexpr int kMaxDecodeBlocks = 4096;
constexpr int kMaxDecodeTasks = 8192;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Decode workspace layout (bytes from ws); nothing in it needs to be
// initialised, every word is written before it is read within a call:
//   plan   header (chunk rows, chunk count) + n_att[kMaxSeqs] + flag[kMaxSeqs]
//   part   per chunk and head: m, l, o[D]
//   pend   per row and head: scaled logit of the current step
struct DecodeWs {
  size_t plan_off, part_off, pend_off, total;
};

enum PlanField { kPlanC = 0, kPlanTasks = 1, kPlanHdr = 16 };

inline DecodeWs decode_ws_layout(int B, int HK, int G, int D, int64_t rows_per_layer) {
  DecodeWs w;
  const size_t segs = (size_t)B * HK;
  const size_t max_chunks = (size_t)kMaxDecodeTasks + segs;
  w.plan_off = 0;
  w.part_off = align_up(sizeof(int32_t) * (kPlanHdr + 2 * (size_t)kMaxSeqs), 256);
  w.pend_off = w.part_off + align_up(max_chunks * (size_t)G * (D + 2) * sizeof(float), 256);
  w.total = w.pend_off + align_up((size_t)rows_per_layer * G * sizeof(float), 256);
  return w;
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
  int32_t* plan;         // ws
  float* part;
  float* pend;
  int32_t* dev_status;
  int32_t target_tasks;  // attention chunks to aim for (0: one per resident block)
  int32_t min_chunk;     // smallest chunk, rows (0: default)
};

lethe_status launch_decode(const DecodeArgs& a, lethe_dtype dt, int D, int G, hipStream_t s);

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

struct SelectArgs {
  const float* score;
  const int32_t* len;
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t L, B, HK;
  const int32_t* budget;  // [B][L]
  int32_t recent, sink;
  uint8_t* keep;
  int32_t* dev_status;
};

lethe_status launch_select(const SelectArgs& a, hipStream_t s);

struct CompactArgs {
  void* k;
  void* v;
  float* score;
  int32_t* len;
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t L, B, HK;
  int32_t row_bytes;      // D * element size
  const uint8_t* keep;
  int32_t* counts;        // ws [L][B][HK]
  int32_t* dev_status;
};

lethe_status launch_compact(const CompactArgs& a, hipStream_t s);

}  // namespace lethe
