// Compaction internals: the tile queue's layout, the workspace it needs and
// the launch arguments (lethe_kv_compact).
#pragma once

#include "lethe_internal.h"

namespace lethe {

// Compaction moves rows in tiles of this many source rows.
constexpr int kCompactTile = 256;

// Tiles one queue entry holds at most (and at most kCompactTile kept rows
// between them).
constexpr int kCompactGroup = 4;

// One queue entry of the compaction: up to kCompactGroup consecutive tiles of
// one segment, holding at most kCompactTile kept rows between them.  The
// entries of a segment are consecutive in the queue, in row order, and so are
// their tiles' flags.
struct CompactItem {
  long long row0;  // first row of the segment (layer offset included)
  int32_t j0;      // first source row of the entry's first tile, relative to the segment
  int32_t end;     // one past the entry's last source row (<= len)
  int32_t base;    // destination of the entry's first kept row (rows kept before j0)
  int32_t tiles;   // tiles in the entry
  int32_t flag0;   // flag index of the entry's first tile
  // Flag indices of the earlier tiles whose source rows the entry's stores
  // overwrite: wlo .. whi (none if wlo > whi; at most two, since the stores
  // cover at most kCompactTile consecutive rows).
  int32_t wlo, whi;
  int32_t pad[7];
  unsigned long long kept[4 * kCompactGroup];  // bit i of word x: source row j0 + 64 x + i is kept
};
static_assert(sizeof(CompactItem) == 192, "queue entry");

// Queue entries a compaction workspace holds: every segment's tiles, each
// segment rounding up once.
inline int64_t compact_queue_cap(int64_t rows_per_layer, int L, int B, int HK) {
  return (int64_t)L * ((rows_per_layer + kCompactTile - 1) / kCompactTile + (int64_t)B * HK);
}

// Compaction workspace: kept counts [L][B][HK], queue entries, per-tile flags
// (and one flag that is never set).
inline size_t compact_counts_bytes(int L, int B, int HK) { return align_up((size_t)L * B * HK * sizeof(int32_t), 256); }
inline size_t compact_ws_bytes(int64_t rows_per_layer, int L, int B, int HK) {
  const size_t q = (size_t)compact_queue_cap(rows_per_layer, L, B, HK);
  return compact_counts_bytes(L, B, HK) + align_up(q * sizeof(CompactItem), 256) +
         align_up((q + 1) * sizeof(int32_t), 256);
}

struct CompactArgs {
  void* k;
  void* v;
  float* score;
  int32_t* len;
  const int64_t* seq_base;
  const int32_t* cap;
  int64_t rows_per_layer;
  int32_t l0;             // first layer of the call
  int32_t L, B, HK;       // L: layers of the call (l0 .. l0 + L - 1)
  int32_t row_bytes;      // D * element size
  const uint8_t* keep;
  int32_t* counts;        // ws [L][B][HK] (the call's layers)
  CompactItem* items;     // ws [qcap]
  int32_t* flags;         // ws [qcap]: per tile, its rows are loaded
  int32_t qcap;           // tiles (and so entries) the queue holds at most; flags[qcap] is never set
  int32_t spin_limit;     // flag polls a move block may spend in all
  int32_t test_wait;      // non-zero: every entry also waits for flags[qcap] (failure-path tests)
  // Decode state, returned to zero by the last launch: tiles appended (low
  // 32 bits) and entries appended (high 32 bits); entries taken.
  unsigned long long* qctl;
  int32_t* ticket;
  int32_t* hint;          // decode state [L][B]: tiling lengths, set to the new len
  int32_t* dev_status;
};

lethe_status launch_compact(const CompactArgs& a, hipStream_t s);

}  // namespace lethe
