// In-place, order-preserving compaction of K, V and score rows, gfx950.
//
// Three launches.
//
// compact_plan_kernel, one wavefront per (layer, sequence, KV head) segment:
// rows before the first evicted row stay where they are (it is found with 32
// independent flag loads per lane).  From the 256-row tile holding that row
// to the end, the wavefront takes the keep mask and kept count of every tile
// and groups consecutive tiles into queue entries of up to four tiles that
// keep at most 256 rows between them (sparse tiles, as in the first round of
// a full cache, share an entry; dense ones have one each).  It appends the
// entries, in row order, to a work queue (one append per block of eight
// segments); an entry carries its source rows, their keep masks, the
// destination of its first kept row (the rows kept before it) and the flags
// of the earlier tiles its stores overwrite.  Every tile has a flag.
//
// compact_move_kernel, persistent: blocks take queue entries in queue order
// from a ticket counter.  For an entry the block lists the kept rows from the
// masks, loads them into registers (16 bytes per lane), and once every load
// has completed sets its tiles' flags.  It then waits for the flags of the
// earlier tiles whose rows its stores overwrite (at most two: the stores
// cover at most 256 consecutive rows, and every tile spans 256), and stores
// the rows at their destinations.  So that an entry costs about one memory
// round trip, a block asks for its next ticket as soon as it has the current
// one, reads the flags it waits for together with the rows, and loads the
// next entry before its stores go out.  (Tickets of several entries would
// either put consecutive tiles of a segment in one block, one after the
// other, or make an entry wait for a later ticket, which only a launch whose
// blocks are all resident could allow.)
//
// Why the order is right: a destination never exceeds its source, so the
// stores of an entry reach only rows below the entry's end: rows of its own
// tiles (all loaded before the block's barrier) or of earlier tiles of the
// same segment (loaded before their flags were set).  No block reads a row
// another block of the launch writes, so the flags order loads before stores
// and carry no data; they need no acquire or release.  Why every wait ends: a
// block sets its tiles' flags before it waits for anything, and the entries
// holding the tiles it waits for were taken from the ticket counter before
// its own, by blocks that are running or done.  A bounded spin still turns a
// wait that would not end into LETHE_DEV_WAIT_TIMEOUT instead of a hang.
//
// compact_len_kernel sets the new lengths and resets the queue counters for
// the next call.
#include "device_common.h"
#include "compact_internal.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 512;
constexpr int kTile = kCompactTile;
constexpr int kTileWaves = kTile / kWave;
constexpr int kPlanThreads = 512;  // one wavefront per segment
constexpr int kPlanWaves = kPlanThreads / kWave;
// Upper bound on the flag polls of one block over the whole launch (a poll is
// a short sleep and a load from memory, about a microsecond): one to two
// seconds, against at most the launch's own duration (milliseconds) for real
// waits.  A block past it waits no more.  LETHE_COMPACT_SPIN_LIMIT lowers it;
// LETHE_COMPACT_TEST_WAIT=1 makes every entry also wait for a flag nothing
// sets, so that tests can drive the timeout path (every block still exits).
constexpr int kSpinLimit = 1 << 20;
// 16 bytes of a row; a vector type, so arrays of them stay in registers.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
// Queue entries as the move launch sees them: written by the plan launch and
// read-only here, so they may be read through the scalar cache.
typedef __attribute__((address_space(4))) const CompactItem ConstItem;

__device__ inline CompactItem load_item(const ConstItem* p) {
  CompactItem r;
  r.row0 = p->row0;
  r.j0 = p->j0;
  r.end = p->end;
  r.base = p->base;
  r.tiles = p->tiles;
  r.flag0 = p->flag0;
  r.wlo = p->wlo;
  r.whi = p->whi;
#pragma unroll
  for (int x = 0; x < 7; ++x) r.pad[x] = 0;
#pragma unroll
  for (int x = 0; x < 4 * kCompactGroup; ++x) r.kept[x] = p->kept[x];
  return r;
}

__global__ __launch_bounds__(kPlanThreads) void compact_plan_kernel(CompactArgs a) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const long long nseg = (long long)a.L * a.B * a.HK;
  const long long cidx = (long long)blockIdx.x * kPlanWaves + w;  // this wave's segment
  __shared__ int s_m[kPlanWaves];  // moved tiles per segment
  __shared__ int s_e[kPlanWaves];  // queue entries per segment
  __shared__ int s_base, s_ebase;

  // The wave's segment: its length, first evicted row and moved tiles.
  bool valid = false;
  int n = 0, first = 0, ft = 0, nt = 0;
  long long row0 = 0;
  if (cidx < nseg) {
    const int h = (int)(cidx % a.HK);
    const int b = (int)((cidx / a.HK) % a.B);
    const int l = a.l0 + (int)(cidx / ((long long)a.HK * a.B));
    n = a.len[(long long)l * a.B + b];
    const int c = a.cap[b];
    const long long base = a.seq_base[b];
    if (n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer) {
      if (lane == 0) {
        a.counts[cidx] = -1;
        atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
      }
    } else {
      valid = true;
      row0 = (long long)l * a.rows_per_layer + base + (long long)h * c;
    }
  }
  const uint8_t* keep = a.keep + row0;
  first = n;
  if (valid) {
    // First evicted row: 32 independent flag loads per lane and round, the
    // lowest evicted row of the round found by a wave minimum.
    for (int c0 = 0; c0 < n && first == n; c0 += 32 * kWave) {
      uint8_t kv[32];
#pragma unroll
      for (int k = 0; k < 32; ++k) kv[k] = keep[min(c0 + k * kWave + lane, n - 1)];
      int f = n;
#pragma unroll
      for (int k = 31; k >= 0; --k) {
        const int j = c0 + k * kWave + lane;
        if (j < n && kv[k] == 0) f = j;
      }
#pragma unroll
      for (int off = kWave / 2; off > 0; off >>= 1) f = min(f, __shfl_xor(f, off));
      first = f;
    }
    ft = first / kTile;
    nt = first < n ? (n + kTile - 1) / kTile : ft;
  }
  // Pass 1: kept count of every moved tile and the number of entries: runs of
  // up to kCompactGroup tiles that keep at most kTile rows between them.
  int ne = 0;
  {
    int glen = 0, gcnt = 0;
    for (int g = ft; g < nt; g += 4) {
      uint8_t f[4][4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int x = 0; x < 4; ++x) f[u][x] = keep[min((g + u) * kTile + kWave * x + lane, n - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = g + u;
        if (t >= nt) break;
        int kc = 0;
#pragma unroll
        for (int x = 0; x < 4; ++x) kc += __popcll(__ballot(t * kTile + kWave * x + lane < n && f[u][x] != 0));
        if (glen > 0 && (gcnt + kc > kTile || glen == kCompactGroup)) {
          ++ne;
          glen = gcnt = 0;
        }
        ++glen;
        gcnt += kc;
      }
    }
    if (glen > 0) ++ne;
  }
  // One queue append for the block's segments: tiles in the low half of the
  // counter, entries in the high half.
  if (blockIdx.x == 0 && tid == 0) a.flags[a.qcap] = 0;  // the flag nothing sets
  if (lane == 0) {
    s_m[w] = nt - ft;
    s_e[w] = ne;
  }
  __syncthreads();
  if (tid == 0) {
    unsigned long long add = 0;
    for (int x = 0; x < kPlanWaves; ++x) add += ((unsigned long long)s_e[x] << 32) + (unsigned long long)s_m[x];
    int tpos = 0, epos = 0;
    if (add != 0) {
      const unsigned long long old = atomicAdd(a.qctl, add);
      tpos = (int)(old & 0xffffffffull);
      epos = (int)(old >> 32);
      // Only segments that overlap other sequences' rows can overfill the queue.
      if (tpos > a.qcap - (int)(add & 0xffffffffull)) tpos = -1;
    }
    s_base = tpos;
    s_ebase = epos;
  }
  __syncthreads();
  if (!valid) return;
  if (first >= n) {
    if (lane == 0) a.counts[cidx] = n;
    return;
  }
  int tpos0 = s_base, epos = s_ebase;  // this segment's first flag and entry
  for (int x = 0; x < w; ++x) {
    tpos0 += s_m[x];
    epos += s_e[x];
  }
  if (s_base < 0) {
    // The block's tiles did not fit the queue (only segments that overlap
    // other sequences' rows get here).  Its entries still count in the entry
    // half of the counter; those below the queue's end become empty entries,
    // which the move launch skips.
    if (lane == 0) {
      for (int e = epos; e < epos + ne && e < a.qcap; ++e) {
        CompactItem* it = a.items + e;
        it->row0 = 0;
        it->j0 = it->end = it->base = it->tiles = it->flag0 = 0;
        it->wlo = 0;
        it->whi = -1;
      }
      a.counts[cidx] = -1;
      atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    }
    return;
  }

  // Pass 2: the same runs, written out.  An entry's header is written when it
  // closes, its mask words as its tiles come.
  int running = ft * kTile;  // rows kept before tile ft: all of them
  int glen = 0, gcnt = 0, gt0 = ft, gbase = running;
  auto close_entry = [&]() {
    if (lane == 0) {
      CompactItem* it = a.items + epos;
      it->row0 = row0;
      it->j0 = gt0 * kTile;
      it->end = min((gt0 + glen) * kTile, n);
      it->base = gbase;
      it->tiles = glen;
      it->flag0 = tpos0 + (gt0 - ft);
      // Destinations gbase + [0, gcnt) lie in the source ranges of tiles lo ..
      // hi; those before tile ft never move and are never overwritten.
      const int lo = max(ft, gbase / kTile);
      const int hi = min(gt0 - 1, (gbase + gcnt - 1) / kTile);
      const bool wait = gcnt > 0 && lo <= hi;
      it->wlo = wait ? tpos0 + (lo - ft) : 0;
      it->whi = wait ? tpos0 + (hi - ft) : -1;
    }
    ++epos;
  };
  for (int g = ft; g < nt; g += 4) {
    uint8_t f[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int x = 0; x < 4; ++x) f[u][x] = keep[min((g + u) * kTile + kWave * x + lane, n - 1)];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = g + u;
      if (t >= nt) break;
      unsigned long long km[4];
      int kc = 0;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        km[x] = __ballot(t * kTile + kWave * x + lane < n && f[u][x] != 0);
        kc += __popcll(km[x]);
      }
      if (glen > 0 && (gcnt + kc > kTile || glen == kCompactGroup)) {
        close_entry();
        glen = gcnt = 0;
        gt0 = t;
        gbase = running;
      }
      if (lane == 0) {
#pragma unroll
        for (int x = 0; x < 4; ++x) a.items[epos].kept[4 * glen + x] = km[x];
        a.flags[tpos0 + (t - ft)] = 0;
      }
      ++glen;
      gcnt += kc;
      running += kc;
    }
  }
  close_entry();
  if (lane == 0) a.counts[cidx] = running;
}

template <int RB>  // row bytes of K (= of V)
__global__ __launch_bounds__(kThreads) void compact_move_kernel(CompactArgs a) {
  constexpr int TPR = RB / 16;              // threads per row
  constexpr int RPP = kThreads / TPR;       // rows per pass
  constexpr int PASSES = kTile / RPP;
  static_assert(kTile % RPP == 0, "tile");
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int sub = tid % TPR;
  __shared__ int s_t;
  __shared__ int s_src[kTile];  // the tile's kept rows in order
  // Written by the plan launch; capped as the plan capped its appends.
  const int total = min((int)(*a.qctl >> 32), a.qcap);
  int spins = 0;  // thread 0's polls so far
  const ConstItem* items = (const ConstItem*)a.items;

  if (tid == 0) s_t = atomicAdd(a.ticket, 1);
  __syncthreads();
  // Block-uniform, so the entries load into scalar registers.
  int t = __builtin_amdgcn_readfirstlane(s_t);
  CompactItem it;
  if (t < total) it = load_item(items + t);
  while (t < total) {
    // The next ticket; its reply is only read after this tile's loads.
    int tnext = 0;
    if (tid == 0) tnext = atomicAdd(a.ticket, 1);
    char* K = reinterpret_cast<char*>(a.k) + it.row0 * RB;
    char* V = reinterpret_cast<char*>(a.v) + it.row0 * RB;
    float* S = a.score + it.row0;

    // The entry's kept rows in order: wavefront w lists mask words w and
    // w + 8 (words past the entry's tiles count as empty).
    constexpr int kWords = 4 * kCompactGroup;
    int cw[kWords];
    int cnt = 0;
#pragma unroll
    for (int x = 0; x < kWords; ++x) {
      cw[x] = x < 4 * it.tiles ? __popcll(it.kept[x]) : 0;
      cnt += cw[x];
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int x = w + (kThreads / kWave) * half;
      unsigned long long m = 0;  // word x, without indexing by x
      int before = 0;
#pragma unroll
      for (int y = 0; y < kWords; ++y) {
        m = y == x ? it.kept[y] : m;
        before += y < x ? cw[y] : 0;
      }
      if (x < 4 * it.tiles && ((m >> lane) & 1ull)) {
        before += __popcll(m & ((1ull << lane) - 1ull));
        s_src[before] = it.j0 + kWave * x + lane;
      }
    }
    __syncthreads();
    // Rows whose destination is their source (before the first evicted row
    // of the segment's first moved tile) are left alone.  K and V rows are
    // copied once and not touched again in this launch: their loads and
    // stores carry the non-temporal policy.
    u32x4_t rk[PASSES], rv[PASSES];
    float rs[PASSES];
    unsigned moved = 0;  // bit p: the row of pass p moves
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int i = p * RPP + tid / TPR;
      if (i < cnt) {
        const int src = s_src[i];
        if (src != it.base + i) {
          moved |= 1u << p;
          rk[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(K + (long long)src * RB + sub * 16));
          rv[p] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(V + (long long)src * RB + sub * 16));
          rs[p] = sub == 0 ? S[src] : 0.0f;
        }
      }
    }
    // First look at the flags this entry waits for, in flight with the rows.
    int fnear = 1, ffar = 1;
    if (tid == 0 && it.wlo <= it.whi) {
      fnear = __hip_atomic_load(&a.flags[it.whi], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ffar = __hip_atomic_load(&a.flags[it.wlo], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0);
    if (tid == 0) s_t = tnext;
    __syncthreads();  // every load of the tile has completed
    if (tid < it.tiles) __hip_atomic_store(&a.flags[it.flag0 + tid], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (tid == 0) {
      auto wait_flag = [&](int k) {
        while (spins <= a.spin_limit &&
               __hip_atomic_load(&a.flags[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
          if (++spins > a.spin_limit) {
            atomicOr(a.dev_status, LETHE_DEV_WAIT_TIMEOUT);
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
      };
      if (fnear == 0 || ffar == 0)
        for (int k = it.wlo; k <= it.whi; ++k) wait_flag(k);
      if (a.test_wait) wait_flag(a.qcap);
    }
    const int tn = __builtin_amdgcn_readfirstlane(s_t);
    CompactItem itn = it;
    if (tn < total) itn = load_item(items + tn);  // in flight during the stores
    __syncthreads();  // the earlier tiles this one overwrites have loaded their rows; s_t read
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int i = p * RPP + tid / TPR;
      const long long dst = it.base + i;
      // (Not s_src: threads already on the next tile may be rewriting it.)
      if ((moved >> p) & 1u) {
        __builtin_nontemporal_store(rk[p], reinterpret_cast<u32x4_t*>(K + dst * RB + sub * 16));
        __builtin_nontemporal_store(rv[p], reinterpret_cast<u32x4_t*>(V + dst * RB + sub * 16));
        if (sub == 0) S[dst] = rs[p];
      }
    }
    t = tn;
    it = itn;
  }
}

// New length of every (layer, sequence) of the call: the kept count, equal
// across heads.
// Also returns the queue counters to zero for the next call.
__global__ void compact_len_kernel(CompactArgs a) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) {
    *a.qctl = 0;
    *a.ticket = 0;
  }
  if (i >= (long long)a.L * a.B) return;
  const int* cnt = a.counts + i * a.HK;
  int mn = cnt[0], mx = cnt[0];
  for (int h = 1; h < a.HK; ++h) {
    mn = min(mn, cnt[h]);
    mx = max(mx, cnt[h]);
  }
  if (mn < 0) return;  // bad layout, already flagged
  if (mn != mx) atomicOr(a.dev_status, LETHE_DEV_HEAD_MISMATCH);
  const long long lb = (long long)a.l0 * a.B + i;
  a.len[lb] = mn;
  a.hint[lb] = mn;
}

int env_int(const char* name, int dflt) {
  const char* e = getenv(name);
  const int v = e ? atoi(e) : 0;
  return v > 0 ? v : dflt;
}

int move_blocks() {
  // Persistent grid: two resident blocks per CU (the 256-byte-row kernel
  // holds 119 VGPRs, four waves per SIMD).
  static const int n = env_int("LETHE_COMPACT_BLOCKS", 512);
  return n;
}

}  // namespace

// ---------------------------------------------------------------------------
// Plan of a compaction that the next decode step carries out
// ---------------------------------------------------------------------------
// One block per (layer, sequence), one wavefront per KV head.  The wavefront
// walks its segment's keep mask 64 rows at a time (16 loads a lane in
// flight) and records, per 32-row step, the kept rows before the step and the
// step's keep mask; it also finds the first step holding an evicted row and
// clears the step flags the decode will set.  The block then checks that the
// heads keep the same count (the new length is shared by the heads).
constexpr int kPlanBatch = 16;  // 64-row groups a lane loads before it uses the first

__device__ inline int wave_sum_i32(int v) {
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Heads a plan block holds counts for (host-checked).
constexpr int kPlanMaxHeads = 64;

__global__ __launch_bounds__(kWave * 8) void step_plan_kernel(PlanArgs a) {
  const int lb = blockIdx.x;
  const int l = lb / a.B;
  const int b = lb - l * a.B;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int nw = blockDim.x / kWave;
  __shared__ int s_kept[kPlanMaxHeads];
  __shared__ int s_part[8];
  // Steps of the earlier sequences of this layer: HK * ceil(cap / 32) each.
  int part = 0;
  for (int bb = tid; bb < b; bb += blockDim.x) part += (max(a.cap[bb], 0) + 31) >> 5;
  part = wave_sum_i32(part);
  if (lane == 0) s_part[w] = part;
  __syncthreads();
  long long before = 0;
  for (int x = 0; x < nw; ++x) before += s_part[x];
  const int n = a.len[lb];
  const int c = a.cap[b];
  const long long base = a.seq_base[b];
  const int cs = (max(c, 0) + 31) >> 5;  // steps of one KV head's segment
  // Segments that overlap (capacities summing past the layer) would run past
  // the layer's steps: flagged like any other bad layout.
  const bool bad = n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer ||
                   (before + cs) * a.HK > a.steps_per_layer;
  for (int h = w; h < a.HK; h += nw) {
    const long long step0 = (long long)l * a.steps_per_layer + before * a.HK + (long long)h * cs;
    int kept = 0, t0 = 0;
    if (!bad) {
      const uint8_t* keep = a.keep + (long long)l * a.rows_per_layer + base + (long long)h * c;
      const int nst = (n + 31) >> 5;
      t0 = nst;
      for (int j0 = 0; j0 < n; j0 += kPlanBatch * kWave) {
        uint8_t kv[kPlanBatch];
#pragma unroll
        for (int u = 0; u < kPlanBatch; ++u) kv[u] = keep[min(j0 + u * kWave + lane, n - 1)];
#pragma unroll
        for (int u = 0; u < kPlanBatch; ++u) {
          const int r0 = j0 + u * kWave;
          if (r0 >= n) break;
          const unsigned long long live = __ballot(r0 + lane < n);
          const unsigned long long m = __ballot(r0 + lane < n && kv[u] != 0);
          const unsigned long long ev = live & ~m;
          if (ev != 0ull && t0 == nst) t0 = (r0 + (int)__builtin_ctzll(ev)) >> 5;
          const long long t = step0 + (r0 >> 5);
          const int lo = __popcll(m & 0xffffffffull);
          if (lane == 0) {
            a.step_plan[2 * t] = kept;
            a.step_plan[2 * t + 1] = (int32_t)(uint32_t)m;
            if (r0 + 32 < n) {
              a.step_plan[2 * t + 2] = kept + lo;
              a.step_plan[2 * t + 3] = (int32_t)(uint32_t)(m >> 32);
            }
          }
          kept += __popcll(m);
        }
      }
      for (int t = lane; t < nst; t += kWave) a.step_flag[step0 + t] = 0;
    }
    if (lane == 0) {
      s_kept[h] = bad ? -1 : kept;
      int32_t* sp = a.seg_plan + ((long long)lb * a.HK + h) * kSegPlanWords;
      sp[0] = n;
      sp[2] = t0;
      sp[3] = (int32_t)step0;
    }
  }
  __syncthreads();
  bool same = true;
  for (int x = 0; x < a.HK; ++x) same = same && s_kept[x] == s_kept[0];
  const bool valid = !bad && same;
  for (int h = tid; h < a.HK; h += blockDim.x)
    a.seg_plan[((long long)lb * a.HK + h) * kSegPlanWords + 1] = valid ? s_kept[h] : -1;
  if (tid == 0) {
    if (bad) atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    else if (!same) atomicOr(a.dev_status, LETHE_DEV_HEAD_MISMATCH);
    a.hint[lb] = valid ? s_kept[0] : n;
  }
}

lethe_status launch_plan(const PlanArgs& a, hipStream_t s) {
  const long long nb = (long long)a.L * a.B;
  if (nb > 0x7fffffffLL) return LETHE_ERR_UNSUPPORTED;
  if (a.HK > kPlanMaxHeads) return LETHE_ERR_UNSUPPORTED;
  const int waves = a.HK < 8 ? a.HK : 8;
  hipLaunchKernelGGL(step_plan_kernel, dim3((unsigned)nb), dim3(kWave * waves), 0, s, a);
  return hipGetLastError() == hipSuccess ? LETHE_OK : LETHE_ERR_HIP;
}

lethe_status launch_compact(const CompactArgs& args, hipStream_t s) {
  static const int spin_limit = env_int("LETHE_COMPACT_SPIN_LIMIT", kSpinLimit);
  static const int test_wait = env_int("LETHE_COMPACT_TEST_WAIT", 0);
  CompactArgs a = args;
  a.spin_limit = std::min(spin_limit, kSpinLimit);
  a.test_wait = test_wait;
  long long nb = (long long)a.L * a.B * a.HK;
  if (nb > 0x7fffffffLL) return LETHE_ERR_UNSUPPORTED;
  if (a.row_bytes != 128 && a.row_bytes != 256 && a.row_bytes != 512) return LETHE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(compact_plan_kernel, dim3((unsigned)((nb + kPlanWaves - 1) / kPlanWaves)), dim3(kPlanThreads),
                     0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  const int mb = (int)std::min<long long>(move_blocks(), std::max(a.qcap, 1));
  switch (a.row_bytes) {
    case 128: hipLaunchKernelGGL(compact_move_kernel<128>, dim3(mb), dim3(kThreads), 0, s, a); break;
    case 256: hipLaunchKernelGGL(compact_move_kernel<256>, dim3(mb), dim3(kThreads), 0, s, a); break;
    case 512: hipLaunchKernelGGL(compact_move_kernel<512>, dim3(mb), dim3(kThreads), 0, s, a); break;
  }
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  long long nl = (long long)a.L * a.B;
  hipLaunchKernelGGL(compact_len_kernel, dim3((unsigned)((nl + 255) / 256)), dim3(256), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

}  // namespace lethe
