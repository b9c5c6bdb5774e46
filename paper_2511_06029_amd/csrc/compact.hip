// In-place, order-preserving compaction of K, V and score rows, gfx950.
//
// Three launches.
//
// compact_plan_kernel, one wavefront per (layer, sequence, KV head) segment:
// rows before the first evicted row stay where they are (it is found with 32
// independent flag loads per lane).  From the 256-row tile holding that row
// to the end, the wavefront takes the keep mask and kept count of every tile
// and appends the tiles, in row order, to a work queue (one append per block
// of eight segments: a single counter serves every append); an entry carries
// the tile's source rows, its keep mask and the destination of its first
// kept row (the rows kept before it).
//
// compact_move_kernel, persistent: blocks take queue entries in queue order
// from a ticket counter.  For an entry the block lists the tile's kept rows
// from the mask, loads them into registers (16 bytes per lane), and once
// every load has completed marks the entry's flag.  It then waits for the
// flags of the earlier tiles of the segment whose rows its stores overwrite
// (at most two: the stores cover at most 256 consecutive rows), and stores
// the rows at their destinations.  So that a tile costs about one memory
// round trip, a block asks for its next ticket as soon as it has the current
// one, reads the flags it waits for together with the rows, and loads the
// next entry before its stores go out.  (Tickets of several entries would
// either put consecutive tiles of a segment in one block, one after the
// other, or make a tile wait for a later ticket, which only a launch whose
// blocks are all resident could allow.)
//
// Why the order is right: a destination never exceeds its source, so the
// stores of a tile reach only rows below the tile's end: rows of the tile
// itself (all loaded before the block's barrier) or of earlier tiles of the
// same segment (loaded before their flags were set).  No block reads a row
// another block of the launch writes, so the flags order loads before stores
// and carry no data; they need no acquire or release.  Why every wait ends: a
// block sets its entry's flag before it waits for anything, and the entries it
// waits for were taken from the ticket counter before its own, by blocks that
// are running or done.  A bounded spin still turns a wait that would not end
// into LETHE_DEV_WAIT_TIMEOUT instead of a hang.
//
// compact_len_kernel sets the new lengths and resets the queue counters for
// the next call.
#include "device_common.h"
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
// waits.  A block past it waits no more.
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
  r.wnear = p->wnear;
  r.wfar = p->wfar;
  r.pad = 0;
#pragma unroll
  for (int x = 0; x < 4; ++x) r.kept[x] = p->kept[x];
  return r;
}

__global__ __launch_bounds__(kPlanThreads) void compact_plan_kernel(CompactArgs a) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const long long nseg = (long long)a.L * a.B * a.HK;
  const long long cidx = (long long)blockIdx.x * kPlanWaves + w;  // this wave's segment
  __shared__ int s_m[kPlanWaves];
  __shared__ int s_base;

  // The wave's segment: its length, first evicted row and moved tiles.
  bool valid = false;
  int n = 0, first = 0, ft = 0, nt = 0;
  long long row0 = 0;
  if (cidx < nseg) {
    const int h = (int)(cidx % a.HK);
    const int b = (int)((cidx / a.HK) % a.B);
    const int l = (int)(cidx / ((long long)a.HK * a.B));
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
  // One queue append for the block's segments.
  if (lane == 0) s_m[w] = nt - ft;
  __syncthreads();
  if (tid == 0) {
    int total = 0;
    for (int x = 0; x < kPlanWaves; ++x) total += s_m[x];
    int pos = 0;
    if (total > 0) {
      pos = atomicAdd(a.qlen, total);
      // Only segments that overlap other sequences' rows can overfill the queue.
      if (pos > a.qcap - total) pos = -1;
    }
    s_base = pos;
  }
  __syncthreads();
  if (!valid) return;
  if (first >= n) {
    if (lane == 0) a.counts[cidx] = n;
    return;
  }
  if (s_base < 0) {
    if (lane == 0) {
      a.counts[cidx] = -1;
      atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    }
    return;
  }
  int pos0 = s_base;
  for (int x = 0; x < w; ++x) pos0 += s_m[x];

  // Tiles ft .. nt-1, four per round: kept mask, kept count, destination of
  // the first kept row, and the earlier tiles the stores overwrite.
  int running = ft * kTile;  // rows kept before tile ft: all of them
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
      if (lane == 0) {
        const int j0 = t * kTile;
        CompactItem it;
        it.row0 = row0;
        it.j0 = j0;
        it.end = min(j0 + kTile, n);
        it.base = running;
        // Destinations running + [0, kc) lie in the source ranges of tiles
        // lo .. hi; those before tile ft never move and are never overwritten.
        const int lo = max(ft, running / kTile);
        const int hi = min(t - 1, (running + kc - 1) / kTile);
        const bool wait = kc > 0 && lo <= hi;
        it.wnear = wait ? t - hi : 0;
        it.wfar = wait ? t - lo : 0;
        it.pad = 0;
#pragma unroll
        for (int x = 0; x < 4; ++x) it.kept[x] = km[x];
        a.items[pos0 + t - ft] = it;
        a.flags[pos0 + t - ft] = 0;
      }
      running += kc;
    }
  }
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
  const int total = min(*a.qlen, a.qcap);
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

    int cw[kTileWaves];
    int cnt = 0;
#pragma unroll
    for (int x = 0; x < kTileWaves; ++x) {
      cw[x] = __popcll(it.kept[x]);
      cnt += cw[x];
    }
    if (tid < kTile) {
      unsigned long long m = it.kept[0];  // the wave's word, without indexing by w
#pragma unroll
      for (int x = 1; x < kTileWaves; ++x) m = w == x ? it.kept[x] : m;
      if ((m >> lane) & 1ull) {
        int before = __popcll(m & ((1ull << lane) - 1ull));
#pragma unroll
        for (int x = 0; x < kTileWaves; ++x) before += x < w ? cw[x] : 0;
        s_src[before] = it.j0 + tid;
      }
    }
    __syncthreads();
    // Rows whose destination is their source (before the first evicted row
    // of the segment's first moved tile) are left alone.
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
          rk[p] = *reinterpret_cast<const u32x4_t*>(K + (long long)src * RB + sub * 16);
          rv[p] = *reinterpret_cast<const u32x4_t*>(V + (long long)src * RB + sub * 16);
          rs[p] = sub == 0 ? S[src] : 0.0f;
        }
      }
    }
    // First look at the flags this tile waits for, in flight with the rows.
    int fnear = 1, ffar = 1;
    if (tid == 0 && it.wnear > 0) {
      fnear = __hip_atomic_load(&a.flags[t - it.wnear], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      ffar = __hip_atomic_load(&a.flags[t - it.wfar], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(0);
    if (tid == 0) s_t = tnext;
    __syncthreads();  // every load of the tile has completed
    if (tid == 0) {
      __hip_atomic_store(&a.flags[t], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (fnear == 0 || ffar == 0) {
        for (int k = it.wnear; k <= it.wfar && spins <= kSpinLimit; ++k) {
          while (__hip_atomic_load(&a.flags[t - k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
            if (++spins > kSpinLimit) {
              atomicOr(a.dev_status, LETHE_DEV_WAIT_TIMEOUT);
              break;
            }
            __builtin_amdgcn_s_sleep(2);
          }
        }
      }
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
        *reinterpret_cast<u32x4_t*>(K + dst * RB + sub * 16) = rk[p];
        *reinterpret_cast<u32x4_t*>(V + dst * RB + sub * 16) = rv[p];
        if (sub == 0) S[dst] = rs[p];
      }
    }
    t = tn;
    it = itn;
  }
}

// New length of every (layer, sequence): the kept count, equal across heads.
// Also returns the queue counters to zero for the next call.
__global__ void compact_len_kernel(CompactArgs a) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) {
    *a.qlen = 0;
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
  a.len[i] = mn;
}

int move_blocks() {
  // Persistent grid: two resident blocks per CU (the 256-byte-row kernel
  // holds 127 VGPRs, four waves per SIMD).
  static const int n = [] {
    const char* e = getenv("LETHE_COMPACT_BLOCKS");
    const int v = e ? atoi(e) : 0;
    return v > 0 ? v : 512;
  }();
  return n;
}

}  // namespace

lethe_status launch_compact(const CompactArgs& a, hipStream_t s) {
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
