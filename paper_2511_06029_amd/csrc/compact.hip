// In-place, order-preserving compaction of K, V and score rows, gfx950.
//
// One block per (layer, sequence, KV head) segment.  Rows before the first
// evicted row (found with 16 independent flag loads per thread) stay where
// they are.  From there the block sweeps the source rows in tiles of 256:
// four wavefronts ballot the keep flags of the tile and list
// the kept rows' source indices in LDS; every thread loads its share of those
// rows (16 bytes per lane) into registers, waits for its loads, the block
// synchronises, and the rows are stored to their destinations (a running
// prefix count).  A destination never exceeds its source, and the stores of a
// tile only reach rows below the tile's end, so no tile overwrites a row that
// a later tile still has to read; within a tile, every load has completed
// before the barrier that precedes the stores.  The next tile's keep flags
// are read before the current tile's stores go out.
#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 512;
constexpr int kTile = 256;
constexpr int kTileWaves = kTile / kWave;
// 16 bytes of a row; a vector type, so arrays of them stay in registers.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

template <int RB>  // row bytes of K (= of V)
__global__ __launch_bounds__(kThreads) void compact_kernel(CompactArgs a) {
  constexpr int TPR = RB / 16;              // threads per row
  constexpr int RPP = kThreads / TPR;       // rows per pass
  constexpr int PASSES = kTile / RPP;
  static_assert(kTile % RPP == 0, "tile");
  const int h = blockIdx.x % a.HK;
  const int b = (blockIdx.x / a.HK) % a.B;
  const int l = blockIdx.x / (a.HK * a.B);
  const int tid = threadIdx.x;
  const long long cidx = ((long long)l * a.B + b) * a.HK + h;
  const int n = a.len[(long long)l * a.B + b];
  const int c = a.cap[b];
  const long long base = a.seq_base[b];
  if (n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer) {
    if (tid == 0) {
      a.counts[cidx] = -1;
      atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    }
    return;
  }
  const long long row0 = (long long)l * a.rows_per_layer + base + (long long)h * c;
  const uint8_t* keep = a.keep + row0;
  char* K = reinterpret_cast<char*>(a.k) + row0 * RB;
  char* V = reinterpret_cast<char*>(a.v) + row0 * RB;
  float* S = a.score + row0;

  // First evicted row.
  __shared__ int s_first;
  __shared__ int s_src[kTile];          // per ballot wave: its kept rows in order
  __shared__ int s_cnt[kTileWaves];
  // 16 independent flag loads per thread and round; the lowest evicted row
  // of the round wins.
  if (tid == 0) s_first = n;
  __syncthreads();
  int first = n;
  for (int c0 = 0; c0 < n; c0 += 16 * kThreads) {
    // Clamped, unconditional loads, all issued before the first is used.
    uint8_t kv[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) kv[k] = keep[min(c0 + k * kThreads + tid, n - 1)];
    int f = n;
#pragma unroll
    for (int k = 15; k >= 0; --k) {
      const int j = c0 + k * kThreads + tid;
      if (j < n && kv[k] == 0) f = j;
    }
    if (f < n) atomicMin(&s_first, f);
    __syncthreads();
    first = s_first;
    __syncthreads();  // every thread has read s_first before it can change again
    if (first < n) break;
  }
  int pos = first;  // next destination row
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int sub = tid % TPR;
  bool kp_next = tid < kTile && first + tid < n && keep[first + tid] != 0;
  for (int j0 = first; j0 < n; j0 += kTile) {
    if (tid < kTile) {
      const bool kp = kp_next;
      const unsigned long long mask = __ballot(kp);
      const int before = __popcll(mask & ((1ull << lane) - 1ull));
      if (kp) s_src[kWave * w + before] = j0 + tid;
      if (lane == 0) s_cnt[w] = __popcll(mask);
    }
    __syncthreads();
    int cw[kTileWaves];
    int cnt = 0;
#pragma unroll
    for (int x = 0; x < kTileWaves; ++x) {
      cw[x] = s_cnt[x];
      cnt += cw[x];
    }
    u32x4_t rk[PASSES], rv[PASSES];
    float rs[PASSES];
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int i = p * RPP + tid / TPR;
      if (i < cnt) {
        int x = 0, off = i;
#pragma unroll
        for (int y = 0; y + 1 < kTileWaves; ++y)
          if (x == y && off >= cw[y]) {
            off -= cw[y];
            x = y + 1;
          }
        const long long src = s_src[kWave * x + off];
        rk[p] = *reinterpret_cast<const u32x4_t*>(K + src * RB + sub * 16);
        rv[p] = *reinterpret_cast<const u32x4_t*>(V + src * RB + sub * 16);
        rs[p] = sub == 0 ? S[src] : 0.0f;
      }
    }
    // The next tile's keep flags (a separate array: no ordering with the rows).
    const int jn = j0 + kTile + tid;
    kp_next = tid < kTile && jn < n && keep[jn] != 0;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // every load of the tile has completed; s_src may be reused
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int i = p * RPP + tid / TPR;
      if (i < cnt) {
        const long long dst = pos + i;
        *reinterpret_cast<u32x4_t*>(K + dst * RB + sub * 16) = rk[p];
        *reinterpret_cast<u32x4_t*>(V + dst * RB + sub * 16) = rv[p];
        if (sub == 0) S[dst] = rs[p];
      }
    }
    pos += cnt;
  }
  if (tid == 0) a.counts[cidx] = pos;
}

// New length of every (layer, sequence): the kept count, equal across heads.
__global__ void compact_len_kernel(CompactArgs a) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
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

}  // namespace

lethe_status launch_compact(const CompactArgs& a, hipStream_t s) {
  long long nb = (long long)a.L * a.B * a.HK;
  if (nb > 0x7fffffffLL) return LETHE_ERR_UNSUPPORTED;
  switch (a.row_bytes) {
    case 128: hipLaunchKernelGGL(compact_kernel<128>, dim3((unsigned)nb), dim3(kThreads), 0, s, a); break;
    case 256: hipLaunchKernelGGL(compact_kernel<256>, dim3((unsigned)nb), dim3(kThreads), 0, s, a); break;
    case 512: hipLaunchKernelGGL(compact_kernel<512>, dim3((unsigned)nb), dim3(kThreads), 0, s, a); break;
    default: return LETHE_ERR_UNSUPPORTED;
  }
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  long long nl = (long long)a.L * a.B;
  hipLaunchKernelGGL(compact_len_kernel, dim3((unsigned)((nl + 255) / 256)), dim3(256), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

}  // namespace lethe
