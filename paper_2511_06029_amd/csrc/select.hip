// Retention masks by radix selection, gfx950.
//
// Three rules share one kernel template:
//  * RASR per segment: one block per (layer, sequence, KV head); the rank key
//    is that head's accumulated score.
//  * RASR shared by the heads of a layer: one block per (layer, sequence); the
//    key is the head-summed score (Eq. 2 collapses attention over heads), the
//    fp32 sum in ascending head order, and the mask goes to every head.
//  * Algorithm 1 (segmented token shrinking) with the size trigger: one block
//    per (layer, sequence) on the head-summed score.  The breakpoint needs no
//    sort: the head-to-cut ratio test holds on a suffix of the ranking (the
//    values never increase along it), so one max pass and one counting pass
//    give the first rank where it holds, and the breakpoint is the first cut
//    point at or after it.  The salient set is then the top-`breakpoint`
//    selection below.
//
// Selection: fp32 keys map to 32-bit words whose unsigned order is the float
// order (+0 and -0 equal, NaN below every number).  An MSB-first radix select
// with 8-bit digits and a 256-bin LDS histogram finds the exact key T of the
// m-th best candidate, how many candidates equal to T are still needed and
// how many there are.  When all of them are needed (the usual case) one
// elementwise pass keeps the candidates at or above T; otherwise an ordered
// pass keeps every candidate above T and the lowest-indexed ones equal to T.
// Candidate sets of up to kRegKeys rows per thread are read once into
// registers, and the radix passes and the elementwise pass use those; larger
// sets are re-read per pass, each thread issuing the loads of eight rows
// before it uses the first.
#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

__device__ inline uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;  // NaN ranks last
  if (u == 0x80000000u) u = 0u;                      // -0 ties with +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inverse of order_key on the keys of numbers (NaN's key 0 is never inverted).
__device__ inline float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Rank value of row j: one head's score, or the fp32 head sum (additions in
// ascending head order, each rounded; no multiply, so nothing contracts).
template <bool kShared>
struct Scores {
  const float* s;       // head 0's segment
  long long hstride;    // rows between the segments of consecutive heads
  int heads;
  __device__ inline float operator()(int j) const {
    if constexpr (!kShared) {
      return s[j];
    } else {
      float acc = s[j];
      for (int h = 1; h < heads; ++h) acc = acc + s[h * hstride + j];
      return acc;
    }
  }
  // The same for rows j[0 .. U) (valid indices): each head's loads of the U
  // rows are issued together, unconditionally.
  template <int U>
  __device__ inline void batch(const int* j, float* v) const {
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = s[j[u]];
    if constexpr (kShared) {
      for (int h = 1; h < heads; ++h) {
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) x[u] = s[h * hstride + j[u]];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = v[u] + x[u];
      }
    }
  }
};

template <int NT>
struct SelectShared {
  uint32_t hist[256];
  uint32_t suffix[257];
  uint32_t digit, need;
  uint32_t red_u[NT / kWave];
  uint32_t red_c[NT / kWave];
  long long scan_tmp[NT / kWave + 1];
  int plan[4];  // lo, hi, m, keep-all flag
};

// Rows a thread loads before it uses the first of them (the passes are bound
// by load latency).
constexpr int kU = 8;

// Key T of the m-th best key among rows [lo, hi) (m >= 1), how many rows
// with key T belong to the best m, and how many rows have key T.  All
// threads get the three.
template <int NT, class KeyFn>
__device__ void radix_select(const KeyFn& rank, int lo, int hi, uint32_t m, SelectShared<NT>& sh,
                             uint32_t* T_out, uint32_t* need_out, uint32_t* count_out) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0, pmask = 0, need = m, count = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) sh.hist[tid] = 0;
    __syncthreads();
    for (int j0 = lo; j0 < hi; j0 += kU * NT) {
      int jj[kU];
      float v[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) jj[u] = min(j0 + u * NT + tid, hi - 1);
      rank.template batch<kU>(jj, v);
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const uint32_t key = order_key(v[u]);
        if (j0 + u * NT + tid < hi && (key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255u], 1u);
      }
    }
    __syncthreads();
    // suffix[d] = matching keys whose digit is >= d: wave 0, four bins a lane.
    if (tid < kWave) {
      const uint32_t h0 = sh.hist[4 * tid], h1 = sh.hist[4 * tid + 1];
      const uint32_t h2 = sh.hist[4 * tid + 2], h3 = sh.hist[4 * tid + 3];
      const uint32_t tot = h0 + h1 + h2 + h3;
      uint32_t incl = tot;  // sum over lanes tid .. 63
      for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t v = __shfl_down(incl, o);
        if (tid + o < kWave) incl += v;
      }
      const uint32_t above = incl - tot;
      sh.suffix[4 * tid + 3] = above + h3;
      sh.suffix[4 * tid + 2] = above + h3 + h2;
      sh.suffix[4 * tid + 1] = above + h3 + h2 + h1;
      sh.suffix[4 * tid] = incl;
      if (tid == 0) sh.suffix[256] = 0;
    }
    __syncthreads();
    if (tid < 256 && sh.suffix[tid] >= need && sh.suffix[tid + 1] < need) {
      sh.digit = (uint32_t)tid;
      sh.need = need - sh.suffix[tid + 1];
    }
    __syncthreads();
    prefix |= sh.digit << shift;
    pmask |= 255u << shift;
    need = sh.need;
    count = sh.hist[sh.digit];
    __syncthreads();
  }
  *T_out = prefix;
  *need_out = need;
  *count_out = count;
}

// Keys a thread keeps in registers: candidate sets of up to kRegKeys * NT rows
// are read from memory once.
constexpr int kRegKeys = 32;

// radix_select over keys held in registers: thread t holds the keys of
// candidates t, t + NT, ... (key[u] for u < cnt; cnt is the same for all
// threads, slots past the candidates hold 0 and are not counted).
template <int NT>
__device__ void radix_select_regs(const uint32_t (&key)[kRegKeys], const bool (&valid)[kRegKeys], uint32_t m,
                                  SelectShared<NT>& sh, uint32_t* T_out, uint32_t* need_out, uint32_t* count_out) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0, pmask = 0, need = m, count = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) sh.hist[tid] = 0;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kRegKeys; ++u)
      if (valid[u] && (key[u] & pmask) == prefix) atomicAdd(&sh.hist[(key[u] >> shift) & 255u], 1u);
    __syncthreads();
    if (tid < kWave) {
      const uint32_t h0 = sh.hist[4 * tid], h1 = sh.hist[4 * tid + 1];
      const uint32_t h2 = sh.hist[4 * tid + 2], h3 = sh.hist[4 * tid + 3];
      const uint32_t tot = h0 + h1 + h2 + h3;
      uint32_t incl = tot;
      for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t v = __shfl_down(incl, o);
        if (tid + o < kWave) incl += v;
      }
      const uint32_t above = incl - tot;
      sh.suffix[4 * tid + 3] = above + h3;
      sh.suffix[4 * tid + 2] = above + h3 + h2;
      sh.suffix[4 * tid + 1] = above + h3 + h2 + h1;
      sh.suffix[4 * tid] = incl;
      if (tid == 0) sh.suffix[256] = 0;
    }
    __syncthreads();
    if (tid < 256 && sh.suffix[tid] >= need && sh.suffix[tid + 1] < need) {
      sh.digit = (uint32_t)tid;
      sh.need = need - sh.suffix[tid + 1];
    }
    __syncthreads();
    prefix |= sh.digit << shift;
    pmask |= 255u << shift;
    need = sh.need;
    count = sh.hist[sh.digit];
    __syncthreads();
  }
  *T_out = prefix;
  *need_out = need;
  *count_out = count;
}

// Block-wide max of a key and sum of a count; every thread gets both.
template <int NT>
__device__ void block_max_count(uint32_t key, uint32_t cnt, SelectShared<NT>& sh, uint32_t* kmax,
                                uint32_t* csum) {
  for (int o = kWave / 2; o > 0; o >>= 1) {
    key = max(key, (uint32_t)__shfl_xor(key, o));
    cnt += (uint32_t)__shfl_xor(cnt, o);
  }
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    sh.red_u[w] = key;
    sh.red_c[w] = cnt;
  }
  __syncthreads();
  uint32_t k = 0, c = 0;
  for (int i = 0; i < NT / kWave; ++i) {
    k = max(k, sh.red_u[i]);
    c += sh.red_c[i];
  }
  __syncthreads();
  *kmax = k;
  *csum = c;
}

template <int NT, int MODE>
__global__ __launch_bounds__(NT) void select_kernel(SelectArgs a) {
  constexpr bool kShared = MODE != kSelectRasr;
  constexpr bool kShrink = MODE == kSelectShrink;
  const int h = kShared ? 0 : (int)(blockIdx.x % a.HK);
  const int lb = kShared ? (int)blockIdx.x : (int)(blockIdx.x / a.HK);
  const int b = lb % a.B;
  const int l = lb / a.B;
  const int tid = threadIdx.x;
  const int n = a.len[(long long)l * a.B + b];
  const int c = a.cap[b];
  const long long base = a.seq_base[b];
  if (n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer) {
    if (tid == 0) atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    return;
  }
  const long long row0 = (long long)l * a.rows_per_layer + base + (long long)h * c;
  const Scores<kShared> rank{a.score + row0, (long long)c, a.HK};
  uint8_t* keep = a.keep + row0;
  const int nheads = kShared ? a.HK : 1;
  __shared__ SelectShared<NT> sh;

  // Plan: candidate rows [lo, hi), how many of them to keep (m), and the
  // forced rows, which are [0, fs) and [fr, n).
  int lo = 0, hi = 0, m = 0, fs = 0, fr = n;
  bool all = false;
  if constexpr (!kShrink) {
    int k = a.budget[(long long)b * a.L + l];
    if (k < 0) k = 0;
    if (k >= n) {
      all = true;
    } else {
      const int r = min(a.recent, k);
      const int sk = min(a.sink, k - r);
      m = k - r - sk;
      lo = sk;
      hi = n - r;
      fs = sk;
      fr = n - r;
    }
  } else {
    const long long lev0 = max(a.evict[(long long)l * a.B + b], 0);
    long long lev = lev0;
    long long bp = kShrinkNotTriggered;
    if (n <= lev0) {
      all = true;
    } else {
      // Head of the ranking and the NaN count.
      uint32_t kmax = 0, nnan = 0;
      {
        uint32_t km = 0, cn = 0;
        for (int j = tid; j < n; j += NT) {
          const float v = rank(j);
          km = max(km, order_key(v));
          cn += (v != v) ? 1u : 0u;
        }
        block_max_count<NT>(km, cn, sh, &kmax, &nnan);
      }
      bp = kShrinkNoBreakpoint;
      const float head = key_value(kmax);
      if (kmax != 0u && head > 0.0f && a.segments > 1) {
        // cnt = rows whose ratio head / value stays below tau (tau * value >
        // head, exact in fp64): ranks [cnt, n - nnan) pass the test.
        const double dh = (double)head, dt = (double)a.tau;
        uint32_t cn = 0, unused = 0;
        for (int j = tid; j < n; j += NT) {
          const float v = rank(j);
          cn += (v == v && dt * (double)v > dh) ? 1u : 0u;
        }
        uint32_t cnt = 0;
        block_max_count<NT>(0u, cn, sh, &unused, &cnt);
        const long long D = a.segments;
        long long d = ((long long)cnt * D + n - 1) / n;  // first d with n*d >= cnt*D
        if (d < 1) d = 1;
        if (d <= D - 1) {
          const long long cut = ((long long)n * d) / D;
          if (cut < (long long)n - (long long)nnan) bp = cut;
        }
      }
      if (bp >= 0) {
        m = (int)bp;
        lo = 0;
        hi = n;
        fs = min(a.sink, n);
        fr = n - min(a.recent, n);
        lev = max(lev0, bp + (long long)a.recent);
      } else {
        all = true;
        lev = 2 * lev0;
      }
      if (lev > 0x7fffffffLL) lev = 0x7fffffffLL;
    }
    if (tid == 0) {
      a.evict[(long long)l * a.B + b] = (int32_t)lev;
      if (a.breakpoint) a.breakpoint[(long long)l * a.B + b] = (int32_t)bp;
    }
  }

  if (all) {
    for (int hh = 0; hh < nheads; ++hh)
      for (int j = tid; j < n; j += NT) keep[(long long)hh * c + j] = 1;
    return;
  }
  uint32_t T = 0, need = 0, countT = 0;
  if (m > 0 && hi - lo <= kRegKeys * NT) {
    // The candidates' keys in registers, read once (eight rows' loads at a
    // time); the radix passes and the keep pass use them.
    uint32_t key[kRegKeys];
    bool valid[kRegKeys];
#pragma unroll
    for (int u0 = 0; u0 < kRegKeys; u0 += kU) {
      if (lo + u0 * NT < hi) {  // block-uniform
        int jj[kU];
        float v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) jj[u] = min(lo + (u0 + u) * NT + tid, hi - 1);
        rank.template batch<kU>(jj, v);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          valid[u0 + u] = lo + (u0 + u) * NT + tid < hi;
          key[u0 + u] = order_key(v[u]);
        }
      } else {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          valid[u0 + u] = false;
          key[u0 + u] = 0u;
        }
      }
    }
    radix_select_regs<NT>(key, valid, (uint32_t)m, sh, &T, &need, &countT);
    if (need == countT) {
      // Forced rows, then every candidate at or above T.
      for (int j = tid; j < fs; j += NT)
        for (int hh = 0; hh < nheads; ++hh) keep[(long long)hh * c + j] = 1;
      for (int j = max(fr, hi) + tid; j < n; j += NT)
        for (int hh = 0; hh < nheads; ++hh) keep[(long long)hh * c + j] = 1;
#pragma unroll
      for (int u = 0; u < kRegKeys; ++u) {
        const int j = lo + u * NT + tid;
        if (valid[u]) {
          const uint8_t kp = (j < fs || j >= fr || key[u] >= T) ? 1 : 0;
          for (int hh = 0; hh < nheads; ++hh) keep[(long long)hh * c + j] = kp;
        }
      }
      return;
    }
  } else if (m > 0) {
    radix_select<NT>(rank, lo, hi, (uint32_t)m, sh, &T, &need, &countT);
  }
  if (m == 0 || need == countT) {
    // Every candidate with key T is kept (or none is a candidate to keep):
    // no tie to break, so each row is decided on its own.
    for (int j0 = 0; j0 < n; j0 += kU * NT) {
      float v[kU];
      if (m > 0) {
        int jj[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) jj[u] = min(max(j0 + u * NT + tid, lo), hi - 1);
        rank.template batch<kU>(jj, v);
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int j = j0 + u * NT + tid;
        if (j < n) {
          const bool cand = m > 0 && j >= lo && j < hi;
          const uint8_t kp = (j < fs || j >= fr || (cand && order_key(v[u]) >= T)) ? 1 : 0;
          for (int hh = 0; hh < nheads; ++hh) keep[(long long)hh * c + j] = kp;
        }
      }
    }
    return;
  }
  // Ordered pass: ties with key T are taken by increasing row index.
  long long carry = 0;
  for (int j0 = 0; j0 < n; j0 += NT) {
    const int j = j0 + tid;
    const bool cand = j >= lo && j < hi && j < n;
    const uint32_t key = (cand && m > 0) ? order_key(rank(j)) : 0u;
    const bool eq = cand && m > 0 && key == T;
    long long total;
    const long long pos = block_excl_scan<NT>(eq ? 1 : 0, sh.scan_tmp, &total);
    if (j < n) {
      const bool forced = j < fs || j >= fr;
      const bool chosen = cand && m > 0 && (key > T || (eq && carry + pos < (long long)need));
      const uint8_t kp = (forced || chosen) ? 1 : 0;
      for (int hh = 0; hh < nheads; ++hh) keep[(long long)hh * c + j] = kp;
    }
    carry += total;
  }
}

}  // namespace

lethe_status launch_select(const SelectArgs& a, hipStream_t s) {
  const long long nb = (long long)a.L * a.B * (a.mode == kSelectRasr ? a.HK : 1);
  if (nb > 0x7fffffffLL) return LETHE_ERR_UNSUPPORTED;
  if (nb == 0) return LETHE_OK;
  switch (a.mode) {
    case kSelectRasr:
      hipLaunchKernelGGL((select_kernel<256, kSelectRasr>), dim3((unsigned)nb), dim3(256), 0, s, a);
      break;
    case kSelectRasrShared:
      hipLaunchKernelGGL((select_kernel<1024, kSelectRasrShared>), dim3((unsigned)nb), dim3(1024), 0, s, a);
      break;
    case kSelectShrink:
      hipLaunchKernelGGL((select_kernel<1024, kSelectShrink>), dim3((unsigned)nb), dim3(1024), 0, s, a);
      break;
    default:
      return LETHE_ERR_INVALID;
  }
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

}  // namespace lethe
