// RASR retention mask by radix selection, gfx950.
//
// One block per (layer, sequence, KV head) segment.  The fp32 scores are mapped
// to 32-bit keys whose unsigned order is the float order (+0 and -0 equal, NaN
// below every number).  An MSB-first radix select with 8-bit digits and a
// 256-bin LDS histogram finds the exact key T of the m-th best candidate and
// how many candidates equal to T are still needed; a final ordered pass keeps
// every candidate above T and the lowest-indexed ones equal to T.
#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 256;

__device__ inline uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;  // NaN ranks last
  if (u == 0x80000000u) u = 0u;                      // -0 ties with +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__global__ __launch_bounds__(kThreads) void select_kernel(SelectArgs a) {
  const int h = blockIdx.x % a.HK;
  const int b = (blockIdx.x / a.HK) % a.B;
  const int l = blockIdx.x / (a.HK * a.B);
  const int tid = threadIdx.x;
  const int n = a.len[(long long)l * a.B + b];
  const int c = a.cap[b];
  const long long base = a.seq_base[b];
  if (n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer) {
    if (tid == 0) atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    return;
  }
  const long long row0 = (long long)l * a.rows_per_layer + base + (long long)h * c;
  const float* s = a.score + row0;
  uint8_t* keep = a.keep + row0;
  int k = a.budget[(long long)b * a.L + l];
  if (k < 0) k = 0;
  if (k >= n) {
    for (int j = tid; j < n; j += kThreads) keep[j] = 1;
    return;
  }
  const int r = min(a.recent, k);
  const int sk = min(a.sink, k - r);
  const int m = k - r - sk;
  const int lo = sk, hi = n - r;

  __shared__ uint32_t hist[256];
  __shared__ uint32_t suffix[257];
  __shared__ uint32_t s_digit, s_need;
  __shared__ long long scan_tmp[kThreads / kWave + 1];

  uint32_t prefix = 0, pmask = 0, need = (uint32_t)m;
  if (m > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0;
      __syncthreads();
      for (int j = lo + tid; j < hi; j += kThreads) {
        uint32_t key = order_key(s[j]);
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      // suffix[d] = number of matching candidates whose digit is >= d.
      if (tid == 0) {
        uint32_t acc = 0;
        suffix[256] = 0;
        for (int d = 255; d >= 0; --d) {
          acc += hist[d];
          suffix[d] = acc;
        }
      }
      __syncthreads();
      if (suffix[tid] >= need && suffix[tid + 1] < need) {
        s_digit = (uint32_t)tid;
        s_need = need - suffix[tid + 1];
      }
      __syncthreads();
      prefix |= s_digit << shift;
      pmask |= 255u << shift;
      need = s_need;
      __syncthreads();
    }
  }
  const uint32_t T = prefix;
  // Ordered pass: ties with key T are taken by increasing row index.
  long long carry = 0;
  for (int j0 = 0; j0 < n; j0 += kThreads) {
    const int j = j0 + tid;
    bool cand = j >= lo && j < hi && j < n;
    uint32_t key = cand ? order_key(s[j]) : 0u;
    bool eq = cand && m > 0 && key == T;
    long long total;
    long long rank = block_excl_scan<kThreads>(eq ? 1 : 0, scan_tmp, &total);
    if (j < n) {
      bool kp = !cand || (m > 0 && (key > T || (eq && carry + rank < (long long)need)));
      keep[j] = kp ? 1 : 0;
    }
    carry += total;
  }
}

}  // namespace

lethe_status launch_select(const SelectArgs& a, hipStream_t s) {
  long long nb = (long long)a.L * a.B * a.HK;
  if (nb > 0x7fffffffLL) return LETHE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)nb), dim3(kThreads), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

}  // namespace lethe
