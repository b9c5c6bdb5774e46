// Layer sparsity (Eq. 1 on the head-summed importance of Eq. 2) and the
// integer budget split across layers, gfx950.
//
// hoyer_kernel: one block per (sequence b, layer l).  Streams the H_KV score
// vectors of the live rows once (4 bytes per row), forms a_j = sum_h s_h,j in
// fp64, and reduces |a|_1 and |a|_2^2 in fp64 (the score vectors of a layer can
// hold 10^5 rows of widely varying magnitude).  The loads of eight rows of up
// to four heads are issued together: the kernel is bound by load latency.
// budget_kernel: one wavefront per sequence runs the split, a lane per layer
// (up to four layers a lane for L <= 256).
#include <math.h>

#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void hoyer_kernel(SparsityArgs a) {
  const int b = blockIdx.x % a.B;
  const int l = blockIdx.x / a.B;
  const int tid = threadIdx.x;
  const int n = a.len[(long long)l * a.B + b];
  const int c = a.cap[b];
  const long long base = a.seq_base[b];
  const bool bad = n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer;
  if (bad) {
    if (tid == 0) {
      a.sparsity_out[(long long)b * a.L + l] = 0.0f;
      atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    }
    return;
  }
  const float* s0 = a.score + (long long)l * a.rows_per_layer + base;
  // Rows tid, tid + kThreads, ... in order; kU rows and up to four heads of
  // loads in flight per thread before the first use.
  constexpr int kU = 8;
  double l1 = 0.0, l2 = 0.0;
  for (int j0 = 0; j0 < n; j0 += kU * kThreads) {
    double aj[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) aj[u] = 0.0;
    for (int h0 = 0; h0 < a.HK; h0 += 4) {
      // Clamped, unconditional loads (a guarded load would be waited for
      // inside its own branch); the values past the ends are not used.
      float x[4][kU];
#pragma unroll
      for (int hh = 0; hh < 4; ++hh)
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int j = min(j0 + u * kThreads + tid, n - 1);
          x[hh][u] = s0[(long long)min(h0 + hh, a.HK - 1) * c + j];
        }
#pragma unroll
      for (int hh = 0; hh < 4; ++hh)
#pragma unroll
        for (int u = 0; u < kU; ++u)
          if (h0 + hh < a.HK) aj[u] += (double)x[hh][u];
    }
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (j0 + u * kThreads + tid < n) {
        l1 += fabs(aj[u]);
        l2 += aj[u] * aj[u];
      }
  }
  __shared__ double red[2][kThreads / kWave];
  l1 = wave_sum_d(l1);
  l2 = wave_sum_d(l2);
  const int lane = tid & (kWave - 1), w = tid / kWave;
  if (lane == 0) {
    red[0][w] = l1;
    red[1][w] = l2;
  }
  __syncthreads();
  if (tid == 0) {
    double L1 = 0.0, L2 = 0.0;
    for (int i = 0; i < kThreads / kWave; ++i) {
      L1 += red[0][i];
      L2 += red[1][i];
    }
    double S = 0.0;
    if (n > 1 && L2 > 0.0) {
      double rn = sqrt((double)n);
      S = (rn - L1 / sqrt(L2)) / (rn - 1.0);
      S = fmin(fmax(S, 0.0), 1.0);
    }
    a.sparsity_out[(long long)b * a.L + l] = (float)S;
  }
}

// Proportional integer split with floors and caps (see lethe.h).  One
// wavefront per sequence; lane x holds layers x, x + 64, ... (at most
// kMaxLayers / 64 per lane, unrolled into registers).  All quotas of a pass
// are taken against the same R and W, as the rule says; the leftover tokens
// go to the layers whose rank by (remainder desc, layer asc) is below the
// leftover count.
constexpr int kLpl = kMaxLayers / kWave;  // layers per lane

__device__ inline unsigned long long wave_sum_u64(unsigned long long v) {
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__global__ __launch_bounds__(kWave) void budget_kernel(SparsityArgs a) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int L = a.L;
  long long f[kLpl], cp[kLpl];
  unsigned long long w[kLpl], rem[kLpl];
  int out[kLpl];
  bool act[kLpl];
  long long sum_n = 0, sum_f = 0;
  const float* Sp = a.sparsity_in ? a.sparsity_in : a.sparsity_out;
#pragma unroll
  for (int k = 0; k < kLpl; ++k) {
    const int l = lane + kWave * k;
    f[k] = cp[k] = 0;
    w[k] = 0;
    rem[k] = 0;
    act[k] = false;
    out[k] = 0;
    if (l >= L) continue;
    long long nl = a.len[(long long)l * a.B + b];
    if (nl < 0) nl = 0;
    long long fl = (long long)a.recent + (long long)a.sink;
    if (fl > nl) fl = nl;
    f[k] = fl;
    cp[k] = nl;
    sum_n += nl;
    sum_f += fl;
    float S = Sp[(long long)b * L + l];
    if (a.sparsity_in) a.sparsity_out[(long long)b * L + l] = S;
    if (!(S >= 0.0f)) S = 0.0f;
    if (S > 1.0f) S = 1.0f;
    const float scaled = __fmul_rn(__fsub_rn(1.0f, S), 16777216.0f);
    w[k] = 1ull + (unsigned long long)(unsigned int)floorf(scaled);
  }
  sum_n = (long long)wave_sum_u64((unsigned long long)sum_n);
  sum_f = (long long)wave_sum_u64((unsigned long long)sum_f);
  int* outp = a.budget_out + (long long)b * L;
  const long long G = a.global_budget[b];
  if (sum_n <= G || sum_f > G) {
#pragma unroll
    for (int k = 0; k < kLpl; ++k)
      if (lane + kWave * k < L) outp[lane + kWave * k] = (int)cp[k];
    if (sum_n > G && lane == 0) atomicOr(a.dev_status, LETHE_DEV_INFEASIBLE);
    return;
  }
  unsigned long long R = (unsigned long long)(G - sum_f);
#pragma unroll
  for (int k = 0; k < kLpl; ++k) {
    act[k] = cp[k] > f[k];
    out[k] = (int)f[k];
  }
  for (;;) {
    unsigned long long wa = 0;
#pragma unroll
    for (int k = 0; k < kLpl; ++k) wa += act[k] ? w[k] : 0ull;
    const unsigned long long W = wave_sum_u64(wa);
    unsigned long long q[kLpl];
    bool capped_any = false;
    unsigned long long taken = 0;
#pragma unroll
    for (int k = 0; k < kLpl; ++k) {
      q[k] = act[k] ? (R * w[k]) / W : 0ull;
      const bool cap_k = act[k] && (unsigned long long)f[k] + q[k] >= (unsigned long long)cp[k];
      capped_any |= cap_k;
      if (cap_k) taken += (unsigned long long)(cp[k] - f[k]);
    }
    if (__any(capped_any)) {
      // Every layer that reaches its cap in this pass is fixed at once.
#pragma unroll
      for (int k = 0; k < kLpl; ++k) {
        if (act[k] && (unsigned long long)f[k] + q[k] >= (unsigned long long)cp[k]) {
          out[k] = (int)cp[k];
          act[k] = false;
        }
      }
      R -= wave_sum_u64(taken);
      continue;
    }
    unsigned long long given = 0;
#pragma unroll
    for (int k = 0; k < kLpl; ++k) {
      if (!act[k]) continue;
      rem[k] = (R * w[k]) % W;
      out[k] = (int)(f[k] + (long long)q[k]);
      given += q[k];
    }
    const unsigned long long left = R - wave_sum_u64(given);
    // Rank of each active layer among the active layers by (remainder desc,
    // layer asc); the first `left` of them get one more token.
    int rank[kLpl];
#pragma unroll
    for (int k = 0; k < kLpl; ++k) rank[k] = 0;
    for (int j = 0; j < L; ++j) {
      const int jl = j % kWave, jk = j / kWave;
      unsigned long long rj = 0;
      bool aj = false;
#pragma unroll
      for (int k = 0; k < kLpl; ++k) {
        if (k == jk) {
          rj = __shfl(rem[k], jl);
          aj = __shfl(act[k] ? 1 : 0, jl) != 0;
        }
      }
      if (!aj) continue;
#pragma unroll
      for (int k = 0; k < kLpl; ++k) {
        const int l = lane + kWave * k;
        if (act[k] && (rj > rem[k] || (rj == rem[k] && j < l))) ++rank[k];
      }
    }
#pragma unroll
    for (int k = 0; k < kLpl; ++k)
      if (act[k] && (unsigned long long)rank[k] < left) out[k] += 1;
    break;
  }
#pragma unroll
  for (int k = 0; k < kLpl; ++k)
    if (lane + kWave * k < L) outp[lane + kWave * k] = out[k];
}

}  // namespace

lethe_status launch_sparsity(const SparsityArgs& a, hipStream_t s) {
  if (!a.sparsity_in) {
    hipLaunchKernelGGL(hoyer_kernel, dim3(a.B * a.L), dim3(kThreads), 0, s, a);
    if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  }
  hipLaunchKernelGGL(budget_kernel, dim3(a.B), dim3(kWave), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

}  // namespace lethe
