// Layer sparsity (Eq. 1 on the head-summed importance of Eq. 2) and the
// integer budget split across layers, gfx950.
//
// hoyer_kernel: one block per (sequence b, layer l).  Streams the H_KV score
// vectors of the live rows once (4 bytes per row), forms a_j = sum_h s_h,j in
// fp64, and reduces |a|_1 and |a|_2^2 in fp64 (the score vectors of a layer can
// hold 10^5 rows of widely varying magnitude).
// budget_kernel: one thread per sequence runs the split over <= 256 layers.
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
  double l1 = 0.0, l2 = 0.0;
  for (int j = tid; j < n; j += kThreads) {
    double aj = 0.0;
    for (int h = 0; h < a.HK; ++h) aj += (double)s0[(long long)h * c + j];
    l1 += fabs(aj);
    l2 += aj * aj;
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

// Proportional integer split with floors and caps (see lethe.h).
__global__ void budget_kernel(SparsityArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.B) return;
  const int L = a.L;
  long long f[kMaxLayers], cp[kMaxLayers];
  unsigned long long w[kMaxLayers], rem[kMaxLayers];
  unsigned char act[kMaxLayers], pick[kMaxLayers];
  long long sum_n = 0, sum_f = 0;
  int* out = a.budget_out + (long long)b * L;
  const float* Sp = a.sparsity_in ? a.sparsity_in : a.sparsity_out;
  for (int l = 0; l < L; ++l) {
    long long nl = a.len[(long long)l * a.B + b];
    if (nl < 0) nl = 0;
    long long fl = (long long)a.recent + (long long)a.sink;
    if (fl > nl) fl = nl;
    f[l] = fl;
    cp[l] = nl;
    sum_n += nl;
    sum_f += fl;
    float S = Sp[(long long)b * L + l];
    if (a.sparsity_in) a.sparsity_out[(long long)b * L + l] = S;
    if (!(S >= 0.0f)) S = 0.0f;
    if (S > 1.0f) S = 1.0f;
    float scaled = __fmul_rn(__fsub_rn(1.0f, S), 16777216.0f);
    w[l] = 1ull + (unsigned long long)(unsigned int)floorf(scaled);
  }
  const long long G = a.global_budget[b];
  if (sum_n <= G || sum_f > G) {
    for (int l = 0; l < L; ++l) out[l] = (int)cp[l];
    if (sum_n > G) atomicOr(a.dev_status, LETHE_DEV_INFEASIBLE);
    return;
  }
  unsigned long long R = (unsigned long long)(G - sum_f);
  for (int l = 0; l < L; ++l) {
    act[l] = cp[l] > f[l];
    out[l] = (int)f[l];
  }
  for (;;) {
    unsigned long long W = 0;
    for (int l = 0; l < L; ++l)
      if (act[l]) W += w[l];
    bool capped = false;
    for (int l = 0; l < L; ++l) {
      pick[l] = 0;
      if (!act[l]) continue;
      unsigned long long ql = (R * w[l]) / W;
      if ((unsigned long long)f[l] + ql >= (unsigned long long)cp[l]) pick[l] = 1, capped = true;
    }
    if (capped) {
      unsigned long long taken = 0;
      for (int l = 0; l < L; ++l) {
        if (!pick[l]) continue;
        out[l] = (int)cp[l];
        taken += (unsigned long long)(cp[l] - f[l]);
        act[l] = 0;
      }
      R -= taken;
      continue;
    }
    unsigned long long given = 0;
    for (int l = 0; l < L; ++l) {
      if (!act[l]) continue;
      unsigned long long ql = (R * w[l]) / W;
      rem[l] = (R * w[l]) % W;
      out[l] = (int)(f[l] + (long long)ql);
      given += ql;
      pick[l] = 0;
    }
    unsigned long long left = R - given;
    for (unsigned long long t = 0; t < left; ++t) {
      int best = -1;
      for (int l = 0; l < L; ++l) {
        if (!act[l] || pick[l]) continue;
        if (best < 0 || rem[l] > rem[best]) best = l;
      }
      pick[best] = 1;
      out[best] += 1;
    }
    break;
  }
}

}  // namespace

lethe_status launch_sparsity(const SparsityArgs& a, hipStream_t s) {
  if (!a.sparsity_in) {
    hipLaunchKernelGGL(hoyer_kernel, dim3(a.B * a.L), dim3(kThreads), 0, s, a);
    if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  }
  const int t = 64;
  hipLaunchKernelGGL(budget_kernel, dim3((a.B + t - 1) / t), dim3(t), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

}  // namespace lethe
