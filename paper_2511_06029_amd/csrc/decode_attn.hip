// Decode attention fused with the RASR importance update (Eq. 5), gfx950.
//
// One call handles one layer for all sequences.  Work is split into chunks of
// C consecutive rows of one (sequence, KV head) segment (split-K flash
// decoding), C chosen on the device from the live lengths so that about
// `nblocks` chunks exist; no length ever travels to the host.
//
// Kernel 1 (attn_chunks), one block per chunk:
//   - streams the chunk's K and V rows once with 16-byte loads, 16 lanes per
//     bf16 row of 128 (8 elements per lane), 4 rows per wavefront load;
//   - every query head g of the KV group: x_j = (scale*log2 e) q_g . k_j,
//     reduced across the lanes of a row with DPP;
//   - online softmax in base 2 per lane: running max m, sum l, output o;
//   - writes x_j (the scaled logits) to the pending buffer, and the chunk's
//     (m, l, o) to the partial buffer;
//   - the block owning the appended row reads it from k_new / v_new and also
//     writes it into the cache.
// Kernel 2 (finalize), one block per chunk:
//   - global (M, L) per head from the segment's partials;
//   - s_j <- gamma s_j + sum_g exp2(x_gj - M_g) / L_g for the chunk's rows;
//   - the chunk-0 block combines the partial outputs into out;
//   - block 0 publishes the new lengths and fills skipped / empty outputs.
#include <math.h>

#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 256;
constexpr int kNumWaves = kThreads / kWave;
constexpr int kFlagOverflow = 1;
constexpr int kFlagBad = 4;
constexpr int kFlagAppended = 16;

struct PlanLds {
  int n_att[kMaxSeqs];
  int nch[kMaxSeqs];
  int base[kMaxSeqs + 1];
  int flag[kMaxSeqs];
  long long tmp[kNumWaves + 1];
  int C;
  int chunks;
};

// Every block computes the same plan from len, cap and seq_base.
__device__ void compute_plan(const DecodeArgs& a, PlanLds& P) {
  const int tid = threadIdx.x;
  const bool app = a.k_new != nullptr;
  long long my_rows = 0;
  for (int b = tid; b < a.B; b += kThreads) {
    int n = a.len[b];
    int c = a.cap[b];
    long long base = a.seq_base[b];
    bool bad = n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer;
    bool ovf = !bad && app && n >= c;
    int f = (bad ? kFlagBad : 0) | (ovf ? kFlagOverflow : 0) | ((app && !bad && !ovf) ? kFlagAppended : 0);
    int na = (bad || ovf) ? 0 : n + (app ? 1 : 0);
    P.n_att[b] = na;
    P.flag[b] = f;
  }
  __syncthreads();
  // Total rows over all segments; every thread sums a strided subset.
  for (int b = tid; b < a.B; b += kThreads) my_rows += (long long)a.HK * P.n_att[b];
  long long total_rows;
  block_excl_scan<kThreads>(my_rows, P.tmp, &total_rows);
  long long per = (total_rows + a.nblocks - 1) / a.nblocks;
  long long C = ((per + 63) / 64) * 64;
  if (C < 64) C = 64;
  // Chunk counts and their prefix over sequences (each thread owns a
  // contiguous run of sequences so the prefix is a plain scan).
  const int per_t = (a.B + kThreads - 1) / kThreads;
  const int b0 = tid * per_t;
  long long local = 0;
  for (int i = 0; i < per_t; ++i) {
    int b = b0 + i;
    if (b < a.B) {
      int nc = (int)((P.n_att[b] + C - 1) / C);
      P.nch[b] = nc;
      local += (long long)a.HK * nc;
    }
  }
  long long total_chunks;
  long long ex = block_excl_scan<kThreads>(local, P.tmp, &total_chunks);
  for (int i = 0; i < per_t; ++i) {
    int b = b0 + i;
    if (b < a.B) {
      P.base[b] = (int)ex;
      ex += (long long)a.HK * P.nch[b];
    }
  }
  if (tid == 0) {
    P.base[a.B] = (int)total_chunks;
    P.C = (int)C;
    P.chunks = (int)total_chunks;
  }
  __syncthreads();
}

// Largest b with base[b] <= ci (base is non-decreasing, base[0] = 0).
__device__ inline int find_seq(const int* base, int B, int ci) {
  int lo = 0, hi = B;  // invariant: base[lo] <= ci < base[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (base[mid] <= ci) lo = mid;
    else hi = mid;
  }
  return lo;
}

template <typename T, int D, int G>
struct AttnCfg {
  static constexpr int EPL = Elem<T>::kPer16B;   // elements per lane per load
  static constexpr int LPR = D / EPL;            // lanes per row
  static constexpr int RPW = kWave / LPR;        // rows per wavefront load
  static constexpr int U = 4;                    // wavefront loads in flight
  static constexpr int ROWS_WAVE = U * RPW;
  static constexpr int ROWS_BLOCK = ROWS_WAVE * kNumWaves;
  static_assert(LPR >= 8 && LPR <= 32, "row split");
  static_assert(G <= LPR, "one pending-writer lane per head");
};

struct CombineLds {
  float m[kNumWaves][8];
  float l[kNumWaves][8];
  float o[kNumWaves][8][128];
};

union AttnLds {
  PlanLds plan;
  CombineLds comb;
};

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void attn_chunks_kernel(DecodeArgs a) {
  using Cfg = AttnCfg<T, D, G>;
  constexpr int EPL = Cfg::EPL, LPR = Cfg::LPR, RPW = Cfg::RPW, U = Cfg::U;
  __shared__ AttnLds lds;
  __shared__ int s_b, s_h, s_r0, s_r1, s_ncache, s_app, s_ci;

  compute_plan(a, lds.plan);
  const int tid = threadIdx.x;
  const int ci = blockIdx.x;
  if (blockIdx.x == 0) {
    // Publish the plan for the finalize kernel, and the device flags.
    int* pl = a.plan;
    int fl = 0;
    for (int b = tid; b < a.B; b += kThreads) {
      pl[kPlanHdr + b] = lds.plan.n_att[b];
      pl[kPlanHdr + kMaxSeqs + b] = lds.plan.nch[b];
      pl[kPlanHdr + 2 * kMaxSeqs + b] = lds.plan.base[b];
      pl[kPlanHdr + 3 * kMaxSeqs + 1 + b] = lds.plan.flag[b];
      fl |= lds.plan.flag[b] & (kFlagOverflow | kFlagBad);
    }
    if (tid == 0) {
      pl[kPlanC] = lds.plan.C;
      pl[kPlanChunks] = lds.plan.chunks;
      pl[kPlanHdr + 2 * kMaxSeqs + a.B] = lds.plan.base[a.B];
    }
    atomic_or_status(a.dev_status, fl);
  }
  if (ci >= lds.plan.chunks) return;  // uniform across the block
  if (tid == 0) {
    int b = find_seq(lds.plan.base, a.B, ci);
    int nc = lds.plan.nch[b];
    int rel = ci - lds.plan.base[b];
    int h = rel / nc;
    int c = rel % nc;
    int na = lds.plan.n_att[b];
    s_b = b;
    s_h = h;
    s_r0 = c * lds.plan.C;
    s_r1 = min(s_r0 + lds.plan.C, na);
    s_app = (lds.plan.flag[b] & kFlagAppended) ? 1 : 0;
    s_ncache = na - s_app;
    s_ci = ci;
  }
  __syncthreads();
  const int b = s_b, h = s_h, r0 = s_r0, r1 = s_r1, ncache = s_ncache;
  const bool app = s_app != 0;
  const int HQ = a.HK * G;
  const long long segrow0 = a.seq_base[b] + (long long)h * a.cap[b];

  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int rg = lane / LPR;  // row within a wavefront load
  const int dp = lane % LPR;  // element slice of the row

  // Query slice, pre-scaled by scale * log2(e).
  float qf[G][EPL];
  {
    const T* qb = reinterpret_cast<const T*>(a.q) + ((long long)b * HQ + (long long)h * G) * D;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      uint4 r = *reinterpret_cast<const uint4*>(qb + (long long)g * D + dp * EPL);
      Elem<T>::unpack(r, qf[g]);
#pragma unroll
      for (int e = 0; e < EPL; ++e) qf[g][e] *= a.scale_log2;
    }
  }

  float m[G], l[G], o[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[g][e] = 0.0f;
  }

  const T* Kb = reinterpret_cast<const T*>(a.k) + segrow0 * D + dp * EPL;
  const T* Vb = reinterpret_cast<const T*>(a.v) + segrow0 * D + dp * EPL;
  float* pend = a.pend + segrow0 * G;

  // Online-softmax update with U rows whose K/V slices are in kr/vr.
  auto consume = [&](const uint4* kr, const uint4* vr, const int* row, const bool* valid) {
    float x[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[EPL];
      Elem<T>::unpack(kr[u], kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float acc = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc = fmaf(qf[g][e], kf[e], acc);
        x[u][g] = group_sum<LPR>(acc);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (valid[u]) {
        float mine = x[u][0];
#pragma unroll
        for (int g = 1; g < G; ++g) mine = (dp == g) ? x[u][g] : mine;
        if (dp < G) pend[(long long)row[u] * G + dp] = mine;
      } else {
#pragma unroll
        for (int g = 0; g < G; ++g) x[u][g] = -INFINITY;
      }
    }
    float vf[U][EPL];
#pragma unroll
    for (int u = 0; u < U; ++u) Elem<T>::unpack(vr[u], vf[u]);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = m[g];
#pragma unroll
      for (int u = 0; u < U; ++u) mx = fmaxf(mx, x[u][g]);
      if (mx == -INFINITY) continue;
      float corr = exp2f(m[g] - mx);
      float lg = l[g] * corr;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] *= corr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float p = exp2f(x[u][g] - mx);
        lg += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] = fmaf(p, vf[u][e], o[g][e]);
      }
      l[g] = lg;
      m[g] = mx;
    }
  };

  // Cached rows [r0, re).
  const int re = min(r1, ncache);
  for (int base = r0 + w * Cfg::ROWS_WAVE; base < re; base += Cfg::ROWS_BLOCK) {
    uint4 kr[U], vr[U];
    int row[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      row[u] = base + u * RPW + rg;
      valid[u] = row[u] < re;
      int rr = valid[u] ? row[u] : (re - 1);
      kr[u] = *reinterpret_cast<const uint4*>(Kb + (long long)rr * D);
      vr[u] = *reinterpret_cast<const uint4*>(Vb + (long long)rr * D);
    }
    consume(kr, vr, row, valid);
  }
  // The appended row (only in the last chunk of its segment), by wave 0.
  if (app && r1 == ncache + 1 && w == 0) {
    const long long nb = ((long long)b * a.HK + h) * D + dp * EPL;
    uint4 kr[U], vr[U];
    int row[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      row[u] = ncache;
      valid[u] = (u == 0) && (rg == 0);
      kr[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.k_new) + nb);
      vr[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.v_new) + nb);
    }
    if (rg == 0) {
      *reinterpret_cast<uint4*>(reinterpret_cast<T*>(a.k_w) + (segrow0 + ncache) * D + dp * EPL) = kr[0];
      *reinterpret_cast<uint4*>(reinterpret_cast<T*>(a.v_w) + (segrow0 + ncache) * D + dp * EPL) = vr[0];
    }
    consume(kr, vr, row, valid);
  }

  // Combine the row groups of the wavefront (lanes with equal dp).
#pragma unroll
  for (int off = LPR; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mo = __shfl_xor(m[g], off);
      float lo = __shfl_xor(l[g], off);
      float mx = fmaxf(m[g], mo);
      float fa = (m[g] == -INFINITY) ? 0.0f : exp2f(m[g] - mx);
      float fb = (mo == -INFINITY) ? 0.0f : exp2f(mo - mx);
      l[g] = l[g] * fa + lo * fb;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        float oo = __shfl_xor(o[g][e], off);
        o[g][e] = o[g][e] * fa + oo * fb;
      }
      m[g] = mx;
    }
  }
  __syncthreads();  // plan LDS is dead from here on; reuse it for the combine
  CombineLds& cb = lds.comb;
  if (rg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) cb.o[w][g][dp * EPL + e] = o[g][e];
      if (dp == 0) {
        cb.m[w][g] = m[g];
        cb.l[w][g] = l[g];
      }
    }
  }
  __syncthreads();
  float* part = a.part + (long long)s_ci * G * (D + 2);
  for (int t = tid; t < G * D; t += kThreads) {
    int g = t / D, d = t % D;
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < kNumWaves; ++i) mx = fmaxf(mx, cb.m[i][g]);
    float lsum = 0.0f, osum = 0.0f;
#pragma unroll
    for (int i = 0; i < kNumWaves; ++i) {
      float f = (cb.m[i][g] == -INFINITY) ? 0.0f : exp2f(cb.m[i][g] - mx);
      lsum += cb.l[i][g] * f;
      osum += cb.o[i][g][d] * f;
    }
    part[g * (D + 2) + 2 + d] = osum;
    if (d == 0) {
      part[g * (D + 2)] = mx;
      part[g * (D + 2) + 1] = lsum;
    }
  }
}

struct FinLds {
  int n_att[kMaxSeqs];
  int nch[kMaxSeqs];
  int base[kMaxSeqs + 1];
  int flag[kMaxSeqs];
  float M[8];
  float invL[8];
};

template <int D, int G>
__global__ __launch_bounds__(kThreads) void finalize_kernel(DecodeArgs a) {
  __shared__ FinLds F;
  const int tid = threadIdx.x;
  const int* pl = a.plan;
  const int chunks = pl[kPlanChunks];
  const int C = pl[kPlanC];
  const int ci = blockIdx.x;
  const int HQ = a.HK * G;
  if (ci >= chunks && ci != 0) return;
  for (int b = tid; b < a.B; b += kThreads) {
    F.n_att[b] = pl[kPlanHdr + b];
    F.nch[b] = pl[kPlanHdr + kMaxSeqs + b];
    F.base[b] = pl[kPlanHdr + 2 * kMaxSeqs + b];
    F.flag[b] = pl[kPlanHdr + 3 * kMaxSeqs + 1 + b];
  }
  if (tid == 0) F.base[a.B] = pl[kPlanHdr + 2 * kMaxSeqs + a.B];
  __syncthreads();
  if (ci == 0) {
    // New lengths, and the outputs of sequences without chunks (empty: 0,
    // skipped: NaN).
    for (int b = tid; b < a.B; b += kThreads)
      if (F.flag[b] & kFlagAppended) a.len[b] = F.n_att[b];
    for (int b = 0; b < a.B; ++b) {
      if (F.n_att[b] != 0) continue;
      float fill = (F.flag[b] & (kFlagOverflow | kFlagBad)) ? __int_as_float(0x7fc00000) : 0.0f;
      float* ob = a.out + (long long)b * HQ * D;
      for (int t = tid; t < HQ * D; t += kThreads) ob[t] = fill;
    }
  }
  if (ci >= chunks) return;
  const int b = find_seq(F.base, a.B, ci);
  const int nc = F.nch[b];
  const int rel = ci - F.base[b];
  const int h = rel / nc;
  const int c = rel % nc;
  const int na = F.n_att[b];
  const bool app = (F.flag[b] & kFlagAppended) != 0;
  const int ncache = na - (app ? 1 : 0);
  const long long segrow0 = a.seq_base[b] + (long long)h * a.cap[b];
  const float* part0 = a.part + (long long)(F.base[b] + h * nc) * G * (D + 2);

  // Global softmax statistics of every head of the group.
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  for (int g = w; g < G; g += kNumWaves) {
    float mx = -INFINITY;
    for (int cc = lane; cc < nc; cc += kWave) mx = fmaxf(mx, part0[(long long)cc * G * (D + 2) + g * (D + 2)]);
    mx = wave_max(mx);
    float ls = 0.0f;
    for (int cc = lane; cc < nc; cc += kWave) {
      const float* p = part0 + (long long)cc * G * (D + 2) + g * (D + 2);
      float mc = p[0];
      ls += (mc == -INFINITY) ? 0.0f : p[1] * exp2f(mc - mx);
    }
    ls = wave_sum(ls);
    if (lane == 0) {
      F.M[g] = mx;
      F.invL[g] = 1.0f / ls;
    }
  }
  __syncthreads();

  // Score update of the chunk's rows.
  const int r0 = c * C, r1 = min(r0 + C, na);
  const float* pend = a.pend + segrow0 * G;
  float* score = a.score + segrow0;
  for (int r = r0 + tid; r < r1; r += kThreads) {
    float acc = 0.0f;
#pragma unroll
    for (int g = 0; g < G; ++g) acc += exp2f(pend[(long long)r * G + g] - F.M[g]) * F.invL[g];
    float s_old = (r < ncache) ? score[r] : 0.0f;
    score[r] = fmaf(a.gamma, s_old, acc);
  }

  // Output of the segment, by its first chunk's block.
  if (c == 0) {
    float* outb = a.out + ((long long)b * HQ + (long long)h * G) * D;
    for (int t = tid; t < G * D; t += kThreads) {
      int g = t / D, d = t % D;
      float acc = 0.0f;
      const float Mg = F.M[g];
      for (int cc = 0; cc < nc; ++cc) {
        const float* p = part0 + (long long)cc * G * (D + 2) + g * (D + 2);
        float mc = p[0];
        float f = (mc == -INFINITY) ? 0.0f : exp2f(mc - Mg);
        acc = fmaf(p[2 + d], f, acc);
      }
      outb[t] = acc * F.invL[g];
    }
  }
}

template <typename T, int D, int G>
lethe_status launch_tdg(const DecodeArgs& a, hipStream_t s) {
  int grid = a.nblocks + a.B * a.HK;
  hipLaunchKernelGGL((attn_chunks_kernel<T, D, G>), dim3(grid), dim3(kThreads), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  hipLaunchKernelGGL((finalize_kernel<D, G>), dim3(grid), dim3(kThreads), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  return LETHE_OK;
}

template <typename T, int D>
lethe_status launch_td(const DecodeArgs& a, int G, hipStream_t s) {
  switch (G) {
    case 1: return launch_tdg<T, D, 1>(a, s);
    case 2: return launch_tdg<T, D, 2>(a, s);
    case 3: return launch_tdg<T, D, 3>(a, s);
    case 4: return launch_tdg<T, D, 4>(a, s);
    case 5: return launch_tdg<T, D, 5>(a, s);
    case 6: return launch_tdg<T, D, 6>(a, s);
    case 7: return launch_tdg<T, D, 7>(a, s);
    case 8: return launch_tdg<T, D, 8>(a, s);
  }
  return LETHE_ERR_UNSUPPORTED;
}

}  // namespace

lethe_status launch_decode(const DecodeArgs& a_in, lethe_dtype dt, int D, int G, hipStream_t s) {
  DecodeArgs a = a_in;
  if (a.nblocks <= 0) a.nblocks = 2048;
  if (a.nblocks > kMaxDecodeBlocks) a.nblocks = kMaxDecodeBlocks;
  if (dt == LETHE_BF16) {
    if (D == 128) return launch_td<bf16_t, 128>(a, G, s);
    if (D == 64) return launch_td<bf16_t, 64>(a, G, s);
  } else {
    if (D == 128) return launch_td<float, 128>(a, G, s);
    if (D == 64) return launch_td<float, 64>(a, G, s);
  }
  return LETHE_ERR_UNSUPPORTED;
}

}  // namespace lethe
