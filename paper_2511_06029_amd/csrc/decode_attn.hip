// Decode attention fused with the RASR importance update (Eq. 5), gfx950.
//
// One call handles one layer for all sequences, in two kernels.
//
// The live rows of every (sequence, KV head) segment are cut into chunks of C
// consecutive rows (split-K flash decoding).  C is chosen on the device from
// the live lengths (about one chunk per resident block, at least min_chunk
// rows), so no length ever travels to the host.  Block t of a launch owns
// chunk t; blocks past the last chunk leave at once.
//
// attn_kernel, one block (4 wavefronts) per chunk, bf16 storage:
//   each wavefront walks 32-row steps of the chunk.  QK^T runs on the matrix
//   cores as S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (16 rows x the G query
//   heads of the KV group padded to 16; K rows are loaded straight into the
//   operand layout, 64 contiguous bytes per row and instruction).  Softmax is
//   online and in base 2, one head per lane.  PV runs as O^T = V^T P^T: the
//   step's V rows are staged in the wavefront's own LDS tile and read back
//   transposed with ds_read_b64_tr_b16; P is split into bf16 high and low
//   parts (two MFMAs) so the products keep fp32-level accuracy.  Every row's
//   scaled logit goes to the pending buffer, the chunk's (m, l, o) partial to
//   the partial buffer.  fp32 storage (head_dim 64 or 128) takes a VALU path
//   with the same outputs.  The block owning a segment's appended row also
//   copies k_new / v_new into the cache.
// finalize_kernel, one block per chunk: the segment's global (M, 1/L) per
//   head from its partials; s_j <- gamma s_j + sum_g exp2(x_gj - M_g) / L_g
//   over the chunk's rows; one slice of the segment's output combined from
//   the partials; block 0 publishes the new lengths and the outputs of
//   skipped or empty sequences.
#include <math.h>
#include <stdlib.h>

#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 256;
constexpr int kNumWaves = kThreads / kWave;
constexpr int kFlagOverflow = 1;
constexpr int kFlagBad = 4;
constexpr int kFlagAppended = 16;
constexpr float kNegBig = -1.0e30f;  // running-max start: finite, below any logit

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef __attribute__((address_space(3))) char lds_char_t;

// ---------------------------------------------------------------------------
// Chunk plan (identical in every block: a pure function of len, cap, seq_base)
// ---------------------------------------------------------------------------
struct PlanLds {
  int n_att[kMaxSeqs];     // rows attended (after the append); 0 when skipped
  int base[kMaxSeqs + 1];  // first chunk of the sequence (prefix of HK * nch)
  unsigned char flag[kMaxSeqs];
  int C;
  int tasks;
};

__device__ inline long long wave_sum_ll(long long v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Chunk size and prefix of chunk counts, by wave 0, from n_att already in P.
__device__ void plan_chunks(const DecodeArgs& a, PlanLds& P, int C_given) {
  const int lane = threadIdx.x;
  long long C = C_given;
  if (C <= 0) {
    long long total = 0;
    for (int b0 = 0; b0 < a.B; b0 += kWave) {
      const int b = b0 + lane;
      total += wave_sum_ll(b < a.B ? (long long)a.HK * P.n_att[b] : 0);
    }
    const long long per = (total + a.target_tasks - 1) / a.target_tasks;
    C = ((per + 63) / 64) * 64;
    if (C < a.min_chunk) C = a.min_chunk;
  }
  int carry = 0;
  for (int b0 = 0; b0 < a.B; b0 += kWave) {
    const int b = b0 + lane;
    const int v = (b < a.B) ? a.HK * (int)((P.n_att[b] + C - 1) / C) : 0;
    int inc = v;
    for (int o = 1; o < kWave; o <<= 1) {
      const int t = __shfl_up(inc, o);
      if (lane >= o) inc += t;
    }
    if (b < a.B) P.base[b] = carry + inc - v;
    carry += __shfl(inc, kWave - 1);
  }
  if (lane == 0) {
    P.base[a.B] = carry;
    P.C = (int)C;
    P.tasks = carry;
  }
}

__device__ void make_plan(const DecodeArgs& a, PlanLds& P) {
  const int lane = threadIdx.x;
  const bool app = a.k_new != nullptr;
  for (int b0 = 0; b0 < a.B; b0 += kWave) {
    const int b = b0 + lane;
    if (b < a.B) {
      const int n = a.len[b];
      const int c = a.cap[b];
      const long long base = a.seq_base[b];
      const bool bad = n < 0 || c < 0 || n > c || base < 0 || base + (long long)a.HK * c > a.rows_per_layer;
      const bool ovf = !bad && app && n >= c;
      P.n_att[b] = (bad || ovf) ? 0 : n + (app ? 1 : 0);
      P.flag[b] = (unsigned char)((bad ? kFlagBad : 0) | (ovf ? kFlagOverflow : 0) |
                                  ((app && !bad && !ovf) ? kFlagAppended : 0));
    }
  }
  plan_chunks(a, P, 0);
}

// Largest b with base[b] <= t (base is non-decreasing, base[0] = 0).
__device__ inline int find_seq(const int* base, int B, int t) {
  int lo = 0, hi = B;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (base[mid] <= t) lo = mid;
    else hi = mid;
  }
  return lo;
}

struct TaskInfo {
  int b, h, c, nc, r0, r1, ncache;
  bool app;
  long long segrow0;
};

__device__ inline TaskInfo task_info(const DecodeArgs& a, const PlanLds& P, int t) {
  TaskInfo ti;
  ti.b = find_seq(P.base, a.B, t);
  const int na = P.n_att[ti.b];
  ti.nc = (na + P.C - 1) / P.C;
  const int rel = t - P.base[ti.b];
  ti.h = rel / ti.nc;
  ti.c = rel % ti.nc;
  ti.r0 = ti.c * P.C;
  ti.r1 = min(ti.r0 + P.C, na);
  ti.app = (P.flag[ti.b] & kFlagAppended) != 0;
  ti.ncache = na - (ti.app ? 1 : 0);
  ti.segrow0 = a.seq_base[ti.b] + (long long)ti.h * a.cap[ti.b];
  return ti;
}

// ---------------------------------------------------------------------------
// Cross-wave combine of per-wave softmax states and the chunk partial.
// ---------------------------------------------------------------------------
struct CombineLds {
  float m[kNumWaves][8];
  float l[kNumWaves][8];
  float o[kNumWaves][8][128];
};

template <int D, int G>
__device__ void write_partial(const DecodeArgs& a, const CombineLds& cb, int t) {
  __syncthreads();
  float* part = a.part + (long long)t * G * (D + 2);
  for (int i = threadIdx.x; i < G * D; i += kThreads) {
    const int g = i / D, d = i % D;
    float mx = kNegBig;
#pragma unroll
    for (int k = 0; k < kNumWaves; ++k) mx = fmaxf(mx, cb.m[k][g]);
    float lsum = 0.0f, osum = 0.0f;
#pragma unroll
    for (int k = 0; k < kNumWaves; ++k) {
      const float f = exp2f(cb.m[k][g] - mx);
      lsum += cb.l[k][g] * f;
      osum += cb.o[k][g][d] * f;
    }
    part[g * (D + 2) + 2 + d] = osum;
    if (d == 0) {
      part[g * (D + 2)] = mx;
      part[g * (D + 2) + 1] = lsum;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 path on the matrix cores
// ---------------------------------------------------------------------------
template <int D>
struct MfmaCfg {
  static constexpr int KK = D / 32;          // k-steps of 32 over the head dim
  static constexpr int NT = D / 16;          // output tiles of 16 dims
  static constexpr int ROWB = D * 2;         // bytes per row
  static constexpr int VSTRIDE = ROWB + 32;  // padded LDS row, bytes
  static constexpr int STEP = 32;            // rows per wavefront step
  static constexpr int LPR = ROWB / 16;      // lanes per row for V loads
  static constexpr int RPL = kWave / LPR;    // rows per V load
  static constexpr int VLOADS = STEP / RPL;
  static constexpr int TILE_BYTES = STEP * VSTRIDE;
};

__device__ inline bf16x8_t zero_bf16x8() {
  bf16x8_t z;
#pragma unroll
  for (int j = 0; j < 8; ++j) z[j] = (__bf16)0.0f;
  return z;
}

template <int D, int G>
__device__ void attn_chunk_mfma(const DecodeArgs& a, const PlanLds& P, char* vtiles, CombineLds& cb, int t) {
  using Cfg = MfmaCfg<D>;
  constexpr int KK = Cfg::KK, NT = Cfg::NT, ROWB = Cfg::ROWB, VSTRIDE = Cfg::VSTRIDE;
  constexpr int STEP = Cfg::STEP, LPR = Cfg::LPR, RPL = Cfg::RPL, VLOADS = Cfg::VLOADS;
  static_assert(G <= 16, "heads of a group are padded to 16 MFMA columns");
  const TaskInfo ti = task_info(a, P, t);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int g4 = lane >> 4;  // lane group: rows 4*g4.. of a 16-row tile
  const int s = lane & 15;   // query head (C/B layouts) or row (A layout)
  const int HQ = a.HK * G;
  char* vb = vtiles + w * Cfg::TILE_BYTES;

  // Q^T operand: lane holds Q[head s][32 kk + 8 g4 .. +8].
  bf16x8_t qb[KK];
  {
    const char* qrow = reinterpret_cast<const char*>(a.q) + (((long long)ti.b * HQ + (long long)ti.h * G + s) * D) * 2;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qb[kk] = (s < G) ? *reinterpret_cast<const bf16x8_t*>(qrow + 64 * kk + 16 * g4) : zero_bf16x8();
  }
  float m = kNegBig, l = 0.0f;
  f32x4_t o[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) o[nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  const char* Kb = reinterpret_cast<const char*>(a.k) + ti.segrow0 * ROWB;
  const char* Vb = reinterpret_cast<const char*>(a.v) + ti.segrow0 * ROWB;
  float* pend = a.pend + ti.segrow0 * G;
  const float sc = a.scale_log2;
  const int re = min(ti.r1, ti.ncache);

  for (int base = ti.r0 + STEP * w; base < re; base += STEP * kNumWaves) {
    bf16x8_t kr[2][KK];
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      const int row = min(base + 16 * T + s, re - 1);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kr[T][kk] = *reinterpret_cast<const bf16x8_t*>(Kb + (long long)row * ROWB + 64 * kk + 16 * g4);
    }
    uint4 vr[VLOADS];
#pragma unroll
    for (int u = 0; u < VLOADS; ++u) {
      const int row = min(base + RPL * u + lane / LPR, re - 1);
      vr[u] = *reinterpret_cast<const uint4*>(Vb + (long long)row * ROWB + 16 * (lane % LPR));
    }
    f32x4_t sacc[2];
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      sacc[T] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) sacc[T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[T][kk], qb[kk], sacc[T], 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < VLOADS; ++u)
      *reinterpret_cast<uint4*>(vb + (RPL * u + lane / LPR) * VSTRIDE + 16 * (lane % LPR)) = vr[u];

    // Logits of rows base + 16 T + 4 g4 + rr for head s.
    float x[2][4];
    float mx = kNegBig;
#pragma unroll
    for (int T = 0; T < 2; ++T) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int row = base + 16 * T + 4 * g4 + rr;
        const float v = sacc[T][rr] * sc;
        const bool ok = row < re;
        if (ok && s < G) pend[(long long)row * G + s] = v;
        x[T][rr] = ok ? v : -INFINITY;
        mx = fmaxf(mx, x[T][rr]);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx);
    const float corr = exp2f(m - mnew);
    float psum = 0.0f;
    bf16x8_t ph, pl;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = exp2f(x[j >> 2][j & 3] - mnew);
      psum += p;
      const __bf16 hi = (__bf16)p;
      ph[j] = hi;
      pl[j] = (__bf16)(p - (float)hi);
    }
    l = l * corr + psum;
    m = mnew;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) o[nt] *= corr;
    // V^T operand through the transposing LDS read: lane s of group g4
    // points at row 4 g4 + s/4 (and 16 more), column 16 nt + 4 (s % 4).
    const int rsub = 4 * g4 + (s >> 2);
    lds_char_t* vbl = (lds_char_t*)(vb);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int col = (16 * nt + 4 * (s & 3)) * 2;
      const bf16x4_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(reinterpret_cast<lds_bf16x4_t*>(vbl + rsub * VSTRIDE + col));
      const bf16x4_t a1 =
          __builtin_amdgcn_ds_read_tr16_b64_v4bf16(reinterpret_cast<lds_bf16x4_t*>(vbl + (rsub + 16) * VSTRIDE + col));
      const bf16x8_t av = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
      o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, ph, o[nt], 0, 0, 0);
      o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pl, o[nt], 0, 0, 0);
    }
  }

  // The appended row (last chunk of its segment), by wave 0: read from
  // k_new / v_new, copied into the cache, and folded into wave 0's state.
  if (ti.app && ti.r1 == ti.ncache + 1 && w == 0) {
    const char* kn = reinterpret_cast<const char*>(a.k_new) + (((long long)ti.b * a.HK + ti.h) * D) * 2;
    const char* vn = reinterpret_cast<const char*>(a.v_new) + (((long long)ti.b * a.HK + ti.h) * D) * 2;
    if (lane < LPR) {
      *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.k_w) + (ti.segrow0 + ti.ncache) * ROWB + 16 * lane) =
          *reinterpret_cast<const uint4*>(kn + 16 * lane);
      *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.v_w) + (ti.segrow0 + ti.ncache) * ROWB + 16 * lane) =
          *reinterpret_cast<const uint4*>(vn + 16 * lane);
    }
    // x_s = scale q_s . k_new: each lane group sums its quarter of the dims.
    float acc = 0.0f;
    const uint32_t* kq = reinterpret_cast<const uint32_t*>(kn);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const bf16x8_t qv = qb[kk];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x2_t q2 = {qv[2 * j], qv[2 * j + 1]};
        const uint32_t k2 = kq[(32 * kk + 8 * g4) / 2 + j];
        acc = __builtin_amdgcn_fdot2_f32_bf16(q2, __builtin_bit_cast(bf16x2_t, k2), acc, false);
      }
    }
    acc += __shfl_xor(acc, 16);
    acc += __shfl_xor(acc, 32);
    const float x = acc * sc;
    if (g4 == 0 && s < G) pend[(long long)ti.ncache * G + s] = x;
    const float mnew = fmaxf(m, x);
    const float corr = exp2f(m - mnew);
    const float p = exp2f(x - mnew);
    l = l * corr + (g4 == 0 ? p : 0.0f);
    m = mnew;
    const uint16_t* vv = reinterpret_cast<const uint16_t*>(vn);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float vf = __uint_as_float((uint32_t)vv[16 * nt + 4 * g4 + rr] << 16);
        o[nt][rr] = o[nt][rr] * corr + p * vf;
      }
    }
  }

  // Per-wave state to LDS: m is common to the four lane groups, l is split.
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  __syncthreads();  // the V tiles alias the combine area
  if (s < G) {
    if (g4 == 0) {
      cb.m[w][s] = m;
      cb.l[w][s] = l;
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) cb.o[w][s][16 * nt + 4 * g4 + rr] = o[nt][rr];
  }
  write_partial<D, G>(a, cb, t);
}

// ---------------------------------------------------------------------------
// fp32 path (VALU): 16-byte loads, D/4 lanes per row.
// ---------------------------------------------------------------------------
template <int D, int G>
__device__ void attn_chunk_f32(const DecodeArgs& a, const PlanLds& P, CombineLds& cb, int t) {
  constexpr int EPL = 4;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  constexpr int U = 4;
  constexpr int ROWS_WAVE = U * RPW;
  constexpr int ROWS_BLOCK = ROWS_WAVE * kNumWaves;
  static_assert(G <= LPR, "one logit-writer lane per head");
  const TaskInfo ti = task_info(a, P, t);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int rg = lane / LPR;
  const int dp = lane % LPR;
  const int HQ = a.HK * G;

  float qf[G][EPL];
  {
    const float* qb = reinterpret_cast<const float*>(a.q) + ((long long)ti.b * HQ + (long long)ti.h * G) * D + dp * EPL;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint4 r = *reinterpret_cast<const uint4*>(qb + (long long)g * D);
      qf[g][0] = __uint_as_float(r.x) * a.scale_log2;
      qf[g][1] = __uint_as_float(r.y) * a.scale_log2;
      qf[g][2] = __uint_as_float(r.z) * a.scale_log2;
      qf[g][3] = __uint_as_float(r.w) * a.scale_log2;
    }
  }
  float m[G], l[G], o[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = kNegBig;
    l[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[g][e] = 0.0f;
  }
  const float* Kb = reinterpret_cast<const float*>(a.k) + ti.segrow0 * D + dp * EPL;
  const float* Vb = reinterpret_cast<const float*>(a.v) + ti.segrow0 * D + dp * EPL;
  float* pend = a.pend + ti.segrow0 * G;

  auto consume = [&](const uint4* kr, const uint4* vr, const int* row, const bool* valid) {
    float x[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[EPL];
      Elem<float>::unpack(kr[u], kf);
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
      float mine = x[u][0];
#pragma unroll
      for (int g = 1; g < G; ++g) mine = (dp == g) ? x[u][g] : mine;
      if (valid[u] && dp < G) pend[(long long)row[u] * G + dp] = mine;
#pragma unroll
      for (int g = 0; g < G; ++g) x[u][g] = valid[u] ? x[u][g] : -INFINITY;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = m[g];
#pragma unroll
      for (int u = 0; u < U; ++u) mx = fmaxf(mx, x[u][g]);
      const float corr = exp2f(m[g] - mx);
      float lg = l[g] * corr;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] *= corr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = exp2f(x[u][g] - mx);
        float vf[EPL];
        Elem<float>::unpack(vr[u], vf);
        lg += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] = fmaf(p, vf[e], o[g][e]);
      }
      l[g] = lg;
      m[g] = mx;
    }
  };

  const int re = min(ti.r1, ti.ncache);
  for (int base = ti.r0 + w * ROWS_WAVE; base < re; base += ROWS_BLOCK) {
    uint4 kr[U], vr[U];
    int row[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      row[u] = base + u * RPW + rg;
      valid[u] = row[u] < re;
      const int rr = valid[u] ? row[u] : (re - 1);
      kr[u] = *reinterpret_cast<const uint4*>(Kb + (long long)rr * D);
      vr[u] = *reinterpret_cast<const uint4*>(Vb + (long long)rr * D);
    }
    consume(kr, vr, row, valid);
  }
  if (ti.app && ti.r1 == ti.ncache + 1 && w == 0) {
    const long long nb = ((long long)ti.b * a.HK + ti.h) * D + dp * EPL;
    uint4 kr[U], vr[U];
    int row[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      row[u] = ti.ncache;
      valid[u] = (u == 0) && (rg == 0);
      kr[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(a.k_new) + nb);
      vr[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(a.v_new) + nb);
    }
    if (rg == 0) {
      *reinterpret_cast<uint4*>(reinterpret_cast<float*>(a.k_w) + (ti.segrow0 + ti.ncache) * D + dp * EPL) = kr[0];
      *reinterpret_cast<uint4*>(reinterpret_cast<float*>(a.v_w) + (ti.segrow0 + ti.ncache) * D + dp * EPL) = vr[0];
    }
    consume(kr, vr, row, valid);
  }
#pragma unroll
  for (int off = LPR; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float mo = __shfl_xor(m[g], off);
      const float lo = __shfl_xor(l[g], off);
      const float mx = fmaxf(m[g], mo);
      const float fa = exp2f(m[g] - mx);
      const float fb = exp2f(mo - mx);
      l[g] = l[g] * fa + lo * fb;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float oo = __shfl_xor(o[g][e], off);
        o[g][e] = o[g][e] * fa + oo * fb;
      }
      m[g] = mx;
    }
  }
  __syncthreads();
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
  write_partial<D, G>(a, cb, t);
}

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------
template <typename T, int D>
struct AttnLds;

template <int D>
struct AttnLds<bf16_t, D> {
  union {
    char vtiles[kNumWaves * MfmaCfg<D>::TILE_BYTES];
    CombineLds cb;
  };
};

template <int D>
struct AttnLds<float, D> {
  CombineLds cb;
};

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void attn_kernel(DecodeArgs a) {
  __shared__ PlanLds P;
  __shared__ __attribute__((aligned(16))) AttnLds<T, D> L;
  const int tid = threadIdx.x;
  if (tid < kWave) make_plan(a, P);
  __syncthreads();
  const int t = blockIdx.x;
  if (t == 0) {
    // Publish the plan for the finalize kernel.
    int* pl = a.plan;
    for (int b = tid; b < a.B; b += kThreads) {
      pl[kPlanHdr + b] = P.n_att[b];
      pl[kPlanHdr + kMaxSeqs + b] = P.flag[b];
    }
    if (tid == 0) {
      pl[kPlanC] = P.C;
      pl[kPlanTasks] = P.tasks;
    }
  }
  if (t >= P.tasks) return;
  if constexpr (sizeof(T) == 2)
    attn_chunk_mfma<D, G>(a, P, L.vtiles, L.cb, t);
  else
    attn_chunk_f32<D, G>(a, P, L.cb, t);
}

struct FinLds {
  PlanLds P;
  float M[8];
  float invL[8];
};

template <int D, int G>
__global__ __launch_bounds__(kThreads) void finalize_kernel(DecodeArgs a) {
  __shared__ FinLds F;
  const int tid = threadIdx.x;
  const int* pl = a.plan;
  const int t = blockIdx.x;
  const int tasks = pl[kPlanTasks];
  if (t >= tasks && t != 0) return;
  for (int b = tid; b < a.B; b += kThreads) {
    F.P.n_att[b] = pl[kPlanHdr + b];
    F.P.flag[b] = (unsigned char)pl[kPlanHdr + kMaxSeqs + b];
  }
  __syncthreads();
  if (tid < kWave) plan_chunks(a, F.P, pl[kPlanC]);
  __syncthreads();
  const int HQ = a.HK * G;
  if (t == 0) {
    for (int b = tid; b < a.B; b += kThreads)
      if (F.P.flag[b] & kFlagAppended) a.len[b] = F.P.n_att[b];
    int fl = 0;
    for (int b = tid; b < a.B; b += kThreads) fl |= F.P.flag[b] & (kFlagOverflow | kFlagBad);
    atomic_or_status(a.dev_status, fl);
    for (int b = 0; b < a.B; ++b) {
      if (F.P.n_att[b] != 0) continue;
      const float fill = (F.P.flag[b] & (kFlagOverflow | kFlagBad)) ? __int_as_float(0x7fc00000) : 0.0f;
      float* ob = a.out + (long long)b * HQ * D;
      for (int i = tid; i < HQ * D; i += kThreads) ob[i] = fill;
    }
  }
  if (t >= tasks) return;
  const TaskInfo ti = task_info(a, F.P, t);
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const float* part0 = a.part + (long long)(F.P.base[ti.b] + ti.h * ti.nc) * G * (D + 2);
  for (int g = w; g < G; g += kNumWaves) {
    float mx = kNegBig;
    for (int cc = lane; cc < ti.nc; cc += kWave) mx = fmaxf(mx, part0[(long long)cc * G * (D + 2) + g * (D + 2)]);
    mx = wave_max(mx);
    float ls = 0.0f;
    for (int cc = lane; cc < ti.nc; cc += kWave) {
      const float* p = part0 + (long long)cc * G * (D + 2) + g * (D + 2);
      ls += p[1] * exp2f(p[0] - mx);
    }
    ls = wave_sum(ls);
    if (lane == 0) {
      F.M[g] = mx;
      F.invL[g] = 1.0f / ls;
    }
  }
  __syncthreads();
  // Scores of the chunk's rows.
  const float* pend = a.pend + ti.segrow0 * G;
  float* score = a.score + ti.segrow0;
  for (int r = ti.r0 + tid; r < ti.r1; r += kThreads) {
    float acc = 0.0f;
#pragma unroll
    for (int g = 0; g < G; ++g) acc += exp2f(pend[(long long)r * G + g] - F.M[g]) * F.invL[g];
    const float s_old = (r < ti.ncache) ? score[r] : 0.0f;
    score[r] = fmaf(a.gamma, s_old, acc);
  }
  // One slice of the segment's output: elements [e0, e1) of its G x D block.
  const int per = (G * D + ti.nc - 1) / ti.nc;
  const int e0 = ti.c * per, e1 = min(e0 + per, G * D);
  float* outb = a.out + ((long long)ti.b * HQ + (long long)ti.h * G) * D;
  for (int e = e0 + tid; e < e1; e += kThreads) {
    const int g = e / D, d = e % D;
    const float Mg = F.M[g];
    float acc = 0.0f;
    int cc = 0;
    for (; cc + 4 <= ti.nc; cc += 4) {
      float mv[4], ov[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float* p = part0 + (long long)(cc + k) * G * (D + 2) + g * (D + 2);
        mv[k] = p[0];
        ov[k] = p[2 + d];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) acc = fmaf(ov[k], exp2f(mv[k] - Mg), acc);
    }
    for (; cc < ti.nc; ++cc) {
      const float* p = part0 + (long long)cc * G * (D + 2) + g * (D + 2);
      acc = fmaf(p[2 + d], exp2f(p[0] - Mg), acc);
    }
    outb[e] = acc * F.invL[g];
  }
}

// Optional tuning overrides, read once: LETHE_DECODE_TASKS (chunks to aim
// for per launch) and LETHE_DECODE_MIN_CHUNK (rows).
int env_int(const char* name) {
  const char* v = getenv(name);
  return v ? atoi(v) : 0;
}

template <typename T, int D, int G>
lethe_status launch_tdg(const DecodeArgs& a_in, hipStream_t s) {
  DecodeArgs a = a_in;
  // Resident blocks per device for this instantiation; the value depends only
  // on the device, so concurrent first calls store the same number.
  static int resident[64];
  static const int env_tasks = env_int("LETHE_DECODE_TASKS");
  static const int env_chunk = env_int("LETHE_DECODE_MIN_CHUNK");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LETHE_ERR_HIP;
  int blocks = (dev >= 0 && dev < 64) ? __atomic_load_n(&resident[dev], __ATOMIC_RELAXED) : 0;
  if (blocks <= 0) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return LETHE_ERR_HIP;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_kernel<T, D, G>, kThreads, 0) != hipSuccess)
      return LETHE_ERR_HIP;
    blocks = cus * (per_cu < 1 ? 1 : per_cu);
    if (dev >= 0 && dev < 64) __atomic_store_n(&resident[dev], blocks, __ATOMIC_RELAXED);
  }
  a.target_tasks = env_tasks > 0 ? env_tasks : blocks;
  if (a.target_tasks > kMaxDecodeTasks) a.target_tasks = kMaxDecodeTasks;
  a.min_chunk = env_chunk > 0 ? ((env_chunk + 63) / 64) * 64 : 256;
  const int grid = a.target_tasks + a.B * a.HK;  // upper bound on the chunk count
  hipLaunchKernelGGL((attn_kernel<T, D, G>), dim3(grid), dim3(kThreads), 0, s, a);
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

lethe_status launch_decode(const DecodeArgs& a, lethe_dtype dt, int D, int G, hipStream_t s) {
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
