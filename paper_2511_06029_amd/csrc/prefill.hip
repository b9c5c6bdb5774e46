// Causal prefill attention that seeds the importance scores (Eq. 2 summed
// over the prompt's queries and the query heads of each KV group), gfx950.
//
// The qlen newest rows of each (sequence, KV head) segment come with queries;
// query i sits at position p = n - qlen + i and attends rows 0 .. p.  Two
// launches:
//
//  1. prefill_fwd_kernel: flash attention forward.  A block holds 32 query
//     positions of one KV group and up to four of its query heads (one head
//     per wavefront) and walks the keys in 32-row steps, K and V tiles shared
//     by the waves through LDS (direct loads, double buffered).  S^T = K Q^T
//     on the matrix cores (v_mfma_f32_16x16x32_bf16), online softmax in base
//     2 with one query per lane column, O^T = V^T P^T with P split into bf16
//     high and low parts for fp32-level accuracy.  Writes out and each
//     query's final (max, 1 / sum).
//  2. prefill_score_kernel: key-major.  A block owns 256 keys (64 per wave,
//     K in registers) and walks every later query tile of every head of the
//     group, recomputing S^T and summing exp2(x - max) / sum over the
//     queries; each key's total is added to its score once, so there are no
//     atomics and the result does not depend on scheduling.
#include <math.h>

#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kPfThreads = 256;
constexpr int kPfWaves = kPfThreads / kWave;
constexpr float kPfNegBig = -1.0e30f;

typedef __bf16 pf_bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 pf_bf16x4_t __attribute__((ext_vector_type(4)));
typedef float pf_f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) pf_bf16x4_t pf_lds_bf16x4_t;
typedef __attribute__((address_space(3))) char pf_lds_char_t;
typedef __attribute__((address_space(3))) void pf_lds_void_t;
typedef __attribute__((address_space(1))) const void pf_global_cvoid_t;

template <int D>
struct PfCfg {
  static constexpr int KK = D / 32;          // k-steps of 32 over the head dim
  static constexpr int NT = D / 16;          // output tiles of 16 dims
  static constexpr int ROWB = D * 2;         // bytes per bf16 row
  static constexpr int CH = ROWB / 16;       // 16-byte chunks per row
  static constexpr int STEP = 32;            // key rows per step
  // K / Q tiles: chunk c of row r at 16-byte slot r CH + (c ^ (r mod CH)), so
  // the 16 rows an operand read touches fall in different LDS banks.
  static constexpr int KTILE = STEP * ROWB;
  static __device__ constexpr int kslot(int r, int c) { return r * CH + (c ^ (r % CH)); }
  // V tiles: load u (one wavefront, 16 bytes a lane) carries rows
  // u + VLOADS j; blocks of 1 KB + 32 bytes keep the rows of one transposing
  // read 8 banks apart.
  static constexpr int LPR = ROWB / 16;
  static constexpr int RPL = kWave / LPR;
  static constexpr int VLOADS = STEP / RPL;
  static constexpr int VBLK = kWave * 16 + 32;
  static constexpr int VTILE = VLOADS * VBLK;
  static __device__ constexpr int vaddr(int r, int c) { return (r % VLOADS) * VBLK + (r / VLOADS) * ROWB + c; }
  static constexpr int BUF = KTILE + VTILE;
};

// s_waitcnt with only a vector-memory count (expcnt and lgkmcnt left free).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Transposing 64-bit LDS read of four bf16 values.  Written as inline
// assembly so that the compiler does not order it after every outstanding
// direct-to-LDS load (it cannot tell which buffer those fill).  The compiler
// does not track these reads either: lgkm_fence() must run before the
// results are used.
__device__ inline pf_bf16x4_t lds_read_tr(const pf_lds_char_t* p) {
  typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
  u32x2_t r;
  const unsigned addr = (unsigned)(unsigned long)p;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(addr));
  return __builtin_bit_cast(pf_bf16x4_t, r);
}

// Waits for every outstanding LDS read.  The operands tie the wait to the
// registers those reads fill, so no use of them can be scheduled before it.
template <int NT>
__device__ inline void lgkm_fence(pf_bf16x8_t (&v)[NT]) {
  static_assert(NT == 4 || NT == 8, "operand tiles");
  if constexpr (NT == 4) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7]));
  }
}

// 64-bit LDS read that waits for its own result (same reason as lds_read_tr).
__device__ inline float2 lds_read_f2(const pf_lds_char_t* p) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  f32x2_t r;
  const unsigned addr = (unsigned)(unsigned long)p;
  asm volatile("ds_read_b64 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(r) : "v"(addr));
  return make_float2(r[0], r[1]);
}

__device__ inline pf_bf16x8_t pf_zero8() {
  pf_bf16x8_t z;
#pragma unroll
  for (int j = 0; j < 8; ++j) z[j] = (__bf16)0.0f;
  return z;
}

// Sizes of one sequence, or false (flagged) when they do not fit together.
struct PfSeq {
  int n, qlen, first;
  long long q0, row0;
};

__device__ inline bool pf_seq(const PrefillArgs& a, int b, int h, PfSeq& sq) {
  const int n = a.len[(long long)a.layer * a.B + b];
  const int qlen = a.q_len[b];
  const int c = a.cap[b];
  const long long base = a.seq_base[b];
  const long long q0 = a.q_start[b];
  const bool ok = n >= 0 && c >= 0 && n <= c && base >= 0 && base + (long long)a.HK * c <= a.rows_per_layer &&
                  qlen >= 0 && qlen <= n && qlen <= a.max_q && n <= a.max_kv && q0 >= 0 && q0 + qlen <= a.q_rows;
  sq.n = n;
  sq.qlen = qlen;
  sq.first = n - qlen;
  sq.q0 = q0;
  sq.row0 = base + (long long)h * c;
  return ok;
}

// ---------------------------------------------------------------------------
// Pass 1: outputs and per-query softmax statistics.
// ---------------------------------------------------------------------------
template <int D, int G>
__global__ __launch_bounds__(kPfThreads) __attribute__((amdgpu_waves_per_eu(2))) void prefill_fwd_kernel(PrefillArgs a) {
  using Cfg = PfCfg<D>;
  constexpr int KK = Cfg::KK, NT = Cfg::NT, ROWB = Cfg::ROWB, CH = Cfg::CH;
  constexpr int NQUAD = (G + 3) / 4;
  constexpr int NBUF = 3;  // tiles st, st + 1 and st + 2 in flight
  constexpr int KLOADS = Cfg::KTILE / (kWave * 16);
  constexpr int LPW = (KLOADS + Cfg::VLOADS) / kPfWaves;  // direct loads per wave and step
  static_assert((KLOADS + Cfg::VLOADS) % kPfWaves == 0, "loads split evenly over the waves");
  __shared__ __attribute__((aligned(16))) char tiles[NBUF][Cfg::BUF];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int g4 = lane >> 4;
  const int s = lane & 15;
  const int ntiles = (a.max_q + 31) / 32;
  int idx = blockIdx.x;
  const int quad = idx % NQUAD;
  idx /= NQUAD;
  const int seg = idx % (a.B * a.HK);
  const int pt = ntiles - 1 - idx / (a.B * a.HK);  // longest rows first
  const int b = seg / a.HK, h = seg % a.HK;
  PfSeq sq;
  if (!pf_seq(a, b, h, sq)) {
    if (tid == 0 && pt == 0 && quad == 0) atomicOr(a.dev_status, LETHE_DEV_BAD_LAYOUT);
    return;
  }
  if (32 * pt >= sq.qlen) return;
  const int HQ = a.HK * G;
  const int g = 4 * quad + w;
  const bool active = g < G;  // wave-uniform
  const int p0 = sq.first + 32 * pt;
  const int kend = min(sq.n, p0 + 32);
  const int nsteps = (kend + Cfg::STEP - 1) / Cfg::STEP;
  const char* Kb = reinterpret_cast<const char*>(a.k) + sq.row0 * ROWB;
  const char* Vb = reinterpret_cast<const char*>(a.v) + sq.row0 * ROWB;
  const float sc = a.scale_log2;

  // Queries of this wave's head as the B operand of S^T = K Q^T: lane (g4, s)
  // of tile qt holds Q[query 32 pt + 16 qt + s][dims 32 kk + 8 g4 ..].
  pf_bf16x8_t qb[2][KK];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int i = 32 * pt + 16 * qt + s;
    const char* qrow = reinterpret_cast<const char*>(a.q) + ((sq.q0 + i) * HQ + (long long)h * G + g) * ROWB;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qb[qt][kk] = (active && i < sq.qlen) ? *reinterpret_cast<const pf_bf16x8_t*>(qrow + 64 * kk + 16 * g4)
                                           : pf_zero8();
  }

  auto issue = [&](int st, int buf) {
    const int j0 = st * Cfg::STEP;
    char* kt = tiles[buf];
    char* vt = tiles[buf] + Cfg::KTILE;
#pragma unroll
    for (int t = w; t < KLOADS + Cfg::VLOADS; t += kPfWaves) {
      if (t < KLOADS) {
        const int q = kWave * t + lane;
        const int r = q / CH, c = (q % CH) ^ (r % CH);
        const int row = min(j0 + r, kend - 1);
        __builtin_amdgcn_global_load_lds((pf_global_cvoid_t*)(Kb + (long long)row * ROWB + 16 * c),
                                         (pf_lds_void_t*)((pf_lds_char_t*)kt + kWave * 16 * t), 16, 0, 0);
      } else {
        const int u = t - KLOADS;
        const int row = min(j0 + u + Cfg::VLOADS * (lane / Cfg::LPR), kend - 1);
        __builtin_amdgcn_global_load_lds((pf_global_cvoid_t*)(Vb + (long long)row * ROWB + 16 * (lane % Cfg::LPR)),
                                         (pf_lds_void_t*)((pf_lds_char_t*)vt + u * Cfg::VBLK), 16, 0, 0);
      }
    }
  };

  float m[2] = {kPfNegBig, kPfNegBig}, l[2] = {0.0f, 0.0f};
  pf_f32x4_t o[NT][2];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) o[nt][0] = o[nt][1] = pf_f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  issue(0, 0);
  if (nsteps > 1) issue(1, 1);
  const int rsub = 4 * g4 + (s >> 2);
  for (int st = 0; st < nsteps; ++st) {
    // This wave's loads of tile st are done once at most the LPW loads of
    // tile st + 1 are outstanding; the barrier makes every wave's visible
    // and guarantees tile st - 1 has been read by all.
    if (st + 1 < nsteps)
      wait_vmcnt<LPW>();
    else
      wait_vmcnt<0>();
    __syncthreads();
    if (st + 2 < nsteps) issue(st + 2, (st + 2) % NBUF);
    if (!active) continue;
    const int j0 = st * Cfg::STEP;
    const char* kt = tiles[st % NBUF];
    const pf_lds_char_t* vt = (const pf_lds_char_t*)(tiles[st % NBUF] + Cfg::KTILE);
    // V^T operands through the transposing LDS read: lane s of group g4
    // points at row 4 g4 + s / 4 and 16 rows further, column 16 nt + 4 (s mod 4).
    pf_bf16x8_t av[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int col = (16 * nt + 4 * (s & 3)) * 2;
      const pf_bf16x4_t a0 = lds_read_tr(vt + Cfg::vaddr(rsub, col));
      const pf_bf16x4_t a1 = lds_read_tr(vt + Cfg::vaddr(rsub + 16, col));
      av[nt] = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    }

    pf_f32x4_t sacc[2][2];
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      pf_bf16x8_t kr[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kr[kk] = *reinterpret_cast<const pf_bf16x8_t*>(kt + 16 * Cfg::kslot(16 * T + s, 4 * kk + g4));
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        sacc[T][qt] = pf_f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          sacc[T][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[kk], qb[qt][kk], sacc[T][qt], 0, 0, 0);
      }
    }

    // Softmax of query 16 qt + s over keys j0 + 16 T + 4 g4 + rr.  Steps
    // wholly below the diagonal (every key precedes every query of the tile
    // and is live) skip the mask.
    const bool interior = j0 + Cfg::STEP - 1 <= p0 && j0 + Cfg::STEP <= kend;
    pf_bf16x8_t ph[2], pl[2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      const int pos = p0 + 16 * qt + s;
      float x[8];
      float mx = kPfNegBig;
      if (interior) {
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          x[jj] = sacc[jj >> 2][qt][jj & 3] * sc;
          mx = fmaxf(mx, x[jj]);
        }
      } else {
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          const int key = j0 + 16 * (jj >> 2) + 4 * g4 + (jj & 3);
          x[jj] = (key <= pos && key < kend) ? sacc[jj >> 2][qt][jj & 3] * sc : -INFINITY;
          mx = fmaxf(mx, x[jj]);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(m[qt], mx);
      const float corr = hw_exp2(m[qt] - mnew);
      float psum = 0.0f;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const float p = hw_exp2(x[jj] - mnew);
        psum += p;
        const __bf16 hi = (__bf16)p;
        ph[qt][jj] = hi;
        pl[qt][jj] = (__bf16)(p - (float)hi);
      }
      l[qt] = l[qt] * corr + psum;
      m[qt] = mnew;
      // Once the running maxima settle most steps leave every lane's
      // correction at exactly 1; the wave then skips the rescale.
      if (__any(corr != 1.0f)) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) o[nt][qt] *= corr;
      }
    }

    // O^T += V^T P^T.
    lgkm_fence<NT>(av);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        o[nt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[nt], ph[qt], o[nt][qt], 0, 0, 0);
        o[nt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[nt], pl[qt], o[nt][qt], 0, 0, 0);
      }
    }
  }
  if (!active) return;

  // l is split over the four lane groups of a query column; m is common.
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    float lt = l[qt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const int i = 32 * pt + 16 * qt + s;
    if (i >= sq.qlen) continue;
    const float inv = 1.0f / lt;
    const long long qrow = (sq.q0 + i) * HQ + (long long)h * G + g;
    float* orow = a.out + qrow * D;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const pf_f32x4_t v = o[nt][qt] * inv;
      *reinterpret_cast<float4*>(orow + 16 * nt + 4 * g4) = make_float4(v[0], v[1], v[2], v[3]);
    }
    if (g4 == 0)
      *reinterpret_cast<float2*>(a.stat + 2 * ((long long)(h * G + g) * a.q_rows + sq.q0 + i)) = make_float2(m[qt], inv);
  }
}

// ---------------------------------------------------------------------------
// Pass 2: importance seeding, key-major.
// ---------------------------------------------------------------------------
constexpr int kPfKeysPerWave = 64;
constexpr int kPfKeysPerBlock = kPfWaves * kPfKeysPerWave;
constexpr int kPfItemQ = 32;  // queries of one head per work item

template <int D, int G>
__global__ __launch_bounds__(kPfThreads) void prefill_score_kernel(PrefillArgs a) {
  using Cfg = PfCfg<D>;
  constexpr int KK = Cfg::KK, ROWB = Cfg::ROWB, CH = Cfg::CH;
  constexpr int QTILE = kPfItemQ * ROWB;
  constexpr int STATB = kPfItemQ * 8;  // (max, 1 / sum) per query
  constexpr int BUFB = QTILE + STATB;
  constexpr int NBUF = 3;
  constexpr int QLOADS = QTILE / (kWave * 16);
  static_assert(QLOADS % kPfWaves == 0, "query loads split evenly over the waves");
  constexpr int LPW = QLOADS / kPfWaves;  // plus one statistics load on wave 0
  __shared__ __attribute__((aligned(16))) char bufs[NBUF][BUFB];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int g4 = lane >> 4;
  const int s = lane & 15;
  const int seg = blockIdx.x % (a.B * a.HK);
  const int kb = blockIdx.x / (a.B * a.HK);  // low keys (most queries) first
  const int b = seg / a.HK, h = seg % a.HK;
  PfSeq sq;
  if (!pf_seq(a, b, h, sq)) return;  // flagged by the forward pass
  const int kblk0 = kPfKeysPerBlock * kb;
  if (sq.qlen == 0 || kblk0 >= sq.n) return;
  const int HQ = a.HK * G;
  const int j0w = kblk0 + kPfKeysPerWave * w;
  const char* Kb = reinterpret_cast<const char*>(a.k) + sq.row0 * ROWB;
  const float sc = a.scale_log2;

  // This wave's 64 keys as the A operand (row 16 T + s, dims 32 kk + 8 g4 ..).
  pf_bf16x8_t kr[4][KK];
#pragma unroll
  for (int T = 0; T < 4; ++T) {
    const int row = min(j0w + 16 * T + s, sq.n - 1);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      kr[T][kk] = *reinterpret_cast<const pf_bf16x8_t*>(Kb + (long long)row * ROWB + 64 * kk + 16 * g4);
  }

  // Work items: (tile of 32 queries, head) for every tile holding a position
  // at or after the block's first key.
  const int it0 = max(0, kblk0 - sq.first) / kPfItemQ;
  const int nit = (sq.qlen + kPfItemQ - 1) / kPfItemQ - it0;
  const int nitems = nit * G;
  auto issue = [&](int item, int buf) {
    const int it = it0 + item / G, g = item % G;
#pragma unroll
    for (int t = w; t < QLOADS; t += kPfWaves) {
      const int q = kWave * t + lane;
      const int r = q / CH, c = (q % CH) ^ (r % CH);
      const int i = min(kPfItemQ * it + r, sq.qlen - 1);
      const char* src = reinterpret_cast<const char*>(a.q) + ((sq.q0 + i) * HQ + (long long)h * G + g) * ROWB + 16 * c;
      __builtin_amdgcn_global_load_lds((pf_global_cvoid_t*)src,
                                       (pf_lds_void_t*)((pf_lds_char_t*)bufs[buf] + kWave * 16 * t), 16, 0, 0);
    }
    if (w == 0 && lane < kPfItemQ / 2) {
      // Statistics of the item's queries: 32 x 8 bytes, two queries a lane.
      // A pair may reach one entry past the live ones (the workspace has
      // slack for it); those entries belong to masked queries.
      const int i = min(kPfItemQ * it + 2 * lane, sq.qlen - 1);
      const float* src = a.stat + 2 * ((long long)(h * G + g) * a.q_rows + sq.q0 + i);
      __builtin_amdgcn_global_load_lds((pf_global_cvoid_t*)src, (pf_lds_void_t*)((pf_lds_char_t*)bufs[buf] + QTILE),
                                       16, 0, 0);
    }
  };

  float acc[4][4];
#pragma unroll
  for (int T = 0; T < 4; ++T)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) acc[T][rr] = 0.0f;

  if (nitems > 0) issue(0, 0);
  if (nitems > 1) issue(1, 1);
  for (int item = 0; item < nitems; ++item) {
    if (item + 1 < nitems) {
      if (w == 0)
        wait_vmcnt<LPW + 1>();
      else
        wait_vmcnt<LPW>();
    } else {
      wait_vmcnt<0>();
    }
    __syncthreads();
    if (item + 2 < nitems) issue(item + 2, (item + 2) % NBUF);
    const int it = it0 + item / G;
    const int pos0 = sq.first + kPfItemQ * it;  // position of the tile's first query
    // Nothing to do when every query of the tile precedes this wave's keys.
    if (pos0 + kPfItemQ - 1 < j0w || j0w >= sq.n) continue;
    const char* qt = bufs[item % NBUF];
    const float* stl = reinterpret_cast<const float*>(qt + QTILE);
    // No masking when every key is live and precedes every (live) query.
    const bool full = j0w + kPfKeysPerWave - 1 <= pos0 && kPfItemQ * (it + 1) <= sq.qlen &&
                      j0w + kPfKeysPerWave <= sq.n;
    constexpr int QH = kPfItemQ / 16;
    // Both query halves' operands and statistics, then every MFMA of the
    // item with the k-step outermost: QH * 4 independent accumulators.
    pf_bf16x8_t qv[QH][KK];
    float off[QH];
#pragma unroll
    for (int qh = 0; qh < QH; ++qh) {
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        qv[qh][kk] = *reinterpret_cast<const pf_bf16x8_t*>(qt + 16 * Cfg::kslot(16 * qh + s, 4 * kk + g4));
      // exp2(x - max) / sum = exp2(x - (max + log2(sum))).
      const float2 st = lds_read_f2((const pf_lds_char_t*)(stl + 2 * (16 * qh + s)));
      off[qh] = st.x - __log2f(st.y);
    }
    pf_f32x4_t sacc[QH][4];
#pragma unroll
    for (int qh = 0; qh < QH; ++qh)
#pragma unroll
      for (int T = 0; T < 4; ++T) sacc[qh][T] = pf_f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int qh = 0; qh < QH; ++qh)
#pragma unroll
        for (int T = 0; T < 4; ++T)
          sacc[qh][T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[T][kk], qv[qh][kk], sacc[qh][T], 0, 0, 0);
#pragma unroll
    for (int qh = 0; qh < QH; ++qh) {
      const int i = kPfItemQ * it + 16 * qh + s;
      const int pos = sq.first + i;
      const bool valid = i < sq.qlen;
#pragma unroll
      for (int T = 0; T < 4; ++T) {
        if (full) {
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) acc[T][rr] += hw_exp2(fmaf(sacc[qh][T][rr], sc, -off[qh]));
        } else {
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int key = j0w + 16 * T + 4 * g4 + rr;
            const float p = hw_exp2(fmaf(sacc[qh][T][rr], sc, -off[qh]));
            acc[T][rr] += (valid && key <= pos && key < sq.n) ? p : 0.0f;
          }
        }
      }
    }
  }

  // Sum over the 16 query columns, then one add per key.
#pragma unroll
  for (int T = 0; T < 4; ++T) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      float v = acc[T][rr];
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      v += __shfl_xor(v, 8);
      acc[T][rr] = v;
    }
  }
  if (s == 0) {
    float* sb = a.score + sq.row0;
#pragma unroll
    for (int T = 0; T < 4; ++T) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int key = j0w + 16 * T + 4 * g4 + rr;
        if (key < sq.n) sb[key] += acc[T][rr];
      }
    }
  }
}

template <int D, int G>
lethe_status launch_prefill_dg(const PrefillArgs& a, hipStream_t s) {
  const long long segs = (long long)a.B * a.HK;
  const long long nq = (a.max_q + 31) / 32;
  const long long fwd_blocks = segs * nq * ((G + 3) / 4);
  const long long score_blocks = segs * ((a.max_kv + kPfKeysPerBlock - 1) / kPfKeysPerBlock);
  if (fwd_blocks > 0x7fffffffLL || score_blocks > 0x7fffffffLL) return LETHE_ERR_UNSUPPORTED;
  if (fwd_blocks > 0) {
    hipLaunchKernelGGL((prefill_fwd_kernel<D, G>), dim3((unsigned)fwd_blocks), dim3(kPfThreads), 0, s, a);
    if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  }
  if (score_blocks > 0 && fwd_blocks > 0) {
    hipLaunchKernelGGL((prefill_score_kernel<D, G>), dim3((unsigned)score_blocks), dim3(kPfThreads), 0, s, a);
    if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  }
  return LETHE_OK;
}

template <int D>
lethe_status launch_prefill_d(const PrefillArgs& a, int G, hipStream_t s) {
  switch (G) {
    case 1: return launch_prefill_dg<D, 1>(a, s);
    case 2: return launch_prefill_dg<D, 2>(a, s);
    case 3: return launch_prefill_dg<D, 3>(a, s);
    case 4: return launch_prefill_dg<D, 4>(a, s);
    case 5: return launch_prefill_dg<D, 5>(a, s);
    case 6: return launch_prefill_dg<D, 6>(a, s);
    case 7: return launch_prefill_dg<D, 7>(a, s);
    case 8: return launch_prefill_dg<D, 8>(a, s);
    default: return LETHE_ERR_UNSUPPORTED;
  }
}

}  // namespace

lethe_status launch_prefill(const PrefillArgs& a, int D, int G, hipStream_t s) {
  if (D == 128) return launch_prefill_d<128>(a, G, s);
  if (D == 64) return launch_prefill_d<64>(a, G, s);
  return LETHE_ERR_UNSUPPORTED;
}

}  // namespace lethe
