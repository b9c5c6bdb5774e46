// Decode attention fused with the RASR importance update (Eq. 5), gfx950.
//
// One launch handles one layer for every sequence.  Each (sequence, KV head)
// segment gets chunks in proportion to its length (split-K flash decoding),
// one block each; the lengths come from the layer's tiling hints in the
// decode state, so every block derives the same map itself (no plan kernel,
// no length on the host).  The cached rows of a segment are cut into 32-row
// steps that the segment's wavefronts take from a per-segment counter, so a
// block that the memory system serves faster simply takes more steps.
//
// Per wavefront and step (bf16 storage):
//  - S^T = K Q^T on the matrix cores (v_mfma_f32_16x16x32_bf16: 16 rows x
//    the group's G query heads padded to 16; K rows load straight into the
//    operand layout).  Online softmax in base 2, one head per lane.
//  - O^T = V^T P^T: the step's V rows reach the wavefront's LDS tile by
//    direct loads and are read back transposed (ds_read_b64_tr_b16); P is
//    split into bf16 high and low parts (two MFMAs) so the products keep
//    fp32-level accuracy.
//  - The next step's K rows are requested as soon as this step's K has gone
//    through the MFMAs, its V once this step's V^T reads have completed.
// fp32 storage takes a VALU path with the same outputs.
//
// Eq. 5 runs one call late: the score update of a step needs the step's final
// max and sum per head, known only once every block is done.  The call keeps
// its query, scale and per-head (M, 1/L); the next call on the layer
// recomputes that step's logits from the K rows it loads anyway (one more
// MFMA chain, Q_prev K^T) and applies s <- gamma s + sum_g exp2(x_g - M_g) / L_g
// to those rows.  launch_flush applies a pending step on its own.  A settling
// call (the step before a prune round) also stores its raw logits per row and
// leaves nothing pending; settle_kernel then applies its update with the same
// arithmetic.
//
// Every block bumps its sequence's counter once all its wavefronts are past
// their last use of len and the pending state; the block that finishes a
// segment publishes the new length and pending step when the count is full
// (nobody of this launch reads them afterwards).  With one block per segment the block writes out and the
// step's (M, 1/L) itself.  Otherwise each block's (m, l, o) partial goes to
// the workspace with write-through stores, then the block bumps its segment's
// counter; the last block of a segment combines the partials.  Counters go
// back to zero.
#include <math.h>
#include <stdlib.h>

#include <atomic>

#include "device_common.h"
#include "lethe_internal.h"

namespace lethe {

namespace {

constexpr int kThreads = 256;
constexpr int kNumWaves = kThreads / kWave;
constexpr long long kFlushBlocks = 2048;  // grid of a flush launch, at most
constexpr float kNegBig = -1.0e30f;  // running-max start: finite, below any logit

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
typedef __attribute__((address_space(3))) char lds_char_t;
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void global_cvoid_t;

// Write-through store and coherent load of two floats exchanged between the
// blocks of one launch (relaxed, agent scope: no cache maintenance, no
// ordering; p is 8-byte aligned).
__device__ inline void st_agent2(float* p, float x, float y) {
  const uint64_t v = (uint64_t)__float_as_uint(x) | ((uint64_t)__float_as_uint(y) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float2 ld_agent2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

// What one block works on.
struct Chunk {
  int b, h, seg, c;
  int ncache;        // rows already in the cache (read by this call)
  int dst_app;       // where the appended row goes (ncache, or the rows kept)
  bool app;          // a row is appended to this sequence
  long long segrow0; // first row of the segment in the layer
  int32_t* next;     // the segment's step counter
  int first, stride; // wave w's first step is first + w; then first + w + stride, ...
                     // (stride 0: from the counter, whose n-th reply is step dyn_base + n)
  int dyn_base;
  int t0;            // compacting call: first step holding an evicted row
  int step0;         // compacting call: index of step 0 in the plan's step arrays
};

// Compacting call: waits until the plan steps [lo, hi] (absolute indices)
// have been read, one lane per step; `ready` (bit k: step spec0 + k was seen
// read already) spares the polls of steps known to be done.  Every lane polls
// at most spin_limit times over the call; past that the call gives up
// waiting and reports LETHE_DEV_WAIT_TIMEOUT.
__device__ inline void wait_steps(const DecodeArgs& a, int lo, int hi, int spec0, uint32_t ready, int& spins) {
  const int lane = threadIdx.x & (kWave - 1);
  const int t = lo + lane;
  const int k = t - spec0;
  bool wait = t <= hi && !(k >= 0 && k < 32 && ((ready >> k) & 1u));
  while (wait) {
    wait = __hip_atomic_load(&a.step_flag[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0;
    if (wait) {
      if (++spins > a.spin_limit) {
        atomicOr(a.dev_status, LETHE_DEV_WAIT_TIMEOUT);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  // The stores that follow stay after the wait.
  asm volatile("" ::: "memory");
}

// A wavefront's steps after its first (which is fixed, so its loads need no
// round trip): from the segment's counter (whichever wave asks first), or
// from the fixed schedule.  step_request issues the request (the counter's
// reply lands in lane 0 of the returned register); step_index reads it when
// it is needed, so the atomic's latency overlaps other work.  Every step
// below the segment's count is held by one wave and each holder asks once
// more, so exactly one wave receives the index equal to the count.
__device__ inline int step_request(const Chunk& ck, int& fixed_next, int lane) {
  if (ck.stride) {
    const int v = fixed_next;
    fixed_next += ck.stride;
    return v;
  }
  int v = 0;
  if (lane == 0) v = ck.dyn_base + __hip_atomic_fetch_add(ck.next, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return v;
}
__device__ inline int step_index(int raw) { return __builtin_amdgcn_readfirstlane(raw); }

// The pending step of a segment: rows [0, rows) get
//   s <- gamma s + sum_g exp2(scale * q_g . k - M_g) * invL_g
// with q the step's queries (qprev half `par`) and (M, invL) from segstat.
template <int G>
struct Pending {
  float* score;         // segment base
  const float* stat;    // M[G], then invL[G]
  const void* q;        // [G][D] storage type
  int rows;
  float gamma;
  float scale;          // softmax scale * log2(e) of that step
};

// ---------------------------------------------------------------------------
// Cross-wave combine of per-wave softmax states and the chunk partial.
// ---------------------------------------------------------------------------
struct CombineLds {
  float m[kNumWaves][8];
  float l[kNumWaves][8];
  float o[kNumWaves][8][128];
};

// The block's partial: per head m, l, then o[D] (pairs of floats).
template <int D, int G>
__device__ void write_partial(const CombineLds& cb, float* part) {
  __syncthreads();
  for (int i = threadIdx.x; i < G * D / 2; i += kThreads) {
    const int g = (2 * i) / D, d = (2 * i) % D;
    float mx = kNegBig;
#pragma unroll
    for (int k = 0; k < kNumWaves; ++k) mx = fmaxf(mx, cb.m[k][g]);
    float lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
    for (int k = 0; k < kNumWaves; ++k) {
      const float f = hw_exp2(cb.m[k][g] - mx);
      lsum += cb.l[k][g] * f;
      o0 += cb.o[k][g][d] * f;
      o1 += cb.o[k][g][d + 1] * f;
    }
    float* pg = part + g * (D + 2);
    st_agent2(pg + 2 + d, o0, o1);
    if (d == 0) st_agent2(pg, mx, lsum);
  }
}

// A segment in one chunk: out and (M, 1/L) per head straight from the
// per-wave states (the same arithmetic as a one-chunk combine).
template <int D, int G>
__device__ void finish_single(const DecodeArgs& a, const Chunk& ck, const CombineLds& cb) {
  __syncthreads();
  float* stat = a.segstat + (long long)ck.seg * 2 * G;
  float* outb = a.out + ((long long)ck.b * a.HK * G + (long long)ck.h * G) * D;
  for (int i = threadIdx.x; i < G * D / 2; i += kThreads) {
    const int g = (2 * i) / D, d = (2 * i) % D;
    float mx = kNegBig;
#pragma unroll
    for (int k = 0; k < kNumWaves; ++k) mx = fmaxf(mx, cb.m[k][g]);
    float lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
    for (int k = 0; k < kNumWaves; ++k) {
      const float f = hw_exp2(cb.m[k][g] - mx);
      lsum += cb.l[k][g] * f;
      o0 += cb.o[k][g][d] * f;
      o1 += cb.o[k][g][d + 1] * f;
    }
    const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;  // no row attended: out = 0
    *reinterpret_cast<float2*>(outb + g * D + d) = make_float2(o0 * inv, o1 * inv);
    if (d == 0) {
      stat[g] = mx;
      stat[G + g] = inv;
    }
  }
}

// Last block of a segment: out and (M, 1/L) per head from the nne partials,
// merged in batches of up to 16 chunks with online rescaling.
template <int D, int G>
__device__ void combine_segment(const DecodeArgs& a, const Chunk& ck, const float* part, int nne) {
  constexpr int NB = 16;
  const int ps = part_stride(G, D);
  float* stat = a.segstat + (long long)ck.seg * 2 * G;
  float* outb = a.out + ((long long)ck.b * a.HK * G + (long long)ck.h * G) * D;
  for (int i = threadIdx.x; i < G * D / 2; i += kThreads) {
    const int g = (2 * i) / D, d = (2 * i) % D;
    const float* pg = part + g * (D + 2);
    float M = kNegBig, lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
    for (int c0 = 0; c0 < nne; c0 += NB) {
      float2 ml[NB], ov[NB];
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const int cc = min(c0 + k, nne - 1);
        ml[k] = ld_agent2(pg + (long long)cc * ps);
        ov[k] = ld_agent2(pg + (long long)cc * ps + 2 + d);
      }
      float bm = M;
#pragma unroll
      for (int k = 0; k < NB; ++k) bm = (c0 + k < nne) ? fmaxf(bm, ml[k].x) : bm;
      const float f = hw_exp2(M - bm);
      lsum *= f;
      o0 *= f;
      o1 *= f;
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const float wgt = (c0 + k < nne) ? hw_exp2(ml[k].x - bm) : 0.0f;
        lsum = fmaf(ml[k].y, wgt, lsum);
        o0 = fmaf(ov[k].x, wgt, o0);
        o1 = fmaf(ov[k].y, wgt, o1);
      }
      M = bm;
    }
    const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;  // no row attended: out = 0
    *reinterpret_cast<float2*>(outb + g * D + d) = make_float2(o0 * inv, o1 * inv);
    if (d == 0) {
      stat[g] = M;
      stat[G + g] = inv;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 path on the matrix cores
// ---------------------------------------------------------------------------
// V rows reach LDS by direct loads (global_load_lds_dwordx4: lane l's 16
// bytes land at base + 16 l).  Load u of a step carries rows u + VLOADS j
// (j < RPL, LPR lanes per row) into block u; blocks are 1 KB plus 32 bytes
// of padding, so the four rows one 16-lane group reads together in the
// transposing read sit 8 banks apart.
template <int D>
struct MfmaCfg {
  static constexpr int KK = D / 32;          // k-steps of 32 over the head dim
  static constexpr int NT = D / 16;          // output tiles of 16 dims
  static constexpr int ROWB = D * 2;         // bytes per row
  static constexpr int STEP = 32;            // rows per wavefront step
  static constexpr int LPR = ROWB / 16;      // lanes per row for V loads
  static constexpr int RPL = kWave / LPR;    // rows per V load
  static constexpr int VLOADS = STEP / RPL;  // loads (LDS blocks) per step
  static constexpr int VBLK = kWave * 16 + 32;
  static constexpr int TILE_BYTES = VLOADS * VBLK;
  // LDS byte offset of row r (of the step), byte c of the row
  static __device__ constexpr int vaddr(int r, int c) { return (r % VLOADS) * VBLK + (r / VLOADS) * ROWB + c; }
};

__device__ inline bf16x8_t zero_bf16x8() {
  bf16x8_t z;
#pragma unroll
  for (int j = 0; j < 8; ++j) z[j] = (__bf16)0.0f;
  return z;
}

// A query group [G][D] (bf16, global memory) as the 16 x D MFMA operand,
// heads past G zero: lane holds Q[head s][32 kk + 8 g4 .. +8].  Serves as B
// of S^T = K Q^T and as A of S = Q K^T.
template <int D, int G>
__device__ inline bf16x8_t q_operand(const char* qgroup, int s, int g4, int kk) {
  return (s < G) ? *reinterpret_cast<const bf16x8_t*>(qgroup + (long long)s * D * 2 + 64 * kk + 16 * g4)
                 : zero_bf16x8();
}

template <int D, int G, bool kCompact, class ReadPending>
__device__ void attn_chunk_mfma(const DecodeArgs& a, const Chunk& ck, const ReadPending& read_pending,
                                char* vtiles, CombineLds& cb) {
  using Cfg = MfmaCfg<D>;
  constexpr int KK = Cfg::KK, NT = Cfg::NT, ROWB = Cfg::ROWB;
  constexpr int STEP = Cfg::STEP, LPR = Cfg::LPR, VLOADS = Cfg::VLOADS;
  static_assert(G <= 8, "pending heads live in lane groups 0 and 1");
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int g4 = lane >> 4;  // lane group: rows 4*g4.. of a 16-row tile
  const int s = lane & 15;   // query head (C/B layouts) or row (A layout)
  const int HQ = a.HK * G;
  char* vb = vtiles + w * Cfg::TILE_BYTES;

  const int re = ck.ncache;
  const int nsteps = (re + STEP - 1) / STEP;
  const char* Kb = reinterpret_cast<const char*>(a.k) + ck.segrow0 * ROWB;
  const char* Vb = reinterpret_cast<const char*>(a.v) + ck.segrow0 * ROWB;
  float* const sseg = a.score + ck.segrow0;
  // Settling call: this step's S = Q K^T per row, in the orientation and
  // arithmetic of the deferred update.
  float* const xlog = (!kCompact && a.logit) ? a.logit + ck.segrow0 * kLogitStride : nullptr;

  // Loads of a step: K rows into the operand registers and the old scores of
  // rows base + 16 g4 + s (lane groups 0 and 1, used if the pending update
  // covers them); V rows straight into the wave's LDS tile.  The next step's
  // K and scores are requested as soon as this step's K has gone through the
  // MFMAs, and its V as soon as this step's V^T reads have completed, so the
  // loads of one step overlap the softmax and PV work of the previous one.
  // The first step is fixed, so its loads leave before anything else is read.
  bf16x8_t kr[2][KK];
  float sold = 0.0f;
  // Compacting call, steps from t0 on (those holding rows that move): the
  // plan entry of the step (rows kept before it, keep mask of its rows), and
  // a first look at the flags of the 8 steps before it (bit k: step t - 8 + k
  // was seen read; steps before t0 never move and count as read).  Both are
  // wave-uniform and come through the scalar cache, whose loads are counted
  // apart from the vector memory operations: waiting for them never waits
  // for the step's K and V loads or for earlier stores.  The plan does not
  // change during the call; a flag only ever goes from 0 to 1 during it, so
  // a stale scalar-cache copy can only under-report, which costs a poll in
  // wait_steps and nothing else.
  int npre = 0;
  uint32_t nmask = ~0u;
  uint32_t nready = 0xffu;
  auto load_k = [&](int bs) {
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      const int row = min(bs + 16 * T + s, re - 1);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kr[T][kk] = *reinterpret_cast<const bf16x8_t*>(Kb + (long long)row * ROWB + 64 * kk + 16 * g4);
    }
    sold = g4 < 2 ? sseg[min(bs + 16 * g4 + s, re - 1)] : 0.0f;
    if constexpr (kCompact) {
      const int t = __builtin_amdgcn_readfirstlane(bs / STEP);
      if (t >= ck.t0) {
        typedef __attribute__((address_space(4))) const int32_t cint_t;
        const cint_t* sp = (const cint_t*)(a.step_plan + 2 * ((long long)ck.step0 + t));
        npre = sp[0];
        nmask = (uint32_t)sp[1];
        const cint_t* fl = (const cint_t*)(a.step_flag + ck.step0 + (t - 8));
        nready = 0;
        if (t - 8 >= ck.t0) {
#pragma unroll
          for (int k = 0; k < 8; ++k) nready |= (fl[k] != 0 ? 1u : 0u) << k;
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k)
            if (t - 8 + k < ck.t0 || fl[k] != 0) nready |= 1u << k;
        }
      }
    }
  };
  // V lines are read whole, once per call, so their loads carry the
  // non-temporal policy (the `nt` bit): they leave L2 early, and the K lines
  // (whose two 64-byte halves come from two loads) and the call's small
  // shared data stay.  K loads keep the default policy.
  constexpr int kVLoadPolicy = 2;  // nt
  auto load_v = [&](int bs) {
#pragma unroll
    for (int u = 0; u < VLOADS; ++u) {
      const int row = min(bs + u + VLOADS * (lane / LPR), re - 1);
      __builtin_amdgcn_global_load_lds((global_cvoid_t*)(Vb + (long long)row * ROWB + 16 * (lane % LPR)),
                                       (lds_void_t*)((lds_char_t*)vb + u * Cfg::VBLK), 16, 0, kVLoadPolicy);
    }
  };
  int fixed_next = ck.first + w + ck.stride;
  // A wave's first step is fixed, except in a compacting call where that
  // step would hold rows that move: every such step comes from the counter,
  // in row order, so a wave waits only for steps claimed before its own, by
  // running waves.
  int idx = ck.first + w;
  if (kCompact && idx >= ck.dyn_base) idx = step_index(step_request(ck, fixed_next, lane));
  if (idx < nsteps) {
    load_k(idx * STEP);
    load_v(idx * STEP);
  }
  int spins = 0;  // flag polls of this lane (compacting call)

  const Pending<G> pd = read_pending();
  const int pre_end = min(pd.rows, re);
  // Both query sets live in registers; so do the pending step's statistics
  // of the heads 4 g4 + rr this lane holds in S = Q_prev K^T.
  const char* qcur = reinterpret_cast<const char*>(a.q) + ((long long)ck.b * HQ + (long long)ck.h * G) * D * 2;
  bf16x8_t qb[KK], qo[KK];
  float pm[4], pi[4];
  const bool any_pending = pre_end > 0;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    qb[kk] = q_operand<D, G>(qcur, s, g4, kk);
    qo[kk] = any_pending ? q_operand<D, G>(reinterpret_cast<const char*>(pd.q), s, g4, kk) : zero_bf16x8();
  }
#pragma unroll
  for (int rr = 0; rr < 4; ++rr) {
    const int hh = 4 * g4 + rr;
    pm[rr] = (any_pending && hh < G) ? pd.stat[hh] : 0.0f;
    pi[rr] = (any_pending && hh < G) ? pd.stat[G + hh] : 0.0f;
  }

  float m = kNegBig, l = 0.0f;
  f32x4_t o[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) o[nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  const float sc = a.scale_log2;

  // One 32-row step whose K is in kr, its V in the wave's LDS tile and its
  // old scores in sold.  `moving` (compacting call, steps from t0 on): only
  // the rows of `cmask` take part, and the kept rows go to rows cpre, cpre +
  // 1, ... of the segment once the steps holding those rows have been read
  // (cready: which of the 8 steps before this one were seen read already).
  // after_k runs once kr is free, after_v once the V tile is.
  auto step = [&](int base, bool moving, int cpre, uint32_t cmask, uint32_t cready, auto&& after_k,
                  auto&& after_v) {
    const bool pstep = base < pre_end;
    const int prow = base + 16 * g4 + s;
    const bool pon = pstep && g4 < 2 && prow < pre_end;
    f32x4_t sacc[2];
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      sacc[T] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) sacc[T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[T][kk], qb[kk], sacc[T], 0, 0, 0);
    }
    if (xlog) {
      // Lane (g4 < 2, s): heads 4 g4 .. 4 g4 + 3 of row 16 T + s, one 16-byte store.
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        f32x4_t sx = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) sx = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qb[kk], kr[T][kk], sx, 0, 0, 0);
        const int row = base + 16 * T + s;
        if (g4 < 2 && row < re) *reinterpret_cast<f32x4_t*>(xlog + (long long)row * kLogitStride + 4 * g4) = sx;
      }
    }
    float pval = 0.0f;  // the row's score after the pending update (pon)
    if (pstep) {
      // S = Q_prev K^T: lane (g4, s) gets heads 4 g4 + rr of row 16 T + s.
      float part[2];
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        f32x4_t so = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          so = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qo[kk], kr[T][kk], so, 0, 0, 0);
        float acc = 0.0f;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) acc = fmaf(hw_exp2(fmaf(so[rr], pd.scale, -pm[rr])), pi[rr], acc);
        part[T] = acc + __shfl_xor(acc, 16);
      }
      pval = fmaf(pd.gamma, sold, g4 == 0 ? part[0] : part[1]);
      if (pon && !moving) pd.score[prow] = pval;
    }
    if constexpr (kCompact) {
      if (moving) {
        // The kept rows go to rows cpre .. cpre + kept - 1: the earlier steps
        // holding those rows must have been read.
        const int kc = __popc(cmask);
        const int t = base / STEP;
        if (kc > 0) {
          const int lo = max(cpre / STEP, ck.t0), hi = min((cpre + kc - 1) / STEP, t - 1);
          if (lo <= hi) wait_steps(a, ck.step0 + lo, ck.step0 + hi, ck.step0 + t - 8, cready, spins);
        }
        // Kept rows to their places: K from the operand registers (lane
        // (g4, s) holds bytes 64 kk + 16 g4 of row 16 T + s), V from the LDS
        // tile (16 bytes a lane), scores with the pending update where due.
        char* Kw = reinterpret_cast<char*>(a.k_w) + ck.segrow0 * ROWB;
        char* Vw = reinterpret_cast<char*>(a.v_w) + ck.segrow0 * ROWB;
        auto dst_of = [&](int r) { return cpre + __popc(cmask & ((1u << r) - 1u)); };
#pragma unroll
        for (int T = 0; T < 2; ++T) {
          const int r = 16 * T + s;
          const int dst = dst_of(r);
          if (((cmask >> r) & 1u) && dst != base + r && dst < ck.dst_app) {
#pragma unroll
            for (int kk = 0; kk < KK; ++kk)
              *reinterpret_cast<bf16x8_t*>(Kw + (long long)dst * ROWB + 64 * kk + 16 * g4) = kr[T][kk];
          }
        }
        constexpr int CPR = ROWB / 16;    // 16-byte pieces per row
        constexpr int RPP = kWave / CPR;  // rows per pass
        const int piece = lane % CPR;
#pragma unroll 1
        for (int i = 0; i < STEP / RPP; ++i) {
          const int r = lane / CPR + RPP * i;
          const int dst = dst_of(r);
          if (((cmask >> r) & 1u) && dst != base + r && dst < ck.dst_app) {
            typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
            typedef __attribute__((address_space(3))) const u32x4_t lds_u32x4_t;
            const u32x4_t v = *reinterpret_cast<lds_u32x4_t*>((lds_char_t*)vb + Cfg::vaddr(r, 16 * piece));
            *reinterpret_cast<u32x4_t*>(Vw + (long long)dst * ROWB + 16 * piece) = v;
          }
        }
        if (g4 < 2) {
          const int r = 16 * g4 + s;
          const int dst = dst_of(r);
          if (((cmask >> r) & 1u) && (dst != prow || pon) && dst < ck.dst_app) sseg[dst] = pon ? pval : sold;
        }
      }
    }
    after_k();

    // Logits of rows base + 16 T + 4 g4 + rr for head s.
    float x[2][4];
    float mx = kNegBig;
#pragma unroll
    for (int T = 0; T < 2; ++T) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int row = base + 16 * T + 4 * g4 + rr;
        const bool live = row < re && (!kCompact || !moving || ((cmask >> (16 * T + 4 * g4 + rr)) & 1u));
        x[T][rr] = live ? sacc[T][rr] * sc : -INFINITY;
        mx = fmaxf(mx, x[T][rr]);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx);
    const float corr = hw_exp2(m - mnew);
    float psum = 0.0f;
    bf16x8_t ph, pl;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = hw_exp2(x[j >> 2][j & 3] - mnew);
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
      const bf16x4_t a0 =
          __builtin_amdgcn_ds_read_tr16_b64_v4bf16(reinterpret_cast<lds_bf16x4_t*>(vbl + Cfg::vaddr(rsub, col)));
      const bf16x4_t a1 =
          __builtin_amdgcn_ds_read_tr16_b64_v4bf16(reinterpret_cast<lds_bf16x4_t*>(vbl + Cfg::vaddr(rsub + 16, col)));
      const bf16x8_t av = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
      o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, ph, o[nt], 0, 0, 0);
      o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pl, o[nt], 0, 0, 0);
    }
    after_v();
  };

  int nidx = nsteps + 1;
  int graw = idx < nsteps ? step_request(ck, fixed_next, lane) : 0;
  while (idx < nsteps) {
    const int base = idx * STEP;
    nidx = step_index(graw);
    const bool more = nidx < nsteps;  // wave-uniform
    const bool moving = kCompact && idx >= ck.t0;
    uint32_t cready = 0;
    if constexpr (kCompact) {
      if (moving) {
        // Every load of this step has arrived (the reply to the claim above
        // came after them): its rows may now be overwritten.
        __builtin_amdgcn_s_waitcnt(0);
        asm volatile("" ::: "memory");
        if (lane == 0) __hip_atomic_store(&a.step_flag[ck.step0 + idx], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        cready = nready;
      }
    }
    step(base, moving, npre, nmask, cready, [&]() {
      if (more) load_k(nidx * STEP);
    }, [&]() {
      if (more) {
        load_v(nidx * STEP);
        graw = step_request(ck, fixed_next, lane);
      }
    });
    idx = nidx;
  }

  // The appended row, by the wave that drew the step index equal to the
  // step count: read from k_new / v_new, copied into the cache, its score
  // started at 0, and folded into the wave's state.
  if (ck.app && idx == nsteps) {
    const char* kn = reinterpret_cast<const char*>(a.k_new) + (((long long)ck.b * a.HK + ck.h) * D) * 2;
    const char* vn = reinterpret_cast<const char*>(a.v_new) + (((long long)ck.b * a.HK + ck.h) * D) * 2;
    if constexpr (kCompact) {
      // The new row's place held an old row until this call read it.
      if (ck.dst_app < re) {
        const int t = ck.dst_app / STEP;
        wait_steps(a, ck.step0 + t, ck.step0 + t, 0, 0u, spins);
      }
    }
    if (lane < LPR) {
      *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.k_w) + (ck.segrow0 + ck.dst_app) * ROWB + 16 * lane) =
          *reinterpret_cast<const uint4*>(kn + 16 * lane);
      *reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.v_w) + (ck.segrow0 + ck.dst_app) * ROWB + 16 * lane) =
          *reinterpret_cast<const uint4*>(vn + 16 * lane);
    }
    if (lane == 0) pd.score[ck.dst_app] = 0.0f;
    if (xlog) {
      // The appended row's logits as a cached row would give them: every
      // column of the B operand is k_new.
      f32x4_t sx = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        sx = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qb[kk], *reinterpret_cast<const bf16x8_t*>(kn + 64 * kk + 16 * g4),
                                                     sx, 0, 0, 0);
      if (g4 < 2 && s == 0) *reinterpret_cast<f32x4_t*>(xlog + (long long)ck.ncache * kLogitStride + 4 * g4) = sx;
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
    const float mnew = fmaxf(m, x);
    const float corr = hw_exp2(m - mnew);
    const float p = hw_exp2(x - mnew);
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
}

// ---------------------------------------------------------------------------
// fp32 path (VALU): 16-byte loads, D/4 lanes per row.
// ---------------------------------------------------------------------------
template <int D, int G, class ReadPending>
__device__ void attn_chunk_f32(const DecodeArgs& a, const Chunk& ck, const ReadPending& read_pending,
                               CombineLds& cb) {
  constexpr int EPL = 4;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  constexpr int U = 4;
  constexpr int ROWS_WAVE = U * RPW;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = tid / kWave;
  const int rg = lane / LPR;
  const int dp = lane % LPR;
  const int HQ = a.HK * G;
  const Pending<G> pd = read_pending();

  // Queries pre-scaled by their step's scale, so both logit sums below are
  // formed the same way.
  float qf[G][EPL], qof[G][EPL];
  {
    const float* qb = reinterpret_cast<const float*>(a.q) + ((long long)ck.b * HQ + (long long)ck.h * G) * D + dp * EPL;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint4 r = *reinterpret_cast<const uint4*>(qb + (long long)g * D);
      qf[g][0] = __uint_as_float(r.x) * a.scale_log2;
      qf[g][1] = __uint_as_float(r.y) * a.scale_log2;
      qf[g][2] = __uint_as_float(r.z) * a.scale_log2;
      qf[g][3] = __uint_as_float(r.w) * a.scale_log2;
    }
  }
  const int re = ck.ncache;
  const int pre_end = min(pd.rows, re);
  const int nsteps = (re + ROWS_WAVE - 1) / ROWS_WAVE;
  float pM[G], pI[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    pM[g] = 0.0f;
    pI[g] = 0.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) qof[g][e] = 0.0f;
  }
  if (pre_end > 0) {
    const float* qp = reinterpret_cast<const float*>(pd.q) + dp * EPL;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint4 r = *reinterpret_cast<const uint4*>(qp + (long long)g * D);
      qof[g][0] = __uint_as_float(r.x) * pd.scale;
      qof[g][1] = __uint_as_float(r.y) * pd.scale;
      qof[g][2] = __uint_as_float(r.z) * pd.scale;
      qof[g][3] = __uint_as_float(r.w) * pd.scale;
      pM[g] = pd.stat[g];
      pI[g] = pd.stat[G + g];
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
  const float* Kb = reinterpret_cast<const float*>(a.k) + ck.segrow0 * D + dp * EPL;
  const float* Vb = reinterpret_cast<const float*>(a.v) + ck.segrow0 * D + dp * EPL;
  float* const xlog = a.logit ? a.logit + ck.segrow0 * kLogitStride : nullptr;

  auto consume = [&](const uint4* kr, const uint4* vr, const bool* valid, bool pstep, const int* row,
                     const float* sold) {
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
        const float xs = group_sum<LPR>(acc);  // every lane takes part
        x[u][g] = valid[u] ? xs : -INFINITY;
        if (xlog && dp == 0 && valid[u]) xlog[(long long)row[u] * kLogitStride + g] = xs;
      }
      if (pstep) {
        float c = 0.0f;
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float acc = 0.0f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc = fmaf(qof[g][e], kf[e], acc);
          const float xs = group_sum<LPR>(acc);
          c = fmaf(hw_exp2(xs - pM[g]), pI[g], c);
        }
        if (dp == 0 && row[u] < pre_end) pd.score[row[u]] = fmaf(pd.gamma, sold[u], c);
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = m[g];
#pragma unroll
      for (int u = 0; u < U; ++u) mx = fmaxf(mx, x[u][g]);
      const float corr = hw_exp2(m[g] - mx);
      float lg = l[g] * corr;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] *= corr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = hw_exp2(x[u][g] - mx);
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

  int fixed_next = ck.first + w + ck.stride;
  auto grab = [&]() { return step_index(step_request(ck, fixed_next, lane)); };
  int idx = ck.first + w;
  for (; idx < nsteps; idx = grab()) {
    const int base = idx * ROWS_WAVE;
    uint4 kr[U], vr[U];
    int row[U];
    bool valid[U];
    float sold[U];
    const bool pstep = base < pre_end;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      row[u] = base + u * RPW + rg;
      valid[u] = row[u] < re;
      const int rr = valid[u] ? row[u] : (re - 1);
      kr[u] = *reinterpret_cast<const uint4*>(Kb + (long long)rr * D);
      vr[u] = *reinterpret_cast<const uint4*>(Vb + (long long)rr * D);
      sold[u] = (pstep && dp == 0 && row[u] < pre_end) ? pd.score[row[u]] : 0.0f;
    }
    consume(kr, vr, valid, pstep, row, sold);
  }
  if (ck.app && idx == nsteps) {
    const long long nb = ((long long)ck.b * a.HK + ck.h) * D + dp * EPL;
    uint4 kr[U], vr[U];
    int row[U];
    bool valid[U];
    float sold[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      row[u] = ck.ncache;
      valid[u] = (u == 0) && (rg == 0);
      sold[u] = 0.0f;
      kr[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(a.k_new) + nb);
      vr[u] = *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(a.v_new) + nb);
    }
    if (rg == 0) {
      *reinterpret_cast<uint4*>(reinterpret_cast<float*>(a.k_w) + (ck.segrow0 + ck.ncache) * D + dp * EPL) = kr[0];
      *reinterpret_cast<uint4*>(reinterpret_cast<float*>(a.v_w) + (ck.segrow0 + ck.ncache) * D + dp * EPL) = vr[0];
    }
    if (lane == 0) pd.score[ck.ncache] = 0.0f;
    consume(kr, vr, valid, false, row, sold);
  }
#pragma unroll
  for (int off = LPR; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float mo = __shfl_xor(m[g], off);
      const float lo = __shfl_xor(l[g], off);
      const float mx = fmaxf(m[g], mo);
      const float fa = hw_exp2(m[g] - mx);
      const float fb = hw_exp2(mo - mx);
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
}

// ---------------------------------------------------------------------------
// Kernel
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

// ---------------------------------------------------------------------------
// Tiling: which chunk of which segment a block works on
// ---------------------------------------------------------------------------
// The launch splits every segment into chunks of about the same number of
// 32-row steps, so that sequences of very different lengths end together.
// The split follows the layer's tiling hints (lengths in the decode state,
// written by flush and compaction only, so every block of a launch reads the
// same values): with S the hinted steps of all segments and nb the chunks
// the call aims for (S / steps_per_chunk between min(min_chunks, nbt) and
// nbt, or nbt itself when the target is fixed), a segment of w hinted steps
// gets nch = clamp(ceil(w / ceil(S / nb)), 1, kMaxChunksPerSeg) chunks, one
// block each.  The blocks of sequence b are consecutive, KV head by KV head:
// block P_b + h nch_b + c is chunk c of segment (b, h).  When every hint is 0
// each segment gets nch_flat chunks.  A hint only shapes the split: every
// chunk count covers the segment's actual rows.  Blocks past the last chunk
// have nothing to do.
struct SeqWords {
  int n, cp;           // len and cap
  long long sbase;     // seq_base
  int pend_len, pend_par;
  float pend_gamma, pend_scale;
};

struct BlockPlan {
  int b = 0, nch = 1, first = 0;  // sequence, its chunks per segment, its first block
  bool valid = false;             // the block has a chunk
};

// Inclusive prefix sum over the 64 lanes of a wavefront (DPP row shifts,
// then the row broadcasts of lanes 15 and 31).
__device__ inline int wave_incl_scan_i32(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// Hinted steps are capped so that their sum over 1024 sequences stays an int.
constexpr int kMaxHintSteps = 1 << 20;

// The plan of block `blk` from R rows of 64 sequences (sequence 64 r + lane).
// With kWords the sequences' own words come in the same round trip and the
// chosen one's are returned in `w` (R = 4 covers up to 256 sequences).
template <int R, bool kWords>
__device__ inline BlockPlan plan_block(const DecodeArgs& a, int blk, SeqWords& w) {
  const int lane = threadIdx.x & (kWave - 1);
  const int B = a.B;
  int hv[R];
  int wn[R], wc[R], wpl[R], wpp[R];
  long long wsb[R];
  float wpg[R], wps[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int bb = min(kWave * r + lane, B - 1);  // clamped: every load is issued
    hv[r] = a.hint[bb];
    if constexpr (kWords) {
      wn[r] = a.len[bb];
      wc[r] = a.cap[bb];
      wsb[r] = a.seq_base[bb];
      wpl[r] = a.pend_len[bb];
      wpp[r] = a.pend_par[bb];
      wpg[r] = a.pend_gamma[bb];
      wps[r] = a.pend_scale[bb];
    }
  }
  int stp[R];
  int sum = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const bool in = kWave * r + lane < B;
    stp[r] = (in && hv[r] > 0) ? min((hv[r] + 31) >> 5, kMaxHintSteps) : 0;
    sum += stp[r];
  }
  const long long total = (long long)__builtin_amdgcn_readlane(wave_incl_scan_i32(sum), kWave - 1) * a.HK;
  int spb = 0;  // steps per chunk; 0: flat split
  if (total > 0) {
    // Chunks of about steps_per_chunk hinted steps, between
    // min(min_chunks, nbt) and nbt chunks in all (nbt when the target is
    // fixed).
    long long nb = a.nbt;
    if (a.adaptive) nb = min(max(total / a.steps_per_chunk, (long long)min(a.min_chunks, a.nbt)), (long long)a.nbt);
    spb = (int)min((total + nb - 1) / nb, (long long)kMaxHintSteps);
  }
  BlockPlan p;
  int carry = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const bool in = kWave * r + lane < B;
    const int nch = spb > 0 ? min(max((stp[r] + spb - 1) / spb, 1), kMaxChunksPerSeg) : a.nch_flat;
    const int cnt = in ? a.HK * nch : 0;
    const int incl = wave_incl_scan_i32(cnt);
    const int ex = carry + incl - cnt;
    const unsigned long long hit = __ballot(cnt > 0 && blk >= ex && blk < ex + cnt);
    if (hit) {
      const int src = (int)__builtin_ctzll(hit);
      p.valid = true;
      p.b = kWave * r + src;
      p.nch = __builtin_amdgcn_readlane(nch, src);
      p.first = __builtin_amdgcn_readlane(ex, src);
      if constexpr (kWords) {
        w.n = __builtin_amdgcn_readlane(wn[r], src);
        w.cp = __builtin_amdgcn_readlane(wc[r], src);
        const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)wsb[r], src);
        const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((unsigned long long)wsb[r] >> 32), src);
        w.sbase = (long long)(((unsigned long long)hi << 32) | lo);
        w.pend_len = __builtin_amdgcn_readlane(wpl[r], src);
        w.pend_par = __builtin_amdgcn_readlane(wpp[r], src);
        w.pend_gamma = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wpg[r]), src));
        w.pend_scale = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wps[r]), src));
      }
    }
    carry += __builtin_amdgcn_readlane(incl, kWave - 1);
  }
  return p;
}

template <typename T, int D, int G, bool kCompact>
__device__ inline void decode_body(const DecodeArgs& a) {
  __shared__ __attribute__((aligned(16))) AttnLds<T, D> S;
  __shared__ int s_last;
  const int tid = threadIdx.x;
  const int blk = (int)blockIdx.x;
  const int HQ = a.HK * G;

  // Every wave plans alike (no barrier); with up to 256 sequences the chosen
  // sequence's words arrive with the hints (one round of 64 sequences up to
  // 64, two up to 128, four up to 256).
  SeqWords sw;
  BlockPlan bp;
  if (a.B <= kWave) {
    bp = plan_block<1, true>(a, blk, sw);
  } else if (a.B <= 2 * kWave) {
    bp = plan_block<2, true>(a, blk, sw);
  } else if (a.B <= 4 * kWave) {
    bp = plan_block<4, true>(a, blk, sw);
  } else {
    bp = plan_block<kMaxSeqs / kWave, false>(a, blk, sw);
    if (bp.valid) {
      const int bb = bp.b;
      sw.n = a.len[bb];
      sw.cp = a.cap[bb];
      sw.sbase = a.seq_base[bb];
      sw.pend_len = a.pend_len[bb];
      sw.pend_par = a.pend_par[bb];
      sw.pend_gamma = a.pend_gamma[bb];
      sw.pend_scale = a.pend_scale[bb];
    }
  }
  if (!bp.valid) return;
  const int b = bp.b;
  const int nch = bp.nch;
  const int o = blk - bp.first;
  const int h = o / nch;
  const int c = o - h * nch;
  const int seg = b * a.HK + h;
  const int seg_first = bp.first + h * nch;  // block (and partial) of chunk 0

  const int n = sw.n;
  const int cp = sw.cp;
  const long long sbase = sw.sbase;
  const bool app = a.k_new != nullptr;
  // Compacting call: the plan of this segment; the rows it keeps replace the
  // cached ones (a plan made for other lengths, or invalid, skips the
  // sequence as a bad layout would).
  int n_keep = n, t0 = 0, step0 = 0;
  bool plan_ok = true;
  if constexpr (kCompact) {
    const int32_t* sp = a.seg_plan + (long long)seg * kSegPlanWords;
    n_keep = sp[1];
    t0 = sp[2];
    step0 = sp[3];
    plan_ok = sp[0] == n && n_keep >= 0 && n_keep <= n && t0 >= 0 && t0 <= (n + 31) / 32 && step0 >= 0 &&
              (long long)step0 + (n + 31) / 32 <= a.plan_steps;
  }
  const bool bad = n < 0 || cp < 0 || n > cp || sbase < 0 || sbase + (long long)a.HK * cp > a.rows_per_layer ||
                   !plan_ok;
  const bool ovf = !bad && app && n_keep >= cp;
  const int n_att = (bad || ovf) ? 0 : n_keep + (app ? 1 : 0);
  const bool settle = a.logit != nullptr;
  // (A compacting call that keeps no row still publishes the new length.)
  if (n_att == 0 && (!kCompact || bad || ovf)) {
    // Skipped (flagged) or empty sequence: its out rows get NaN or 0, nothing
    // else of it changes, and no counter is touched.
    if (c == 0) {
      if (settle && h == 0 && tid == 0) a.apply_rows[b] = 0;
      const float fill = (bad || ovf) ? __int_as_float(0x7fc00000) : 0.0f;
      float* ob = a.out + ((long long)b * HQ + (long long)h * G) * D;
      for (int i = tid; i < G * D; i += kThreads) ob[i] = fill;
      if (h == 0 && tid == 0 && (bad || ovf))
        atomic_or_status(a.dev_status, bad ? LETHE_DEV_BAD_LAYOUT : LETHE_DEV_APPEND_OVERFLOW);
    }
    return;
  }
  const size_t qgroup = ((size_t)b * HQ + (size_t)h * G) * D * sizeof(T);  // bytes
  const size_t qhalf = (size_t)a.B * HQ * D * sizeof(T);

  Chunk ck;
  ck.b = b;
  ck.h = h;
  ck.seg = seg;
  ck.c = c;
  ck.next = &a.seg_cnt[(long long)seg * kCntStride + kStepCounter];
  ck.first = c * kNumWaves;  // wave w starts at step c * waves + w
  ck.stride = (a.deterministic && !kCompact) ? nch * kNumWaves : 0;
  // A compacting call fixes first steps only below t0 (rows that stay); the
  // counter hands out every step from there on.
  ck.dyn_base = kCompact ? min(nch * kNumWaves, t0) : nch * kNumWaves;
  ck.app = app;
  ck.ncache = n;
  ck.dst_app = n_keep;
  ck.t0 = t0;
  ck.step0 = step0;
  ck.segrow0 = sbase + (long long)h * cp;
  const int ps = part_stride(G, D);

  // The pending score step of this sequence (from the words read with the
  // plan).  Every block of the sequence counts itself once all its
  // wavefronts are done with len and the pending state: after the streaming
  // loop, whose closing barrier every wave passes only after its last use of
  // them.  A block that finishes a segment later reads the count: all of
  // them do so after every block of its segment has counted, so the last
  // segment to finish sees the full count and publishes the new length and
  // pending step; earlier finishers that also see it publish the same values.
  int32_t* seq_ctr = &a.seq_cnt[(long long)b * kCntStride];
  const int seq_full = a.HK * nch;
  const int par = sw.pend_par & 1;
  Pending<G> pd0;
  pd0.rows = sw.pend_len > 0 ? min(sw.pend_len, n) : 0;
  pd0.gamma = sw.pend_gamma;
  pd0.scale = sw.pend_scale;
  pd0.score = a.score + ck.segrow0;
  pd0.stat = a.segstat + (long long)seg * 2 * G;
  pd0.q = reinterpret_cast<const char*>(a.qprev) + par * qhalf + qgroup;
  auto read_pending = [&]() { return pd0; };
  auto publish = [&](int seen) {
    if (seen != seq_full) return;
    if (app || kCompact) a.len[b] = n_att;
    // A settling call leaves nothing pending: its second launch applies the
    // step to the n_att rows.
    a.pend_len[b] = settle ? 0 : n_att;
    if (settle) a.apply_rows[b] = n_att;
    a.pend_par[b] = par ^ 1;
    a.pend_gamma[b] = a.gamma;
    a.pend_scale[b] = a.scale_log2;
    __hip_atomic_store(seq_ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };

  {
    if constexpr (sizeof(T) == 2)
      attn_chunk_mfma<D, G, kCompact>(a, ck, read_pending, S.vtiles, S.cb);
    else
      attn_chunk_f32<D, G>(a, ck, read_pending, S.cb);
    // Both routines end with a barrier that every wave reaches after its
    // last use of len and of the pending state.
    if (tid == 0) __hip_atomic_fetch_add(seq_ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (c == 0) {
      // Keep this step's queries of the group for the next call's score update.
      const uint4* src = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(a.q) + qgroup);
      uint4* dst = reinterpret_cast<uint4*>(reinterpret_cast<char*>(a.qprev) + (par ^ 1) * qhalf + qgroup);
      for (int i = tid; i < (int)(G * D * sizeof(T) / 16); i += kThreads) dst[i] = src[i];
    }
    if (nch == 1) {
      int seen = 0;
      if (tid == 0) seen = __hip_atomic_load(seq_ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      finish_single<D, G>(a, ck, S.cb);
      if (tid == 0) {
        publish(seen);
        __hip_atomic_store(ck.next, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      return;
    }
    write_partial<D, G>(S.cb, a.part + (long long)blk * ps);
  }

  // Completion count of the segment: every block, with or without steps.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0)
    s_last = __hip_atomic_fetch_add(&a.seg_cnt[(long long)seg * kCntStride], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == nch - 1;
  __syncthreads();
  if (!s_last) return;
  int seen = 0;
  if (tid == 0) {
    __hip_atomic_store(&a.seg_cnt[(long long)seg * kCntStride], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(ck.next, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    seen = __hip_atomic_load(seq_ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  combine_segment<D, G>(a, ck, a.part + (long long)seg_first * ps, nch);
  if (tid == 0) publish(seen);
}

// bf16: three resident blocks per CU need at most 168 registers per lane.
template <int D, int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void decode_bf16_kernel(DecodeArgs a) {
  decode_body<bf16_t, D, G, false>(a);
}

// The compacting step (one call per layer and prune round): the same three
// resident blocks per CU.
template <int D, int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void decode_bf16_compact_kernel(
    DecodeArgs a) {
  decode_body<bf16_t, D, G, true>(a);
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void decode_f32_kernel(DecodeArgs a) {
  decode_body<float, D, G, false>(a);
}

template <typename T, int D, int G, bool kCompact>
constexpr auto decode_kernel() {
  if constexpr (sizeof(T) == 2 && kCompact)
    return decode_bf16_compact_kernel<D, G>;
  else if constexpr (sizeof(T) == 2)
    return decode_bf16_kernel<D, G>;
  else
    return decode_f32_kernel<D, G>;
}

// ---------------------------------------------------------------------------
// Flush: apply the pending step of every (layer, sequence), block per
// (layer, sequence, KV head); the last block of each (layer, sequence)
// clears its pending length.
// ---------------------------------------------------------------------------
// The segments of a flush block: a contiguous run of at most kThreads.
__device__ inline void flush_range(const FlushArgs& a, long long& i0, long long& n) {
  const long long nseg = (long long)a.L * a.B * a.HK;
  const long long per = (nseg + gridDim.x - 1) / gridDim.x;
  i0 = (long long)blockIdx.x * per;
  n = min(per, nseg - i0);
  if (n < 0) n = 0;
}

// One load round for all of a block's segments: thread t reads segment
// i0 + t's pending length into s_pend[t] and refreshes its (layer, sequence)'s
// tiling hint.  Every segment belongs to one block, which reads its pending
// length before it processes any segment, so the read always precedes the
// clearing by the last block of that (layer, sequence).
__device__ inline void flush_scan(const FlushArgs& a, long long i0, long long n, int* s_pend) {
  const int t = threadIdx.x;
  if (t < n) {
    const long long i = i0 + t;
    const int lb = a.l0 * a.B + (int)(i / a.HK);
    if (i % a.HK == 0) a.hint[lb] = a.len[lb];
    s_pend[t] = a.pend_len[lb];
  }
  __syncthreads();
}

// Every flush block of a (layer, sequence) with a pending step counts itself
// once all its threads are done with the pending state; the last of the H_KV
// blocks clears the pending length and the counter (which the decode state
// holds at zero between flushes).
__device__ inline void flush_done(const FlushArgs& a, int lb) {
  __syncthreads();
  if (threadIdx.x == 0 && atomicAdd(&a.flush_cnt[lb], 1) == a.HK - 1) {
    a.pend_len[lb] = 0;
    a.flush_cnt[lb] = 0;
  }
}

template <typename T, int D, int G>
__device__ void flush_segment_valu(const FlushArgs& a, int lb, int h, int l, int b, int P) {
  constexpr int EPL = Elem<T>::kPer16B;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  const int n = a.len[lb];
  const int cp = a.cap[b];
  const long long sbase = a.seq_base[b];
  if (n < 0 || cp < 0 || n > cp || sbase < 0 || sbase + (long long)a.HK * cp > a.rows_per_layer) return;
  const int rows = min(P, n);
  const int par = a.pend_par[lb] & 1;
  const float gamma = a.pend_gamma[lb];
  const float scale = a.pend_scale[lb];
  const int HQ = a.HK * G;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int rg = lane / LPR;
  const int dp = lane % LPR;
  const long long segrow0 = (long long)l * a.rows_per_layer + sbase + (long long)h * cp;
  const T* qg = reinterpret_cast<const T*>(a.qprev) + (((long long)l * 2 + par) * a.B + b) * HQ * D + (long long)h * G * D;
  const float* st = a.segstat + ((long long)lb * a.HK + h) * 2 * G;
  float qf[G][EPL], M[G], iL[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    Elem<T>::unpack(*reinterpret_cast<const uint4*>(qg + (long long)g * D + dp * EPL), qf[g]);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[g][e] *= scale;
    M[g] = st[g];
    iL[g] = st[G + g];
  }
  const T* Kb = reinterpret_cast<const T*>(a.k) + segrow0 * D + dp * EPL;
  float* score = a.score + segrow0;
  for (int r0 = w * RPW; r0 < rows; r0 += kNumWaves * RPW) {
    const int r = r0 + rg;
    const int rr = min(r, rows - 1);
    float kf[EPL];
    Elem<T>::unpack(*reinterpret_cast<const uint4*>(Kb + (long long)rr * D), kf);
    float c = 0.0f;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float acc = 0.0f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc = fmaf(qf[g][e], kf[e], acc);
      c = fmaf(hw_exp2(group_sum<LPR>(acc) - M[g]), iL[g], c);
    }
    if (dp == 0 && r < rows) score[r] = fmaf(gamma, score[r], c);
  }
}

template <typename T, int D, int G>
__global__ __launch_bounds__(kThreads) void flush_kernel(FlushArgs a) {
  long long i0, n;
  flush_range(a, i0, n);
  __shared__ int s_pend[kThreads];
  flush_scan(a, i0, n, s_pend);
  for (int t = 0; t < n; ++t) {
    const int P = s_pend[t];
    if (P <= 0) continue;
    const long long i = i0 + t;
    const int lb = a.l0 * a.B + (int)(i / a.HK);
    flush_segment_valu<T, D, G>(a, lb, (int)(i % a.HK), lb / a.B, lb % a.B, P);
    flush_done(a, lb);
  }
}

// bf16 flush on the matrix cores, the pending-update half of the decode
// loop on its own: one block per (layer, sequence, KV head); wave w takes the
// 32-row steps w, w + 4, ...; each step's K rows load straight into the
// operand registers (the next step's while this one computes), S = Q_prev K^T
// by MFMA, and s <- gamma s + sum_g exp2(scale x_g - M_g) / L_g.
template <int D, int G>
__device__ void flush_segment_bf16(const FlushArgs& a, int lb, int h, int l, int b, int P) {
  using Cfg = MfmaCfg<D>;
  constexpr int KK = Cfg::KK, ROWB = Cfg::ROWB, STEP = Cfg::STEP;
  static_assert(G <= 8, "pending heads live in lane groups 0 and 1");
  const int n = a.len[lb];
  const int cp = a.cap[b];
  const long long sbase = a.seq_base[b];
  if (n < 0 || cp < 0 || n > cp || sbase < 0 || sbase + (long long)a.HK * cp > a.rows_per_layer) return;
  const int rows = min(P, n);
  if (rows <= 0) return;
  const int par = a.pend_par[lb] & 1;
  const float gamma = a.pend_gamma[lb];
  const float scale = a.pend_scale[lb];
  const int HQ = a.HK * G;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int g4 = lane >> 4;
  const int s = lane & 15;
  const long long segrow0 = (long long)l * a.rows_per_layer + sbase + (long long)h * cp;
  const char* qg = reinterpret_cast<const char*>(a.qprev) +
                   ((((long long)l * 2 + par) * a.B + b) * HQ + (long long)h * G) * D * 2;
  const float* st = a.segstat + ((long long)lb * a.HK + h) * 2 * G;
  bf16x8_t qo[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) qo[kk] = q_operand<D, G>(qg, s, g4, kk);
  float pm[4], pi[4];
#pragma unroll
  for (int rr = 0; rr < 4; ++rr) {
    const int hh = 4 * g4 + rr;
    pm[rr] = hh < G ? st[hh] : 0.0f;
    pi[rr] = hh < G ? st[G + hh] : 0.0f;
  }
  const char* Kb = reinterpret_cast<const char*>(a.k) + segrow0 * ROWB;
  float* sc = a.score + segrow0;
  const int nsteps = (rows + STEP - 1) / STEP;

  bf16x8_t kn[2][KK];
  float sn = 0.0f;
  auto load = [&](int bs) {
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      const int row = min(bs + 16 * T + s, rows - 1);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kn[T][kk] = *reinterpret_cast<const bf16x8_t*>(Kb + (long long)row * ROWB + 64 * kk + 16 * g4);
    }
    sn = g4 < 2 ? sc[min(bs + 16 * g4 + s, rows - 1)] : 0.0f;
  };
  int idx = w;
  if (idx < nsteps) load(idx * STEP);
  while (idx < nsteps) {
    bf16x8_t kc[2][KK];
#pragma unroll
    for (int T = 0; T < 2; ++T)
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) kc[T][kk] = kn[T][kk];
    const float sold = sn;
    const int base = idx * STEP;
    const int nidx = idx + kNumWaves;
    if (nidx < nsteps) load(nidx * STEP);
    float part[2];
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      f32x4_t so = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) so = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qo[kk], kc[T][kk], so, 0, 0, 0);
      float acc = 0.0f;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) acc = fmaf(hw_exp2(fmaf(so[rr], scale, -pm[rr])), pi[rr], acc);
      part[T] = acc + __shfl_xor(acc, 16);
    }
    const int prow = base + 16 * g4 + s;
    if (g4 < 2 && prow < rows) sc[prow] = fmaf(gamma, sold, g4 == 0 ? part[0] : part[1]);
    idx = nidx;
  }
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void flush_bf16_kernel(FlushArgs a) {
  long long i0, n;
  flush_range(a, i0, n);
  __shared__ int s_pend[kThreads];
  flush_scan(a, i0, n, s_pend);
  for (int t = 0; t < n; ++t) {
    const int P = s_pend[t];
    if (P <= 0) continue;
    const long long i = i0 + t;
    const int lb = a.l0 * a.B + (int)(i / a.HK);
    flush_segment_bf16<D, G>(a, lb, (int)(i % a.HK), lb / a.B, lb % a.B, P);
    flush_done(a, lb);
  }
}

// Second launch of a settling call: s <- gamma s + sum_g exp2(x_g - M_g) / L_g
// over the rows each sequence's decode attended, from the logits that launch
// stored and its (M, 1/L); the deferred update's arithmetic, term for term
// (bf16: heads 0-3 and 4-7 summed apart, then added).  nb blocks per segment.
template <typename T, int G>
__global__ __launch_bounds__(kThreads) void settle_kernel(DecodeArgs a, int nb) {
  const int segs = a.B * a.HK;
  const int seg = (int)(blockIdx.x % segs);
  const int c = (int)(blockIdx.x / segs);
  const int b = seg / a.HK;
  const int h = seg - b * a.HK;
  const int rows = a.apply_rows[b];
  if (rows <= 0) return;
  const long long segrow0 = a.seq_base[b] + (long long)h * a.cap[b];
  const float* st = a.segstat + (long long)seg * 2 * G;
  float M[G], iL[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    M[g] = st[g];
    iL[g] = st[G + g];
  }
  float* sc = a.score + segrow0;
  const float* xl = a.logit + segrow0 * kLogitStride;
  for (int j = c * kThreads + (int)threadIdx.x; j < rows; j += nb * kThreads) {
    const f32x4_t x0 = *reinterpret_cast<const f32x4_t*>(xl + (long long)j * kLogitStride);
    const f32x4_t x1 = G > 4 ? *reinterpret_cast<const f32x4_t*>(xl + (long long)j * kLogitStride + 4)
                             : f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    float add;
    if constexpr (sizeof(T) == 2) {
      float lo = 0.0f, hi = 0.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float x = g < 4 ? x0[g & 3] : x1[g & 3];
        const float t = hw_exp2(fmaf(x, a.scale_log2, -M[g]));
        if (g < 4)
          lo = fmaf(t, iL[g], lo);
        else
          hi = fmaf(t, iL[g], hi);
      }
      add = lo + hi;
    } else {
      add = 0.0f;
#pragma unroll
      for (int g = 0; g < G; ++g) add = fmaf(hw_exp2((g < 4 ? x0[g & 3] : x1[g & 3]) - M[g]), iL[g], add);
    }
    sc[j] = fmaf(a.gamma, sc[j], add);
  }
}

// Overrides read at every call: LETHE_DECODE_BLOCKS (chunks the tiling aims
// for) and LETHE_DECODE_DETERMINISTIC (non-zero: every wavefront's steps are
// fixed, so repeated calls are bit-identical; by default a segment's
// wavefronts take their steps after the first from a counter, so a block the
// memory system serves faster takes more of them, and repeated calls differ
// in the last bits of out and the scores).
constexpr int64_t kMinChunksPerSeg = 4;
int env_int(const char* name) {
  const char* v = getenv(name);
  return v ? atoi(v) : 0;
}

// Chunks a launch may use by default: one per 1024 rows of the layer's
// capacity (the only size the host knows), between 512 and 4096; the plan
// takes about kStepsPerChunk hinted steps a chunk within that, and at least
// kMinChunks.  Measured with per-dispatch traces: the Qwen-7B batch-16 cache
// (64 segments of about 5k rows) does best near 768 chunks (14 steps), the
// Llama-8B batch-8 one near 512 (16 steps); the Llama-8B batch-128 ragged
// cache (1024 segments, 0.35M-5.8M live rows by layer) near 800-1024 on its
// smallest layers and 4096 on its largest.
constexpr int64_t kRowsPerTargetChunk = 1024;
constexpr int64_t kMinTarget = 512, kMaxTarget = 4096;
// Adaptive split: hinted steps per chunk a call aims for, and the fewest
// chunks (LETHE_DECODE_STEPS_PER_CHUNK, LETHE_DECODE_MIN_CHUNKS override).
constexpr int kStepsPerChunk = 14;
constexpr int kMinChunks = 512;

template <typename T, int D, int G, bool kCompact = false>
lethe_status launch_tdg(const DecodeArgs& a_in, hipStream_t s) {
  DecodeArgs a = a_in;
  const int env_blocks = env_int("LETHE_DECODE_BLOCKS");
  int64_t target = env_blocks;
  if (target <= 0) {
    target = a.rows_per_layer / kRowsPerTargetChunk;
    if (target < kMinTarget) target = kMinTarget;
    if (target > kMaxTarget) target = kMaxTarget;
  }
  a.deterministic = env_int("LETHE_DECODE_DETERMINISTIC") != 0;
  a.adaptive = env_blocks <= 0;
  const int env_spc = env_int("LETHE_DECODE_STEPS_PER_CHUNK");
  const int env_minc = env_int("LETHE_DECODE_MIN_CHUNKS");
  a.steps_per_chunk = env_spc > 0 ? env_spc : kStepsPerChunk;
  a.min_chunks = env_minc > 0 ? env_minc : kMinChunks;
  const int64_t segs = (int64_t)a.B * a.HK;
  // Flat split (no hints yet): at least four chunks per segment, so that with
  // many segments of ragged lengths the dispatcher hands the slots of early
  // finishers to waiting blocks.
  int64_t nflat = target / segs;
  if (env_blocks <= 0 && nflat < kMinChunksPerSeg) nflat = kMinChunksPerSeg;
  if (nflat > a.part_cap / segs) nflat = a.part_cap / segs;
  if (nflat > kMaxChunksPerSeg) nflat = kMaxChunksPerSeg;
  if (nflat < 1) nflat = 1;
  // Hinted split: about `target` chunks in all, plus at most one more per
  // segment from rounding up; one partial per block in the workspace.
  int64_t nbt = target;
  if (nbt > a.part_cap - segs) nbt = a.part_cap - segs;
  if (nbt > kMaxDecodeTarget) nbt = kMaxDecodeTarget;
  if (nbt < 1) nbt = 1;
  a.nbt = (int32_t)nbt;
  a.nch_flat = (int32_t)nflat;
  int64_t grid = nbt + segs;
  if (grid < segs * nflat) grid = segs * nflat;
  const auto kernel = decode_kernel<T, D, G, kCompact>();
  hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(kThreads), 0, s, a);
  if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  if (a.logit) {
    // About four rows per thread at the average segment capacity.
    int64_t nb = a.rows_per_layer / segs / (4 * kThreads);
    if (nb < 1) nb = 1;
    if (nb > 64) nb = 64;
    const auto settle = settle_kernel<T, G>;
    hipLaunchKernelGGL(settle, dim3((unsigned)(segs * nb)), dim3(kThreads), 0, s, a, (int)nb);
    if (hipGetLastError() != hipSuccess) return LETHE_ERR_HIP;
  }
  return LETHE_OK;
}

template <int D>
lethe_status launch_compact_d(const DecodeArgs& a, int G, hipStream_t s) {
  switch (G) {
    case 1: return launch_tdg<bf16_t, D, 1, true>(a, s);
    case 2: return launch_tdg<bf16_t, D, 2, true>(a, s);
    case 3: return launch_tdg<bf16_t, D, 3, true>(a, s);
    case 4: return launch_tdg<bf16_t, D, 4, true>(a, s);
    case 5: return launch_tdg<bf16_t, D, 5, true>(a, s);
    case 6: return launch_tdg<bf16_t, D, 6, true>(a, s);
    case 7: return launch_tdg<bf16_t, D, 7, true>(a, s);
    case 8: return launch_tdg<bf16_t, D, 8, true>(a, s);
  }
  return LETHE_ERR_UNSUPPORTED;
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

template <typename T, int D, int G>
lethe_status launch_flush_tdg(const FlushArgs& a, hipStream_t s) {
  // Each block takes a contiguous run of at most kThreads segments and reads
  // their pending lengths in one round: with nothing pending (a settled
  // step) the launch costs a few microseconds at any batch.
  const long long nseg = (long long)a.L * a.B * a.HK;
  const unsigned nb = (unsigned)std::min<long long>(nseg, std::max<long long>(kFlushBlocks, (nseg + kThreads - 1) / kThreads));
  if constexpr (sizeof(T) == 2)
    hipLaunchKernelGGL((flush_bf16_kernel<D, G>), dim3(nb), dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((flush_kernel<T, D, G>), dim3(nb), dim3(kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? LETHE_OK : LETHE_ERR_HIP;
}

template <typename T, int D>
lethe_status launch_flush_td(const FlushArgs& a, int G, hipStream_t s) {
  switch (G) {
    case 1: return launch_flush_tdg<T, D, 1>(a, s);
    case 2: return launch_flush_tdg<T, D, 2>(a, s);
    case 3: return launch_flush_tdg<T, D, 3>(a, s);
    case 4: return launch_flush_tdg<T, D, 4>(a, s);
    case 5: return launch_flush_tdg<T, D, 5>(a, s);
    case 6: return launch_flush_tdg<T, D, 6>(a, s);
    case 7: return launch_flush_tdg<T, D, 7>(a, s);
    case 8: return launch_flush_tdg<T, D, 8>(a, s);
  }
  return LETHE_ERR_UNSUPPORTED;
}

}  // namespace

// Chunk partials of lethe_decode_attn_score_noalloc.  Every call on a device
// shares that device's copy; a call writes every partial it reads, so nothing
// needs clearing between calls.  Host code uses only the address
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) char scratch[kDecodeScratchBytes];

lethe_status decode_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::atomic<void*> addr[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LETHE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return LETHE_ERR_UNSUPPORTED;
  void* p = addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    // Concurrent first calls on one device store the same address.
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return LETHE_ERR_HIP;
    addr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return LETHE_OK;
}

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

lethe_status launch_decode_compact(const DecodeArgs& a, int D, int G, hipStream_t s) {
  if (D == 128) return launch_compact_d<128>(a, G, s);
  if (D == 64) return launch_compact_d<64>(a, G, s);
  return LETHE_ERR_UNSUPPORTED;
}

lethe_status launch_flush(const FlushArgs& a, lethe_dtype dt, int D, int G, hipStream_t s) {
  if (dt == LETHE_BF16) {
    if (D == 128) return launch_flush_td<bf16_t, 128>(a, G, s);
    if (D == 64) return launch_flush_td<bf16_t, 64>(a, G, s);
  } else {
    if (D == 128) return launch_flush_td<float, 128>(a, G, s);
    if (D == 64) return launch_flush_td<float, 64>(a, G, s);
  }
  return LETHE_ERR_UNSUPPORTED;
}

}  // namespace lethe
