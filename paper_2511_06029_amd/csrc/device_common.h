// Device helpers for gfx950: element unpacking, cross-lane reductions through
// DPP, and block-wide scans.  Wavefronts are 64 lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lethe {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Storage types.  bf16 is carried as raw 16-bit patterns; widening to fp32 is
// exact (the pattern becomes the high half of the fp32 word).
// ---------------------------------------------------------------------------
struct bf16_t {
  uint16_t bits;
};

template <typename T>
struct Elem;

template <>
struct Elem<bf16_t> {
  static constexpr int kBytes = 2;
  static constexpr int kPer16B = 8;  // elements in one 16-byte load
  __device__ static inline void unpack(const uint4& r, float* f) {
    f[0] = __uint_as_float(r.x << 16);
    f[1] = __uint_as_float(r.x & 0xffff0000u);
    f[2] = __uint_as_float(r.y << 16);
    f[3] = __uint_as_float(r.y & 0xffff0000u);
    f[4] = __uint_as_float(r.z << 16);
    f[5] = __uint_as_float(r.z & 0xffff0000u);
    f[6] = __uint_as_float(r.w << 16);
    f[7] = __uint_as_float(r.w & 0xffff0000u);
  }
};

template <>
struct Elem<float> {
  static constexpr int kBytes = 4;
  static constexpr int kPer16B = 4;
  __device__ static inline void unpack(const uint4& r, float* f) {
    f[0] = __uint_as_float(r.x);
    f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z);
    f[3] = __uint_as_float(r.w);
  }
};

// ---------------------------------------------------------------------------
// DPP lane movement (gfx9 encodings).
// ---------------------------------------------------------------------------
enum DppCtrl : int {
  kDppXor1 = 0xB1,         // quad_perm [1,0,3,2]
  kDppXor2 = 0x4E,         // quad_perm [2,3,0,1]
  kDppRowHalfMirror = 0x141,
  kDppRowMirror = 0x140,
};

template <int CTRL>
__device__ inline float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of N lanes (N in {4, 8, 16, 32, 64}); every lane of
// a group receives the group total.  The pairing order is fixed, so results
// are deterministic.
template <int N>
__device__ inline float group_sum(float v) {
  static_assert(N == 4 || N == 8 || N == 16 || N == 32 || N == 64, "group size");
  v += dpp_mov<kDppXor1>(v);
  v += dpp_mov<kDppXor2>(v);
  if constexpr (N >= 8) v += dpp_mov<kDppRowHalfMirror>(v);
  if constexpr (N >= 16) v += dpp_mov<kDppRowMirror>(v);
  if constexpr (N >= 32) v += __shfl_xor(v, 16);
  if constexpr (N >= 64) v += __shfl_xor(v, 32);
  return v;
}

// 2^x by the hardware instruction alone: results below 2^-126 flush to 0,
// which softmax weights and their rescaling factors never need; 2^-inf = 0.
// (The library exp2f adds a range fix-up of four more instructions.)
__device__ inline float hw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ inline float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ inline double wave_sum_d(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Inclusive scan of an int64 over one wave.
__device__ inline long long wave_incl_scan(long long v) {
  const int lane = threadIdx.x & (kWave - 1);
  for (int o = 1; o < kWave; o <<= 1) {
    long long t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// Exclusive scan of one int64 per thread over a block of NT threads; returns
// the thread's exclusive prefix and writes the block total to *total.
// `tmp` is LDS of at least NT / 64 + 1 int64 words.  Contains barriers.
template <int NT>
__device__ inline long long block_excl_scan(long long v, long long* tmp, long long* total) {
  constexpr int NWV = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  long long inc = wave_incl_scan(v);
  if (lane == kWave - 1) tmp[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long acc = 0;
    for (int i = 0; i < NWV; ++i) {
      long long t = tmp[i];
      tmp[i] = acc;
      acc += t;
    }
    tmp[NWV] = acc;
  }
  __syncthreads();
  long long ex = tmp[w] + inc - v;
  *total = tmp[NWV];
  __syncthreads();
  return ex;
}

__device__ inline void atomic_or_status(int32_t* st, int bits) {
  if (bits) atomicOr(st, bits);
}

}  // namespace lethe
