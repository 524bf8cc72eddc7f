// Workgroup-per-row building blocks shared by the streaming kernels: one
// 256-thread workgroup reduces one logit row.
#pragma once

#include "aal_device.h"

#include <limits.h>

namespace aal {

constexpr int kRowBlock = 256;
constexpr int kRowWaves = kRowBlock / kWave;


// Element group `gi` of a row: one 16-byte vector (VEC) or one element.
template <class TI, bool VEC>
struct Groups {
  static constexpr int E = VEC ? TI::kVec : 1;
  static __device__ __forceinline__ void load(const void* base, int64_t g0, int64_t gi, float (&x)[E]) {
    if constexpr (VEC) {
      TI::unpack(ldvec_nt(base, g0 + gi), x);
    } else {
      x[0] = TI::load1(base, g0 + gi);
    }
  }
};

static __device__ LseState block_lse(LseState st, float sc, LseState* sh) {
  st = wave_lse(st, sc);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sh[w] = st;
  __syncthreads();
  LseState r = sh[0];
#pragma unroll
  for (int i = 1; i < kRowWaves; ++i) r = lse_merge(r, sh[i], sc);
  __syncthreads();
  return r;
}

static __device__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sh[w] = v;
  __syncthreads();
  float r = sh[0];
#pragma unroll
  for (int i = 1; i < kRowWaves; ++i) r += sh[i];
  __syncthreads();
  return r;
}

// Largest value, lowest index among equal values.
static __device__ int block_argmax(float best, int idx, float* shf, int* shi) {
  const float wm = wave_max(best);
  const int wi = wave_min_i(best == wm ? idx : INT_MAX);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    shf[w] = wm;
    shi[w] = wi;
  }
  __syncthreads();
  float m = shf[0];
  int i = shi[0];
#pragma unroll
  for (int k = 1; k < kRowWaves; ++k) {
    if (shf[k] > m || (shf[k] == m && shi[k] < i)) {
      m = shf[k];
      i = shi[k];
    }
  }
  __syncthreads();
  return i;
}


}  // namespace aal
