// Device-side building blocks shared by the libaal kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aal {

constexpr int kWave = 64;
constexpr float kNegInf = -__builtin_huge_valf();

// ----------------------------------------------------------------- elements
// Logits arrive as bf16 (raw uint16) or fp32.  A "vector" is one 16-byte load:
// 8 bf16 or 4 fp32 elements.  bf16 -> fp32 is exact (a shift or a mask).
struct Bf16 {
  using storage = uint16_t;
  static constexpr int kVec = 8;
  static __device__ __forceinline__ void unpack(const uint4& w, float (&x)[8]) {
    x[0] = __builtin_bit_cast(float, w.x << 16);
    x[1] = __builtin_bit_cast(float, w.x & 0xffff0000u);
    x[2] = __builtin_bit_cast(float, w.y << 16);
    x[3] = __builtin_bit_cast(float, w.y & 0xffff0000u);
    x[4] = __builtin_bit_cast(float, w.z << 16);
    x[5] = __builtin_bit_cast(float, w.z & 0xffff0000u);
    x[6] = __builtin_bit_cast(float, w.w << 16);
    x[7] = __builtin_bit_cast(float, w.w & 0xffff0000u);
  }
  static __device__ __forceinline__ float load1(const void* base, int64_t i) {
    uint32_t u = static_cast<const uint16_t*>(base)[i];
    return __builtin_bit_cast(float, u << 16);
  }
};

struct F32 {
  using storage = float;
  static constexpr int kVec = 4;
  static __device__ __forceinline__ void unpack(const uint4& w, float (&x)[4]) {
    x[0] = __builtin_bit_cast(float, w.x);
    x[1] = __builtin_bit_cast(float, w.y);
    x[2] = __builtin_bit_cast(float, w.z);
    x[3] = __builtin_bit_cast(float, w.w);
  }
  static __device__ __forceinline__ float load1(const void* base, int64_t i) {
    return static_cast<const float*>(base)[i];
  }
};

// Native clang vectors (the nontemporal builtins need them).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

static __device__ __forceinline__ uint4 to_uint4(u32x4 v) { return make_uint4(v.x, v.y, v.z, v.w); }

// 16-byte vector load of vector index `vi` (in units of 16 bytes).
static __device__ __forceinline__ uint4 ldvec(const void* base, int64_t vi) {
  return to_uint4(static_cast<const u32x4*>(base)[vi]);
}
// Streaming variant: data read exactly once, no reuse expected.
static __device__ __forceinline__ uint4 ldvec_nt(const void* base, int64_t vi) {
  return to_uint4(__builtin_nontemporal_load(static_cast<const u32x4*>(base) + vi));
}

// Gradient element types.  bf16 stores round to nearest even (one
// v_cvt_pk_bf16_f32 per pair).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
static __device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

struct GBf16 {
  using storage = uint16_t;
  static __device__ __forceinline__ void store1(void* base, int64_t i, float g) {
    static_cast<__bf16*>(base)[i] = static_cast<__bf16>(g);
  }
};
struct GF32 {
  using storage = float;
  static __device__ __forceinline__ void store1(void* base, int64_t i, float g) {
    static_cast<float*>(base)[i] = g;
  }
};

// Store E consecutive gradient values starting at element index e0 (aligned
// to E elements, so the store is 16 bytes for fp32 x4, bf16 x8, and two 16-byte
// stores for fp32 x8).
template <class TG, int E>
static __device__ __forceinline__ void store_vec(void* base, int64_t e0, const float (&g)[E]);

template <>
__device__ __forceinline__ void store_vec<GBf16, 8>(void* base, int64_t e0, const float (&g)[8]) {
  u32x4 w;
  w.x = pack_bf16x2(g[0], g[1]);
  w.y = pack_bf16x2(g[2], g[3]);
  w.z = pack_bf16x2(g[4], g[5]);
  w.w = pack_bf16x2(g[6], g[7]);
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(static_cast<uint16_t*>(base) + e0));
}
template <>
__device__ __forceinline__ void store_vec<GBf16, 4>(void* base, int64_t e0, const float (&g)[4]) {
  u32x2 w;
  w.x = pack_bf16x2(g[0], g[1]);
  w.y = pack_bf16x2(g[2], g[3]);
  __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(static_cast<uint16_t*>(base) + e0));
}
template <>
__device__ __forceinline__ void store_vec<GF32, 4>(void* base, int64_t e0, const float (&g)[4]) {
  f32x4 w = {g[0], g[1], g[2], g[3]};
  __builtin_nontemporal_store(w, reinterpret_cast<f32x4*>(static_cast<float*>(base) + e0));
}
template <>
__device__ __forceinline__ void store_vec<GF32, 8>(void* base, int64_t e0, const float (&g)[8]) {
  f32x4 a = {g[0], g[1], g[2], g[3]};
  f32x4 b = {g[4], g[5], g[6], g[7]};
  f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(base) + e0);
  __builtin_nontemporal_store(a, p);
  __builtin_nontemporal_store(b, p + 1);
}

// ---------------------------------------------------------------- math
// 2^x on the hardware transcendental unit (v_exp_f32).  Results below the
// normal range flush to zero, far below anything that reaches a sum.
static __device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// --------------------------------------------------------------- wave ops
// Reductions over the 64 lanes of a wave with DPP row operations, then a
// broadcast of lane 63.  `id` is the identity of the operation, which lanes
// outside a row_mask keep.
template <int Ctrl, int RowMask = 0xF>
static __device__ __forceinline__ float dppf(float v, float id) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, id), __builtin_bit_cast(int, v), Ctrl,
                                         RowMask, 0xF, false));
}

// Full-row-mask DPP move: every lane has a source lane for these patterns, so
// no identity is needed and the move can fuse into the consuming ALU op.
template <int Ctrl>
static __device__ __forceinline__ float dppm(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), Ctrl, 0xF, 0xF, true));
}

static __device__ __forceinline__ float readlane63(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

static __device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dppf<0xB1>(v, kNegInf));         // quad_perm [1,0,3,2]
  v = fmaxf(v, dppf<0x4E>(v, kNegInf));         // quad_perm [2,3,0,1]
  v = fmaxf(v, dppf<0x141>(v, kNegInf));        // row_half_mirror
  v = fmaxf(v, dppf<0x140>(v, kNegInf));        // row_mirror
  v = fmaxf(v, dppf<0x142, 0xA>(v, kNegInf));   // row_bcast:15
  v = fmaxf(v, dppf<0x143, 0xC>(v, kNegInf));   // row_bcast:31
  return readlane63(v);
}

static __device__ __forceinline__ float wave_sum(float v) {
  v = v + dppf<0xB1>(v, 0.f);
  v = v + dppf<0x4E>(v, 0.f);
  v = v + dppf<0x141>(v, 0.f);
  v = v + dppf<0x140>(v, 0.f);
  v = v + dppf<0x142, 0xA>(v, 0.f);
  v = v + dppf<0x143, 0xC>(v, 0.f);
  return readlane63(v);
}

// The same reductions over N independent values at once: every DPP step is
// applied to all N values before the next, so DPP data hazards are covered by
// independent work instead of s_nop.  Results are uniform across the wave.
template <int N>
static __device__ __forceinline__ void wave_max_n(float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dppm<0xB1>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dppm<0x4E>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dppm<0x141>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dppm<0x140>(v[i]));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dppf<0x142, 0xA>(v[i], kNegInf));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], dppf<0x143, 0xC>(v[i], kNegInf));
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = readlane63(v[i]);
}

template <int N>
static __device__ __forceinline__ void wave_sum_n(float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = v[i] + dppm<0xB1>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = v[i] + dppm<0x4E>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = v[i] + dppm<0x141>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = v[i] + dppm<0x140>(v[i]);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = v[i] + dppf<0x142, 0xA>(v[i], 0.f);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = v[i] + dppf<0x143, 0xC>(v[i], 0.f);
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = readlane63(v[i]);
}

// Wave merge of N (msc, sum) pairs: msc <- max over lanes (the wave's
// reference), sum <- sum over lanes of sum * 2^(msc_lane - msc).
template <int N>
static __device__ __forceinline__ void wave_lse_n(float (&msc)[N], float (&s)[N]) {
  float M[N];
#pragma unroll
  for (int i = 0; i < N; ++i) M[i] = msc[i];
  wave_max_n(M);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    s[i] = (M[i] == kNegInf) ? 0.f : s[i] * ex2(msc[i] - M[i]);
    msc[i] = M[i];
  }
  wave_sum_n(s);
}

// Transposed wave reductions of N per-lane values (N a multiple of 4): the
// four in-row DPP butterflies leave each row's total on all 16 lanes of the
// row; then the gfx950 cross-row swaps combine two values per instruction
// pair.  permlane16_swap(a, b) returns [a.r0, b.r0, a.r2, b.r2] and
// [a.r1, b.r1, a.r3, b.r3] (rows of 16 lanes), so op of the two holds a's
// rows-0+1 and rows-2+3 totals on rows 0 and 2 and b's on rows 1 and 3;
// permlane32_swap(x, y) returns [x.lo, y.lo] and [x.hi, y.hi].  On return the
// total of value 4j+q is out[j] on every lane of row q (lanes 16q..16q+15).
// About 5.5 instructions per value instead of the 10 of the broadcast form.
template <class Op, int N>
static __device__ __forceinline__ void wave_reduce_t(float (&x)[N], float (&out)[N / 4], Op op) {
  static_assert(N % 4 == 0, "values in groups of four");
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dppm<0xB1>(x[i]));   // quad_perm [1,0,3,2]
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dppm<0x4E>(x[i]));   // quad_perm [2,3,0,1]
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dppm<0x141>(x[i]));  // row_half_mirror
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = op(x[i], dppm<0x140>(x[i]));  // row_mirror
  float h[N / 2];
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x[2 * i]),
                                                    __builtin_bit_cast(unsigned, x[2 * i + 1]), false, false);
    h[i] = op(__builtin_bit_cast(float, unsigned(r[0])), __builtin_bit_cast(float, unsigned(r[1])));
  }
#pragma unroll
  for (int j = 0; j < N / 4; ++j) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, h[2 * j]),
                                                    __builtin_bit_cast(unsigned, h[2 * j + 1]), false, false);
    out[j] = op(__builtin_bit_cast(float, unsigned(r[0])), __builtin_bit_cast(float, unsigned(r[1])));
  }
}
struct OpAdd {
  __device__ __forceinline__ float operator()(float a, float b) const { return a + b; }
};
struct OpMax {
  __device__ __forceinline__ float operator()(float a, float b) const { return fmaxf(a, b); }
};
// The total of value i after wave_reduce_t, as a wave-uniform value.
template <int NQ>
static __device__ __forceinline__ float reduced_t(const float (&out)[NQ], int i) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, out[i / 4]), 16 * (i % 4)));
}

// Integer minimum over the wave (DPP steps as above), broadcast to all lanes.
template <int Ctrl, int RowMask = 0xF>
static __device__ __forceinline__ int dppi(int v, int id) {
  return __builtin_amdgcn_update_dpp(id, v, Ctrl, RowMask, 0xF, false);
}
static __device__ __forceinline__ int wave_min_i(int v) {
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true));
  v = min(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true));
  v = min(v, dppi<0x142, 0xA>(v, INT_MAX));
  v = min(v, dppi<0x143, 0xC>(v, INT_MAX));
  return __builtin_amdgcn_readlane(v, 63);
}

// fp64 sums are needed once per row only: a butterfly through __shfl_xor is
// enough there.

static __device__ __forceinline__ double wave_sum_d(double v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Inclusive prefix sum over lanes in lane order (fp64, deterministic).
static __device__ __forceinline__ double wave_incl_scan_d(double v) {
  const int lane = threadIdx.x & (kWave - 1);
  for (int off = 1; off < kWave; off <<= 1) {
    double o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

// ------------------------------------------------------- online (max, sum)
// Running log-sum-exp state of one lane over raw logits z at scale
// sc = log2(e)/T:  sum = sum_v 2^(z_v*sc - msc) with msc = fl(m*sc),
// m = max z seen so far.  All terms share one reference, and merging two
// states rescales the smaller one by 2^(msc_small - msc_big).
struct LseState {
  float m;    // max raw logit (-inf if none)
  float msc;  // fl(m * sc)
  float s;    // sum of 2^(z*sc - msc)
};

static __device__ __forceinline__ LseState lse_init() { return {kNegInf, kNegInf, 0.f}; }

// Fold a chunk whose max is cm and whose terms will be added by the caller
// against the returned reference.  Returns false if everything so far is -inf.
static __device__ __forceinline__ bool lse_rebase(LseState& st, float cm, float sc) {
  float mn = fmaxf(st.m, cm);
  if (mn == kNegInf) return false;
  float mscn = mn * sc;
  st.s *= ex2(st.msc - mscn);  // msc = -inf on the first chunk: factor 0
  st.m = mn;
  st.msc = mscn;
  return true;
}

// msc is always recomputed as fl(m*sc), so every holder of the same m holds
// the same reference.
static __device__ __forceinline__ LseState lse_merge(LseState a, LseState b, float sc) {
  float m = fmaxf(a.m, b.m);
  if (m == kNegInf) return lse_init();
  float msc = m * sc;
  float s = a.s * ex2(a.msc - msc) + b.s * ex2(b.msc - msc);
  return {m, msc, s};
}

// Wave-wide merge (result uniform across the wave).
static __device__ __forceinline__ LseState wave_lse(LseState st, float sc) {
  float m = wave_max(st.m);
  if (m == kNegInf) return lse_init();
  float msc = m * sc;
  float s = wave_sum(st.s * ex2(st.msc - msc));
  return {m, msc, s};
}

}  // namespace aal
