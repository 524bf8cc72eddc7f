// Building blocks of the register-resident schedules: buffer-resource
// loads and stores (straight to LDS for staging), LDS-only barriers, tagged
// 64-bit exchange words with bounded polls, and the row-partial folds.
#pragma once

#include "aal_device.h"

#include <limits.h>

#include <stdlib.h>

#include <atomic>

namespace aal {
namespace {

constexpr unsigned kSpinLimit = 1u << 22;  // polls (~1 us each): seconds, far above any legitimate wait

// The operand is the whole 128-bit tuple, so the data stays in the register
// quadruple the 16-byte loads write (unpacked copies are not kept live across
// phases, which would double the register footprint).
__device__ __forceinline__ void pin(u32x4& x) { asm volatile("" : "+v"(x)); }

__device__ __forceinline__ u32x4 neg_inf_vec(Bf16) { return u32x4{0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u}; }
__device__ __forceinline__ u32x4 neg_inf_vec(F32) { return u32x4{0xff800000u, 0xff800000u, 0xff800000u, 0xff800000u}; }

// Buffer resources: a wave-uniform 128-bit descriptor (base, byte range) in
// SGPRs.  Accesses take a 32-bit per-lane byte offset plus an SGPR offset,
// so no per-access 64-bit address arithmetic is needed.  For a raw buffer the
// per-lane offset is range-checked: a store at or past the range is dropped.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRawBufferWord3 = 0x00020000;  // gfx9 raw (untyped) dword access
constexpr int kNontemporal = 2;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), short(0), int(bytes), kRawBufferWord3);
}
// CP: the cache-policy bits of the access (nontemporal by default)
template <int CP = kNontemporal>
__device__ __forceinline__ u32x4 bld16(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, CP);
}
// The same 16 bytes per lane, delivered straight to LDS: lane l of the wave
// writes bytes [16 l, 16 l + 16) from `dst` (wave-uniform), no VGPRs involved.
typedef __attribute__((address_space(3))) void lds_void_t;
template <int CP = kNontemporal>
__device__ __forceinline__ void bld16_lds(rsrc_t r, void* dst, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)dst, 16, voff, soff, 0, CP);
}
// s_waitcnt vmcnt(0) as an instruction the compiler's wait-count tracking sees
// (gfx9 encoding: vmcnt 0, expcnt 7, lgkmcnt 15).
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// s_waitcnt vmcnt(N): at most N of the wave's vector-memory instructions are
// outstanding.  They complete in issue order, so every instruction issued
// before the last N has completed (loads into LDS included, which the
// compiler's own wait counts do not track).
template <int N>
__device__ __forceinline__ void wait_vmem_le() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | 0x0F70 | ((N >> 4) << 14));
}
// s_waitcnt lgkmcnt(0) alone (vmcnt 63, expcnt 7): the wave's LDS reads have
// completed.
__device__ __forceinline__ void wait_lds_all() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Workgroup barrier for LDS data only.  __syncthreads() is also a release
// fence for every LDS write, which includes staging loads still in flight, so
// it would wait for them; the workgroup exchanges in this kernel go through
// ordinary LDS stores (and global atomics that carry their own tags), so
// draining the LDS queue is all a barrier needs.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// One vector of gradient values at per-lane byte offset `off` of a row.
template <class TG, int E, int CP = kNontemporal>
__device__ __forceinline__ void store_g(rsrc_t r, uint32_t off, const float (&g)[E]) {
  if constexpr (sizeof(typename TG::storage) == 2 && E == 8) {
    const u32x4 w = {pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3]), pack_bf16x2(g[4], g[5]),
                     pack_bf16x2(g[6], g[7])};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, off, 0, CP);
  } else if constexpr (sizeof(typename TG::storage) == 2 && E == 4) {
    const u32x2 w = {pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3])};
    __builtin_amdgcn_raw_buffer_store_b64(w, r, off, 0, CP);
  } else if constexpr (E == 4) {
    const u32x4 w = {__builtin_bit_cast(uint32_t, g[0]), __builtin_bit_cast(uint32_t, g[1]),
                     __builtin_bit_cast(uint32_t, g[2]), __builtin_bit_cast(uint32_t, g[3])};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, off, 0, CP);
  } else {
    const u32x4 w0 = {__builtin_bit_cast(uint32_t, g[0]), __builtin_bit_cast(uint32_t, g[1]),
                      __builtin_bit_cast(uint32_t, g[2]), __builtin_bit_cast(uint32_t, g[3])};
    const u32x4 w1 = {__builtin_bit_cast(uint32_t, g[4]), __builtin_bit_cast(uint32_t, g[5]),
                      __builtin_bit_cast(uint32_t, g[6]), __builtin_bit_cast(uint32_t, g[7])};
    __builtin_amdgcn_raw_buffer_store_b128(w0, r, off, 0, CP);
    __builtin_amdgcn_raw_buffer_store_b128(w1, r, off + 16u, 0, CP);
  }
}

// One gradient value (through the same buffer path, so it lands after an
// earlier vector store of the same thread to the same address).
template <class TG>
__device__ __forceinline__ void store_one(rsrc_t r, uint32_t off, float g) {
  if constexpr (sizeof(typename TG::storage) == 2) {
    const __bf16 h = static_cast<__bf16>(g);
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, h), r, off, 0, 0);
  } else {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, g), r, off, 0, 0);
  }
}

template <class TI, int E>
__device__ __forceinline__ void unpackv(const u32x4& w, float (&x)[E]) {
  TI::unpack(make_uint4(w.x, w.y, w.z, w.w), x);
}

// Per-element mask bits kept in VGPRs between two phases.  push_bit appends
// one bit per lane from a wave lane mask (the result of a compare) with a
// single add-with-carry: bits = 2 bits + carry, so after n pushes the i-th
// pushed bit (from 0) sits at position n - 1 - i.  The compiler rewrites
// 2 bits + b as a shift and an OR of a selected constant (three or four
// instructions), hence the inline assembly.
__device__ __forceinline__ void push_bit(uint32_t& bits, uint64_t lanes) {
  uint64_t carry_out;
  asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(bits), "=s"(carry_out) : "v"(bits), "s"(lanes));
}
// a where bit `pos` of bits is set, else b: a sign-extended one-bit field
// selects whole words through a bitfield insert.
__device__ __forceinline__ float select_bit(uint32_t bits, int pos, float a, float b) {
  const int32_t m = __builtin_amdgcn_sbfe(int32_t(bits), pos, 1);
  float r;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "v"(a), "v"(b));
  return r;
}

__device__ __forceinline__ uint64_t tagged(float v, uint32_t tag) {
  return (uint64_t(tag) << 32) | __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ void publish(uint64_t* p, float v, uint32_t tag) {
  __hip_atomic_store(p, tagged(v, tag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t peek(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float value_of(uint64_t x) { return __builtin_bit_cast(float, uint32_t(x)); }

// Reads the N consecutive tagged words at p, waiting until all carry `tag`.
template <int N>
__device__ __forceinline__ void collect(const uint64_t* p, uint32_t tag, unsigned* err, float (&out)[N]) {
  uint64_t x[N];
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = peek(p + i);
  unsigned spins = 0;
  for (;;) {
    bool ok = true;
#pragma unroll
    for (int i = 0; i < N; ++i) ok = ok && uint32_t(x[i] >> 32) == tag;
    if (ok) break;
    if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) break;
    if (++spins > kSpinLimit) {
      __hip_atomic_store(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] = peek(p + i);
  }
#pragma unroll
  for (int i = 0; i < N; ++i) out[i] = value_of(x[i]);
}

// Merge (msc, s) into (m, acc): references are fl(max * sc), monotone in max.
__device__ __forceinline__ void lse_fold(float& m, float& acc, float msc, float s) {
  const float nm = fmaxf(m, msc);
  if (nm != kNegInf) {
    acc = acc * ex2(m - nm) + s * ex2(msc - nm);
    m = nm;
  }
}
// Merge (value, index, payload) keeping the larger value, then the lower
// index; the payload (the draft logit at that index) travels with it.
__device__ __forceinline__ void argmax_fold(float& bv, float& bi, float& bz, float v, float i, float z) {
  if (v > bv || (v == bv && __builtin_bit_cast(int, i) < __builtin_bit_cast(int, bi))) {
    bv = v;
    bi = i;
    bz = z;
  }
}

// log2 p - log2 q for the KL term's p (log p - log q), finite wherever p = 0
// (t = -inf, where the difference is -inf, or undefined when q = 0 too): one
// max instead of a test of p, since 0 times the lowest finite float is 0,
// the limit of p log p.  Where q = 0 < p the difference stays +inf (KL is
// infinite).  On NaN operands the hardware max returns the other operand.
__device__ __forceinline__ float kl_diff(float t, float u) { return fmaxf(t - u, -3.402823466e38f); }

// A thread's part of the greedy token of one row: the lowest column among its
// elements that holds m, the maximum of those elements, with the draft logit
// at that column as the payload.  xs are the row's target logits as
// unpacked from its NV vectors, dw the row's packed draft vectors; element e
// of vector v sits in column base + v * kBlock * E + e.  With the maximum
// known beforehand (the normaliser needs it anyway) a compare and a select
// per element suffice, and the payload is chosen as the packed draft word of
// the matching pair (one select per word) and unpacked once at the end.
// m = -inf (no finite element) gives index INT_MAX and payload -inf, as
// a strict running comparison against -inf would.
template <class TI, int NV, int E, int kBlock>
__device__ __forceinline__ void first_max(const float (&xs)[NV][E], const u32x4 (&dw)[NV], float m, int base,
                                          float& bidx, float& bz) {
  constexpr int EPW = E / 4;  // elements per 32-bit word: 2 (bf16) or 1 (fp32)
  int li = 0;
  uint32_t w = 0;
#pragma unroll
  for (int v = NV - 1; v >= 0; --v)
#pragma unroll
    for (int q = 3; q >= 0; --q) {
      bool hit = false;
#pragma unroll
      for (int h = EPW - 1; h >= 0; --h) {
        const int e = q * EPW + h;
        if (xs[v][e] == m) {
          li = v * E + e;  // an inline constant; the column is formed once below
          hit = true;
        }
      }
      if (hit) w = dw[v][q];
    }
  float z;
  if constexpr (EPW == 2) {
    z = __builtin_bit_cast(float, (li & 1) ? (w & 0xffff0000u) : (w << 16));
  } else {
    z = __builtin_bit_cast(float, w);
  }
  const bool none = m == kNegInf;
  bidx = __builtin_bit_cast(float, none ? INT_MAX : base + (li / E) * (kBlock * E) + li % E);
  bz = none ? kNegInf : z;
}

// Wave-wide argmax of (value, index) pairs, lowest index on ties, with the
// payload of the winning lane.  All lanes receive the result.
__device__ __forceinline__ void wave_argmax(float& bv, float& bi, float& bz) {
  float m[1] = {bv};
  wave_max_n(m);
  const int x = wave_min_i(bv == m[0] ? __builtin_bit_cast(int, bi) : INT_MAX);
  const uint64_t own = __builtin_amdgcn_ballot_w64(bv == m[0] && __builtin_bit_cast(int, bi) == x);
  const int src = own != 0 ? __builtin_ctzll(own) : 0;
  bz = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, bz), src));
  bv = m[0];
  bi = __builtin_bit_cast(float, x);
}

// The value the resident kernels' error word starts at: 0, or 1 when the
// environment variable AAL_TEST_PRESET_TIMEOUT is "1" — the state a poll
// time-out leaves, so that tests can drive the time-out path (every bounded
// wait then ends at once, the kernel drains and the loss reads NaN) without
// waiting seconds for a real one.
inline uint64_t initial_error_word() {
  const char* v = getenv("AAL_TEST_PRESET_TIMEOUT");
  return (v != nullptr && v[0] == '1' && v[1] == '\0') ? 1u : 0u;
}

struct DevInfo {
  int cus = 0;
  bool coop = false;
};

// Per-device attributes, cached in a fixed table of atomics: nothing here has
// a destructor to run at process exit.  A device beyond the table is queried
// on every call.
constexpr int kMaxCachedDevices = 64;
std::atomic<int> g_dev_cus[kMaxCachedDevices];   // 0 = not yet queried
std::atomic<int> g_dev_coop[kMaxCachedDevices];

DevInfo device_info() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return {};
  if (dev < kMaxCachedDevices) {
    const int cus = g_dev_cus[dev].load(std::memory_order_acquire);
    if (cus != 0) return {cus, g_dev_coop[dev].load(std::memory_order_relaxed) != 0};
  }
  int cus = 0, coop = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return {};
  if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess) return {};
  if (dev < kMaxCachedDevices) {
    g_dev_coop[dev].store(coop, std::memory_order_relaxed);
    g_dev_cus[dev].store(cus, std::memory_order_release);
  }
  return {cus, coop != 0};
}

}  // namespace
}  // namespace aal
