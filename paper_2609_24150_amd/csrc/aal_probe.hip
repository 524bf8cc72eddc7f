// Streaming probe: the practical HBM rate of a traffic mix on this device,
// measured with the access the loss kernels use (16-byte nontemporal loads
// and stores through buffer resources).  A measurement aid for reporting
// the kernels against the ceiling of their own mix; not part of the method.
#include "aal_device.h"
#include "aal_internal.h"
#include "aal_resident_common.h"

namespace aal {
namespace {

constexpr int kProbeBlock = 256;
constexpr int kProbeUnroll = 4;  // independent 16-byte loads per source in flight per thread

// NS sources summed (32-bit wrapping adds) into dst when WR; otherwise a store
// of the flag only where a summed word is all ones (data-dependent, so every
// load stays live; callers fill the sources so that it does not happen).
// Buffer i covers n 16-byte vectors; the grid strides over them in tiles of
// kProbeUnroll vectors per thread.
template <int NS, bool WR>
__global__ __launch_bounds__(kProbeBlock) void k_stream_probe(const u32x4* a, const u32x4* b, const u32x4* c,
                                                              u32x4* d, int64_t n, uint32_t* flag) {
  const int64_t step = int64_t(gridDim.x) * kProbeBlock;
  for (int64_t base = int64_t(blockIdx.x) * kProbeBlock * kProbeUnroll + threadIdx.x; base < n;
       base += step * kProbeUnroll) {
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t i = base + int64_t(u) * kProbeBlock;
      v[u] = i < n ? __builtin_nontemporal_load(a + i) : u32x4{0u, 0u, 0u, 0u};
    }
    if constexpr (NS > 1) {
#pragma unroll
      for (int u = 0; u < kProbeUnroll; ++u) {
        const int64_t i = base + int64_t(u) * kProbeBlock;
        if (i < n) v[u] += __builtin_nontemporal_load(b + i);
      }
    }
    if constexpr (NS > 2) {
#pragma unroll
      for (int u = 0; u < kProbeUnroll; ++u) {
        const int64_t i = base + int64_t(u) * kProbeBlock;
        if (i < n) v[u] += __builtin_nontemporal_load(c + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t i = base + int64_t(u) * kProbeBlock;
      if (i >= n) continue;
      if constexpr (WR) {
        __builtin_nontemporal_store(v[u], d + i);
      } else if (v[u].x == 0xFFFFFFFFu && v[u].y == 0xFFFFFFFFu) {
        flag[0] = 1u;
      }
    }
  }
}

template <int NS>
hipError_t launch_ns(const void* a, const void* b, const void* c, void* d, int64_t n, uint32_t* flag, int grid,
                     hipStream_t stream) {
  const auto* pa = static_cast<const u32x4*>(a);
  const auto* pb = static_cast<const u32x4*>(b);
  const auto* pc = static_cast<const u32x4*>(c);
  auto* pd = static_cast<u32x4*>(d);
  if (d != nullptr) {
    k_stream_probe<NS, true><<<grid, kProbeBlock, 0, stream>>>(pa, pb, pc, pd, n, flag);
  } else {
    k_stream_probe<NS, false><<<grid, kProbeBlock, 0, stream>>>(pa, pb, pc, pd, n, flag);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_stream_probe(const void* const src[3], int n_src, void* dst, size_t bytes, uint32_t* flag,
                               hipStream_t stream) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int64_t n = int64_t(bytes / 16);
  // four 256-thread workgroups per CU (measured: 2 reads + 1 write streams
  // fastest with 3-4, 5% slower with 8), fewer when the buffers are small
  const int64_t tiles = (n + int64_t(kProbeBlock) * kProbeUnroll - 1) / (int64_t(kProbeBlock) * kProbeUnroll);
  const int grid = int(tiles < int64_t(4) * cus ? tiles : int64_t(4) * cus);
  switch (n_src) {
    case 1: return launch_ns<1>(src[0], nullptr, nullptr, dst, n, flag, grid, stream);
    case 2: return launch_ns<2>(src[0], src[1], nullptr, dst, n, flag, grid, stream);
    default: return launch_ns<3>(src[0], src[1], src[2], dst, n, flag, grid, stream);
  }
}

}  // namespace aal
