// Simulated acceptance length and group-relative advantage.
//
//   k_sim_rows    one workgroup per logit row (prefix p, rollout g, position k).
//                 One sweep over both rows: the target's max / sum-exp, and for
//                 the draft a (max, sum) pair per tile of contiguous tokens, so
//                 that the cumulative draft mass is known tile by tile in token
//                 order.  The draft token is the inverse-CDF sample with u1
//                 (the first token whose cumulative mass exceeds u1 times the
//                 total): a wave scans the tile masses in fp64, re-reads the one
//                 tile that holds the crossing and finds the token.  It is
//                 accepted iff u2 q(x) < p(x)  (sampling verification, Eq.
//                 acc_sample).
//   k_group_adv   one workgroup per prefix: reward = accepted positions before
//                 the first rejection, then (r - mean) / (std + eps) over the G
//                 rollouts (Eq. advantage), optionally clipped.
#include "aal_device.h"
#include "aal_internal.h"

namespace aal {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / kWave;

static __device__ __forceinline__ double bcast_d(double v, int lane) { return __shfl(v, lane, 64); }

template <class TI, bool VEC>
struct SimGroups {
  static constexpr int E = VEC ? TI::kVec : 1;
  static __device__ __forceinline__ void load(const void* base, int64_t g0, int gi, int ng, float (&x)[E]) {
    if (gi < ng) {
      if constexpr (VEC) {
        TI::unpack(ldvec_nt(base, g0 + gi), x);
      } else {
        x[0] = TI::load1(base, g0 + gi);
      }
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) x[e] = kNegInf;
    }
  }
};

// Mass of tile t relative to the row reference msc: sum_t * 2^(msc_t - msc).
static __device__ __forceinline__ double tile_mass(const float2* ts, int t, float msc) {
  return double(ts[t].y) * double(ex2(ts[t].x - msc));
}

template <class TI, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void k_sim_rows(const void* __restrict__ zd, const void* __restrict__ zt, int V,
                                                     float sc, const float* __restrict__ u1,
                                                     const float* __restrict__ u2, int32_t* __restrict__ token,
                                                     int32_t* __restrict__ accept) {
  using Gr = SimGroups<TI, VEC>;
  constexpr int E = Gr::E;
  constexpr int TG = kWave * U;  // element groups per tile
  extern __shared__ float2 tile_stat[];  // (msc_t, sum_t) per tile
  __shared__ LseState sh_lse[kWaves];
  __shared__ int sh_ctile;
  __shared__ double sh_base, sh_theta;
  __shared__ float sh_msc, sh_l2s;

  const int64_t row = blockIdx.x;
  const int ng = V / E;
  const int ntiles = (ng + TG - 1) / TG;
  const int64_t g0 = row * int64_t(ng);
  const int64_t e0 = row * int64_t(V);
  const int w = threadIdx.x / kWave;
  const int lane = threadIdx.x & (kWave - 1);

  LseState st = lse_init();
  for (int t = w; t < ntiles; t += kWaves) {
    float xd[U][E], xt[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = t * TG + u * kWave + lane;
      Gr::load(zd, g0, gi, ng, xd[u]);
      Gr::load(zt, g0, gi, ng, xt[u]);
    }
    float lm = kNegInf;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) lm = fmaxf(lm, xd[u][e]);
    const float tm = wave_max(lm);
    float tmsc = kNegInf, tsum = 0.f;
    if (tm != kNegInf) {
      tmsc = tm * sc;
      float ls = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) ls += ex2(__builtin_fmaf(xd[u][e], sc, -tmsc));
      tsum = wave_sum(ls);
    }
    if (lane == 0) tile_stat[t] = make_float2(tmsc, tsum);

    float ct = kNegInf;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) ct = fmaxf(ct, xt[u][e]);
    if (lse_rebase(st, ct, sc)) {
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) acc += ex2(__builtin_fmaf(xt[u][e], sc, -st.msc));
      st.s += acc;
    }
  }
  __syncthreads();
  // target normaliser (block-wide, deterministic order)
  {
    LseState ws = wave_lse(st, sc);
    if (lane == 0) sh_lse[w] = ws;
    __syncthreads();
    st = sh_lse[0];
#pragma unroll
    for (int i = 1; i < kWaves; ++i) st = lse_merge(st, sh_lse[i], sc);
  }

  // Wave 0: locate the tile whose cumulative draft mass crosses u1 * total.
  if (w == 0) {
    float msc = kNegInf;
    for (int t = lane; t < ntiles; t += kWave) msc = fmaxf(msc, tile_stat[t].x);
    msc = wave_max(msc);
    const int per = (ntiles + kWave - 1) / kWave;
    const int t0 = min(lane * per, ntiles);
    const int t1 = min(t0 + per, ntiles);
    double ls = 0.0;
    for (int t = t0; t < t1; ++t) ls += tile_mass(tile_stat, t, msc);
    const double incl = wave_incl_scan_d(ls);
    const double total = bcast_d(incl, kWave - 1);
    const double theta = double(u1[row]) * total;
    double excl = __shfl_up(incl, 1, 64);
    if (lane == 0) excl = 0.0;
    const unsigned long long bal = __ballot(incl > theta);
    const int L = bal ? (__ffsll(bal) - 1) : (kWave - 1);
    if (lane == L) {
      double c = excl, last_base = excl;
      int ct = -1, last_pos = -1;
      for (int t = t0; t < t1; ++t) {
        const double mt = tile_mass(tile_stat, t, msc);
        if (mt > 0.0) {
          last_pos = t;
          last_base = c;
        }
        if (c + mt > theta) {
          ct = t;
          break;
        }
        c += mt;
      }
      if (ct < 0) {  // rounding left theta at or past the end of this lane's tiles
        ct = last_pos >= 0 ? last_pos : max(t1 - 1, 0);
        c = last_base;
      }
      sh_ctile = ct;
      sh_base = c;
      sh_theta = theta;
    }
    if (lane == 0) {
      sh_msc = msc;
      sh_l2s = float(log2(total));
    }
  }
  __syncthreads();

  if (w == 0) {
    const int ct = sh_ctile;
    const double theta = sh_theta;
    const float msc = sh_msc;
    double cum = sh_base;
    int x = -1;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = ct * TG + u * kWave + lane;
      float xd[E], ev[E];
      Gr::load(zd, g0, gi, ng, xd);
      double ls = 0.0;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        ev[e] = ex2(__builtin_fmaf(xd[e], sc, -msc));
        ls += double(ev[e]);
      }
      const double incl = wave_incl_scan_d(ls);
      const double tot = bcast_d(incl, kWave - 1);
      if (x < 0 && cum + tot > theta) {
        double excl = __shfl_up(incl, 1, 64);
        if (lane == 0) excl = 0.0;
        const unsigned long long bal = __ballot(cum + incl > theta);
        const int L = __ffsll(bal) - 1;
        int xi = -1;
        if (lane == L) {
          double c = cum + excl;
          int last_pos = -1;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            if (ev[e] > 0.f) last_pos = e;
            c += double(ev[e]);
            if (xi < 0 && c > theta) xi = e;
          }
          if (xi < 0) xi = last_pos >= 0 ? last_pos : 0;
          xi += gi * E;
        }
        x = __shfl(xi, L, 64);
      }
      cum += tot;
    }
    if (x < 0) {
      // Rounding left theta past the re-read tile mass: take the tile's last
      // token with positive mass, else its last finite token.
      int pos = -1, fin = -1;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int gi = ct * TG + u * kWave + lane;
        float xd[E];
        Gr::load(zd, g0, gi, ng, xd);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if (xd[e] != kNegInf) fin = max(fin, gi * E + e);
          if (ex2(__builtin_fmaf(xd[e], sc, -msc)) > 0.f) pos = max(pos, gi * E + e);
        }
      }
      for (int off = 32; off > 0; off >>= 1) {
        pos = max(pos, __shfl_xor(pos, off, 64));
        fin = max(fin, __shfl_xor(fin, off, 64));
      }
      x = pos >= 0 ? pos : (fin >= 0 ? fin : 0);
    }
    if (lane == 0) {
      const float zdx = TI::load1(zd, e0 + x);
      const float ztx = TI::load1(zt, e0 + x);
      const float q = ex2(__builtin_fmaf(zdx, sc, -msc) - sh_l2s);
      const float p = ex2(__builtin_fmaf(ztx, sc, -st.msc) - __log2f(st.s));
      token[row] = x;
      accept[row] = (u2[row] * q < p) ? 1 : 0;
    }
  }
}

__device__ double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = v;
  __syncthreads();
  double r = sh[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r += sh[i];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kBlock) void k_group_adv(const int32_t* __restrict__ accept, int G, int K,
                                                      int32_t* __restrict__ reward, float* __restrict__ adv,
                                                      float eps, int ddof, float clip) {
  __shared__ double sh[kWaves];
  const int64_t p = blockIdx.x;
  double lsum = 0.0;
  for (int g = threadIdx.x; g < G; g += kBlock) {
    const int32_t* a = accept + (p * G + g) * int64_t(K);
    int r = 0;
    while (r < K && a[r] != 0) ++r;
    reward[p * G + g] = r;
    lsum += double(r);
  }
  const double mean = block_sum_d(lsum, sh) / double(G);
  double lss = 0.0;
  for (int g = threadIdx.x; g < G; g += kBlock) {
    const double d = double(reward[p * G + g]) - mean;
    lss += d * d;
  }
  const double sd = sqrt(block_sum_d(lss, sh) / double(G - ddof));
  for (int g = threadIdx.x; g < G; g += kBlock) {
    double A = (double(reward[p * G + g]) - mean) / (sd + double(eps));
    if (clip > 0.f) A = fmin(fmax(A, -double(clip)), double(clip));
    adv[p * G + g] = float(A);
  }
}

template <class TI, bool VEC, int U>
hipError_t launch_rows(const SimArgs& a) {
  constexpr int E = VEC ? TI::kVec : 1;
  const int ng = a.V / E;
  const int ntiles = (ng + kWave * U - 1) / (kWave * U);
  const size_t lds = size_t(ntiles) * sizeof(float2);
  const int64_t rows = int64_t(a.P) * a.G * a.K;
  k_sim_rows<TI, VEC, U><<<dim3(unsigned(rows)), kBlock, lds, a.stream>>>(a.zd, a.zt, a.V, a.sc, a.u1, a.u2,
                                                                          a.token, a.accept);
  return hipGetLastError();
}

template <class TI>
hipError_t launch_rows_t(const SimArgs& a) {
  if (a.V % TI::kVec == 0) return launch_rows<TI, true, 2>(a);
  return launch_rows<TI, false, 8>(a);
}

}  // namespace

// Largest tile count: V <= 2^21 with 512-element tiles.
static_assert(sizeof(float2) * ((1 << 21) / 512) <= 32768, "tile table fits in 32 KiB of LDS");

hipError_t launch_sim(const SimArgs& a) {
  hipError_t e = (a.in == DType::kBf16) ? launch_rows_t<Bf16>(a) : launch_rows_t<F32>(a);
  if (e != hipSuccess) return e;
  k_group_adv<<<dim3(unsigned(a.P)), kBlock, 0, a.stream>>>(a.accept, a.G, a.K, a.reward, a.advantage, a.eps,
                                                           a.ddof, a.clip);
  return hipGetLastError();
}

}  // namespace aal
