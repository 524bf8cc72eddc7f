// GRPO loss on the simulated greedy acceptance length (Section "GRPO Loss on
// Acceptance Length"), forward and backward w.r.t. the current draft logits.
//
//   k_grpo_rows    one workgroup per row, three logit sets: greedy tokens of
//                  the current draft S^theta and the reference draft S^ref,
//                  the target's greedy token x* (or a given label), and the
//                  log-probabilities log pi_theta(S^theta), log pi_ref(S^theta)
//                  at the common temperature.
//   k_grpo_groups  one thread per group of m windows: accepted lengths
//                  tau^theta, tau^ref, the debiased reward (Eq.
//                  debiased_reward), the clipped per-token geometric-mean
//                  ratio, the group advantage (Eq. advantage), the clipped
//                  surrogate and dloss/dlog rho of every window.
//   k_grpo_loss    one workgroup: mean of the group losses, fixed order.
//   k_grpo_grad    one workgroup per row: the row's share of dloss/dlog rho,
//                  summed over the windows that contain it, times the
//                  log-softmax Jacobian (1/T)(1[v = S^theta] - pi_theta(v)).
#include "aal_device.h"
#include "aal_grpo_math.h"
#include "aal_internal.h"
#include "aal_rowops.h"

#include <limits.h>

namespace aal {
namespace {

constexpr int kBlock = kRowBlock;
constexpr int kWaves = kRowWaves;
constexpr float kLn2 = 0.693147180559945309417f;

template <class TI, bool VEC, int U, bool TARGET>
__global__ __launch_bounds__(kBlock) void k_grpo_rows(const void* __restrict__ zth, const void* __restrict__ zrf,
                                                      const void* __restrict__ zt, const int32_t* __restrict__ labels,
                                                      int V, float sc, GrpoRow* __restrict__ rows) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  __shared__ LseState sh_lse[kWaves];
  __shared__ float sh_f[kWaves];
  __shared__ int sh_i[kWaves];

  const int64_t row = blockIdx.x;
  const int ng = V / E;
  const int64_t g0 = row * int64_t(ng);
  const int64_t e0 = row * int64_t(V);

  LseState sth = lse_init(), srf = lse_init();
  float bth = kNegInf, brf = kNegInf, bt = kNegInf;
  int ith = INT_MAX, irf = INT_MAX, it = INT_MAX;
  for (int base = threadIdx.x; base < ng; base += kBlock * U) {
    float xa[U][E], xb[U][E], xc[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = base + u * kBlock;
      if (gi < ng) {
        Gr::load(zth, g0, gi, xa[u]);
        Gr::load(zrf, g0, gi, xb[u]);
        if constexpr (TARGET) Gr::load(zt, g0, gi, xc[u]);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) xa[u][e] = xb[u][e] = xc[u][e] = kNegInf;
      }
    }
    float ca = kNegInf, cb = kNegInf;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) {
        ca = fmaxf(ca, xa[u][e]);
        cb = fmaxf(cb, xb[u][e]);
        const int idx = (base + u * kBlock) * E + e;
        if (xa[u][e] > bth) { bth = xa[u][e]; ith = idx; }
        if (xb[u][e] > brf) { brf = xb[u][e]; irf = idx; }
        if constexpr (TARGET) {
          if (xc[u][e] > bt) { bt = xc[u][e]; it = idx; }
        }
      }
    if (lse_rebase(sth, ca, sc)) {
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) acc += ex2(__builtin_fmaf(xa[u][e], sc, -sth.msc));
      sth.s += acc;
    }
    if (lse_rebase(srf, cb, sc)) {
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) acc += ex2(__builtin_fmaf(xb[u][e], sc, -srf.msc));
      srf.s += acc;
    }
  }
  sth = block_lse(sth, sc, sh_lse);
  srf = block_lse(srf, sc, sh_lse);
  int s_th = block_argmax(bth, ith, sh_f, sh_i);
  int s_rf = block_argmax(brf, irf, sh_f, sh_i);
  int xs;
  if constexpr (TARGET) {
    xs = block_argmax(bt, it, sh_f, sh_i);
    if (xs == INT_MAX) xs = 0;
  } else {
    xs = min(max(labels[row], 0), V - 1);  // out-of-range labels are clamped
  }
  if (s_th == INT_MAX) s_th = 0;  // no finite logit: unspecified, stay in bounds
  if (s_rf == INT_MAX) s_rf = 0;
  if (threadIdx.x == 0) {
    const float l2th = __log2f(sth.s), l2rf = __log2f(srf.s);
    const float za = TI::load1(zth, e0 + s_th);
    const float zb = TI::load1(zrf, e0 + s_th);  // the reference at the current draft's token
    GrpoRow o{};
    o.s_theta = s_th;
    o.s_ref = s_rf;
    o.xstar = xs;
    o.lp_theta = (__builtin_fmaf(za, sc, -sth.msc) - l2th) * kLn2;
    o.lp_ref = (__builtin_fmaf(zb, sc, -srf.msc) - l2rf) * kLn2;
    o.msc = sth.msc;
    o.l2s = l2th;
    rows[row] = o;
  }
}

struct GroupParams {
  const GrpoRow* rows;
  int layout;
  int64_t n_groups;
  int G, S, m, K;
  const int32_t* anchors;  // sequences layout
  float eps, adv_clip, eps_clip, rho_min, rho_max;
  float* win_coef;   // [n_groups * m] dloss / dlog rho
  float* group_loss; // [n_groups]
  int32_t* tau_theta;  // optional outputs [n_groups * m]
  int32_t* tau_ref;
  float* advantage;
  float* log_rho;
};

// First row of window i of group gi.
__device__ __forceinline__ int64_t window_row0(const GroupParams& p, int64_t gi, int i) {
  if (p.layout == 0) return (gi * p.m + i) * int64_t(p.K);
  const int64_t b = gi / p.G;
  const int a = min(max(p.anchors[gi], 0), p.S - (p.m - 1) - p.K);  // clamped into the sequence
  return b * p.S + a + i;
}

__global__ __launch_bounds__(kBlock) void k_grpo_groups(GroupParams p) {
  const int64_t gi = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (gi >= p.n_groups) return;
  const int m = p.m;
  auto row_at = [&](int i, int k) {
    const GrpoRow& w = p.rows[window_row0(p, gi, i) + k];
    return GrpoRowIn{w.s_theta, w.s_ref, w.xstar, w.lp_theta, w.lp_ref};
  };
  p.group_loss[gi] = float(grpo_group(m, p.K, row_at, p.eps, p.adv_clip, p.eps_clip, p.rho_min, p.rho_max,
                                      1.0 / (double(p.n_groups) * m), p.win_coef + gi * m,
                                      p.tau_theta ? p.tau_theta + gi * m : nullptr,
                                      p.tau_ref ? p.tau_ref + gi * m : nullptr,
                                      p.advantage ? p.advantage + gi * m : nullptr,
                                      p.log_rho ? p.log_rho + gi * m : nullptr));
}

__global__ __launch_bounds__(kBlock) void k_grpo_loss(const float* __restrict__ group_loss, int64_t n,
                                                      float* __restrict__ loss) {
  __shared__ double sh[kWaves];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += kBlock) acc += double(group_loss[i]);
  acc = wave_sum_d(acc);
  if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = sh[0];
    for (int i = 1; i < kWaves; ++i) t += sh[i];
    loss[0] = float(t / double(n));
  }
}

template <class TI, class TG, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void k_grpo_grad(const void* __restrict__ zth, int V, float sc, float inv_t,
                                                      const float* __restrict__ grad_scale, GroupParams p,
                                                      void* __restrict__ grad) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  __shared__ float sh_c;
  const int64_t row = blockIdx.x;
  const GrpoRow s = p.rows[row];
  if (threadIdx.x == 0) {
    // the row's share (1/K) of dloss/dlog rho of every window that contains it
    double c = 0.0;
    if (p.layout == 0) {
      const int64_t w = row / p.K;
      c = double(p.win_coef[w]);
    } else {
      const int64_t b = row / p.S;
      const int pos = int(row - b * p.S);
      for (int g = 0; g < p.G; ++g) {
        const int64_t gi = b * p.G + g;
        const int a = min(max(p.anchors[gi], 0), p.S - (p.m - 1) - p.K);
        const int i0 = max(0, pos - a - p.K + 1), i1 = min(p.m - 1, pos - a);
        for (int i = i0; i <= i1; ++i) c += double(p.win_coef[gi * p.m + i]);
      }
    }
    const double scale = grad_scale ? double(*grad_scale) : 1.0;
    sh_c = float(c / p.K * scale * double(inv_t));
  }
  __syncthreads();
  const float c = sh_c;
  const int ng = V / E;
  const int64_t g0 = row * int64_t(ng);
  for (int base = threadIdx.x; base < ng; base += kBlock * U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = base + u * kBlock;
      if (gi >= ng) break;
      float x[E], g[E];
      Gr::load(zth, g0, gi, x);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float pv = ex2(__builtin_fmaf(x[e], sc, -s.msc) - s.l2s);
        g[e] = c * (((gi * E + e) == s.s_theta ? 1.f : 0.f) - pv);
      }
      if constexpr (VEC) {
        store_vec<TG, E>(grad, (g0 + gi) * E, g);
      } else {
        TG::store1(grad, g0 + gi, g[0]);
      }
    }
  }
}

template <class TI, class TG, bool VEC, int U>
void grad_launch(const GrpoArgs& a, const GroupParams& gp) {
  k_grpo_grad<TI, TG, VEC, U><<<dim3(unsigned(a.R)), kBlock, 0, a.stream>>>(a.zth, a.V, a.sc, a.inv_t,
                                                                           a.grad_scale, gp, a.grad);
}

template <class TI>
hipError_t launch_typed(const GrpoArgs& a) {
  const bool vec = (a.V % TI::kVec) == 0;
  const bool tgt = a.labels == nullptr;
  const unsigned R = unsigned(a.R);
  if (vec) {
    if (tgt) k_grpo_rows<TI, true, 2, true><<<R, kBlock, 0, a.stream>>>(a.zth, a.zrf, a.zt, a.labels, a.V, a.sc, a.rows);
    else k_grpo_rows<TI, true, 2, false><<<R, kBlock, 0, a.stream>>>(a.zth, a.zrf, a.zt, a.labels, a.V, a.sc, a.rows);
  } else {
    if (tgt) k_grpo_rows<TI, false, 4, true><<<R, kBlock, 0, a.stream>>>(a.zth, a.zrf, a.zt, a.labels, a.V, a.sc, a.rows);
    else k_grpo_rows<TI, false, 4, false><<<R, kBlock, 0, a.stream>>>(a.zth, a.zrf, a.zt, a.labels, a.V, a.sc, a.rows);
  }
  GroupParams gp{};
  gp.rows = a.rows;
  gp.layout = a.layout;
  gp.n_groups = a.n_groups;
  gp.G = a.G;
  gp.S = a.S;
  gp.m = a.m;
  gp.K = a.K;
  gp.anchors = a.anchors;
  gp.eps = a.eps;
  gp.adv_clip = a.adv_clip;
  gp.eps_clip = a.eps_clip;
  gp.rho_min = a.rho_min;
  gp.rho_max = a.rho_max;
  gp.win_coef = a.win_coef;
  gp.group_loss = a.group_loss;
  gp.tau_theta = a.tau_theta;
  gp.tau_ref = a.tau_ref;
  gp.advantage = a.advantage;
  gp.log_rho = a.log_rho;
  k_grpo_groups<<<dim3(unsigned((a.n_groups + kBlock - 1) / kBlock)), kBlock, 0, a.stream>>>(gp);
  k_grpo_loss<<<1, kBlock, 0, a.stream>>>(a.group_loss, a.n_groups, a.loss);
  if (a.grad) {
    if (a.gd == DType::kBf16) {
      if (vec) grad_launch<TI, GBf16, true, 4>(a, gp);
      else grad_launch<TI, GBf16, false, 8>(a, gp);
    } else {
      if (vec) grad_launch<TI, GF32, true, 4>(a, gp);
      else grad_launch<TI, GF32, false, 8>(a, gp);
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_grpo(const GrpoArgs& a) {
  return a.in == DType::kBf16 ? launch_typed<Bf16>(a) : launch_typed<F32>(a);
}

}  // namespace aal
