// Multi-kernel streaming schedule for the EAL and WTV losses.
//
//   k_row_stats   one workgroup per logit row: max / sum-exp of the tempered
//                 draft (and target) logits; EAL: greedy target token and
//                 a = q(x*)  (Eq. acc_greedy); WTV: a second sweep for
//                 a = sum_v min(p, q) and Q< = sum_{q<p} q  (Eq. acc_sample).
//   k_window_scan one thread per window: prefix products P_j, E = sum_k P_k
//                 (Eq. eal_generic), suffix sums S_j and the gradient
//                 coefficient dloss/da_j = -P_j S_j / N  (Eqs. loss_eal, loss_tv).
//   k_loss        deterministic reduction loss = -(1/N) sum_n E_n.
//   k_grad        one workgroup per row: re-streams the logits and writes
//                 dloss/dz_draft through the softmax Jacobian.
//
// This schedule handles every shape; the register-resident schedule is the
// fast path for shapes it supports.
#include "aal_device.h"
#include "aal_internal.h"
#include "aal_rowops.h"

#include <limits.h>

namespace aal {
namespace {

constexpr int kBlock = kRowBlock;
constexpr int kWaves = kRowWaves;

template <class TI, int MODE, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void k_row_stats(const void* __restrict__ zd, const void* __restrict__ zt,
                                                      int V, float scd, float sct,
                                                      RowStats* __restrict__ stats) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  __shared__ LseState sh_lse[kWaves];
  __shared__ float sh_f[kWaves];
  __shared__ int sh_i[kWaves];

  const int64_t row = blockIdx.x;
  const int ng = V / E;
  const int64_t g0 = row * int64_t(ng);
  const int64_t e0 = row * int64_t(V);

  LseState sd = lse_init(), st = lse_init();
  float best = kNegInf;
  int bidx = INT_MAX;

  for (int base = threadIdx.x; base < ng; base += kBlock * U) {
    float xd[U][E], xt[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = base + u * kBlock;
      if (gi < ng) {
        Gr::load(zd, g0, gi, xd[u]);
        Gr::load(zt, g0, gi, xt[u]);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) xd[u][e] = xt[u][e] = kNegInf;
      }
    }
    float cm = kNegInf;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) cm = fmaxf(cm, xd[u][e]);
    if (lse_rebase(sd, cm, scd)) {
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) acc += ex2(__builtin_fmaf(xd[u][e], scd, -sd.msc));
      sd.s += acc;
    }
    if constexpr (MODE == int(Mode::kWtv)) {
      float ct = kNegInf;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) ct = fmaxf(ct, xt[u][e]);
      if (lse_rebase(st, ct, sct)) {
        float acc = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int e = 0; e < E; ++e) acc += ex2(__builtin_fmaf(xt[u][e], sct, -st.msc));
        st.s += acc;
      }
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (xt[u][e] > best) {
            best = xt[u][e];
            bidx = (base + u * kBlock) * E + e;
          }
    }
  }

  sd = block_lse(sd, scd, sh_lse);
  const float l2sd = __log2f(sd.s);
  RowStats out;
  out.msc_d = sd.msc;
  out.l2s_d = l2sd;
  out.coef = 0.f;
  if constexpr (MODE == int(Mode::kEal)) {
    int x = block_argmax(best, bidx, sh_f, sh_i);
    if (x == INT_MAX) x = 0;  // a row with no finite target logit: unspecified, stay in bounds
    const float zx = TI::load1(zd, e0 + x);
    out.a = ex2(__builtin_fmaf(zx, scd, -sd.msc) - l2sd);
    out.xstar = x;
    out.msc_t = 0.f;
    out.l2s_t = 0.f;
    out.qlt = 0.f;
  } else {
    st = block_lse(st, sct, sh_lse);
    const float l2st = __log2f(st.s);
    float smin = 0.f, qlt = 0.f;
    for (int base = threadIdx.x; base < ng; base += kBlock * U) {
      float xd[U][E], xt[U][E];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int gi = base + u * kBlock;
        if (gi < ng) {
          Gr::load(zd, g0, gi, xd[u]);
          Gr::load(zt, g0, gi, xt[u]);
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) xd[u][e] = xt[u][e] = kNegInf;
        }
      }
      float am = 0.f, aq = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float ld = __builtin_fmaf(xd[u][e], scd, -sd.msc) - l2sd;
          const float lt = __builtin_fmaf(xt[u][e], sct, -st.msc) - l2st;
          const float m = ex2(fminf(ld, lt));
          am += m;
          aq += (ld < lt) ? m : 0.f;
        }
      smin += am;
      qlt += aq;
    }
    smin = block_sum(smin, sh_f);
    qlt = block_sum(qlt, sh_f);
    out.a = smin;
    out.qlt = qlt;
    out.msc_t = st.msc;
    out.l2s_t = l2st;
    out.xstar = -1;
  }
  if (threadIdx.x == 0) stats[row] = out;
}

// One thread per window.  P_j = prod_{i<j} a_i, E = sum_{k=1..K} P_k,
// S_{K-1} = 1, S_j = 1 + a_{j+1} S_{j+1};  dE/da_j = P_j S_j.
__global__ __launch_bounds__(kBlock) void k_window_scan(RowStats* __restrict__ stats, int64_t N, int K, int mode,
                                                        float inv_t_d, const float* __restrict__ grad_scale,
                                                        float* __restrict__ window_e, float* __restrict__ accept,
                                                        int32_t* __restrict__ xstar) {
  const int64_t n = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (n >= N) return;
  RowStats* s = stats + n * K;
  double P[64];
  double p = 1.0, E = 0.0;
  for (int j = 0; j < K; ++j) {
    P[j] = p;
    p *= double(s[j].a);
    E += p;
  }
  const double scale = grad_scale ? double(*grad_scale) : 1.0;
  const double inv_n = 1.0 / double(N);
  double S = 1.0;
  for (int j = K - 1; j >= 0; --j) {
    const float a = s[j].a;
    const double g = -P[j] * S * inv_n;  // dloss/da_j
    const double factor = (mode == int(Mode::kEal)) ? double(a) * double(inv_t_d) : double(inv_t_d);
    s[j].coef = float(g * scale * factor);
    if (accept) accept[n * K + j] = a;
    if (xstar) xstar[n * K + j] = s[j].xstar;
    S = 1.0 + double(a) * S;
  }
  window_e[n] = float(E);
}

// err (may be null): a resident kernel's error word; set, the loss is NaN (a
// poll timed out and the per-window values are incomplete).
__global__ __launch_bounds__(kBlock) void k_loss(const float* __restrict__ window_e, int64_t N,
                                                 float* __restrict__ loss, const unsigned* __restrict__ err) {
  __shared__ double sh[kWaves];
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < N; i += kBlock) acc += double(window_e[i]);
  acc = wave_sum_d(acc);
  if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = sh[0];
    for (int i = 1; i < kWaves; ++i) t += sh[i];
    loss[0] = (err != nullptr && *err != 0u) ? __builtin_nanf("") : float(-t / double(N));
  }
}

template <class TI, class TG, int MODE, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void k_grad(const void* __restrict__ zd, const void* __restrict__ zt, int V,
                                                 float scd, float sct, const RowStats* __restrict__ stats,
                                                 void* __restrict__ grad) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  const int64_t row = blockIdx.x;
  const int ng = V / E;
  const int64_t g0 = row * int64_t(ng);
  const RowStats s = stats[row];
  const float c = s.coef;
  const float cA = c * (1.f - s.qlt);  // WTV, entries with q < p
  const float cB = -c * s.qlt;         // WTV, the others
  for (int base = threadIdx.x; base < ng; base += kBlock * U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = base + u * kBlock;
      if (gi >= ng) break;
      float xd[E], g[E];
      Gr::load(zd, g0, gi, xd);
      if constexpr (MODE == int(Mode::kEal)) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float q = ex2(__builtin_fmaf(xd[e], scd, -s.msc_d) - s.l2s_d);
          const float d = (gi * E + e == s.xstar) ? 1.f : 0.f;
          g[e] = c * (d - q);
        }
      } else {
        float xt[E];
        Gr::load(zt, g0, gi, xt);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float ld = __builtin_fmaf(xd[e], scd, -s.msc_d) - s.l2s_d;
          const float lt = __builtin_fmaf(xt[e], sct, -s.msc_t) - s.l2s_t;
          const float q = ex2(ld);
          g[e] = q * ((ld < lt) ? cA : cB);
        }
      }
      if constexpr (VEC) {
        store_vec<TG, E>(grad, (g0 + gi) * E, g);
      } else {
        TG::store1(grad, g0 + gi, g[0]);
      }
    }
  }
}

template <class TI, int MODE>
hipError_t launch_typed(const LossArgs& a) {
  const int64_t rows = a.N * a.K;
  const bool vec = (a.V % TI::kVec) == 0;
  constexpr int M = MODE;
  if (vec) {
    k_row_stats<TI, M, true, 4><<<dim3(unsigned(rows)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d, a.sc_t,
                                                                                a.ws.stats);
  } else {
    k_row_stats<TI, M, false, 8><<<dim3(unsigned(rows)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d, a.sc_t,
                                                                                 a.ws.stats);
  }
  const unsigned wblocks = unsigned((a.N + kBlock - 1) / kBlock);
  k_window_scan<<<wblocks, kBlock, 0, a.stream>>>(a.ws.stats, a.N, a.K, M, a.inv_t_d, a.grad_scale, a.window_e,
                                                  a.accept, a.xstar);
  k_loss<<<1, kBlock, 0, a.stream>>>(a.window_e, a.N, a.loss, nullptr);
  if (a.grad) {
    if (a.gd == DType::kBf16) {
      if (vec)
        k_grad<TI, GBf16, M, true, 4><<<dim3(unsigned(rows)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d,
                                                                                     a.sc_t, a.ws.stats, a.grad);
      else
        k_grad<TI, GBf16, M, false, 8><<<dim3(unsigned(rows)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d,
                                                                                      a.sc_t, a.ws.stats, a.grad);
    } else {
      if (vec)
        k_grad<TI, GF32, M, true, 4><<<dim3(unsigned(rows)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d,
                                                                                    a.sc_t, a.ws.stats, a.grad);
      else
        k_grad<TI, GF32, M, false, 8><<<dim3(unsigned(rows)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d,
                                                                                     a.sc_t, a.ws.stats, a.grad);
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_loss_reduce(const LossArgs& a, const unsigned* err) {
  k_loss<<<1, kBlock, 0, a.stream>>>(a.window_e, a.N, a.loss, err);
  return hipGetLastError();
}

hipError_t launch_streaming(const LossArgs& a) {
  if (a.in == DType::kBf16) {
    return a.mode == Mode::kEal ? launch_typed<Bf16, int(Mode::kEal)>(a) : launch_typed<Bf16, int(Mode::kWtv)>(a);
  }
  return a.mode == Mode::kEal ? launch_typed<F32, int(Mode::kEal)>(a) : launch_typed<F32, int(Mode::kWtv)>(a);
}

}  // namespace aal
