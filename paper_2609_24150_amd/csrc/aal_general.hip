// Combined training objectives over disjoint windows or over sequences with
// sliding windows (streaming schedule, every shape).
//
//   k_gen_rows  one workgroup per row: max / sum-exp of the tempered draft
//               (and target) logits; the greedy target token or the given
//               label and a_eal = q(x*) (Eq. acc_greedy); when a TV or KL
//               term is asked for, a second sweep for a_tv = sum_v min(p, q),
//               Q< = sum_{q<p} q (Eq. acc_sample) and KL(p || q).
//   k_gen_scan  one thread per row: the windows that contain the row (a
//               sequence's windows slide by one, Section "Window TV Loss"),
//               dE/da summed over them (Eq. eal_generic), the window-mean TV
//               and KL weights, and the row's gradient coefficients; the row
//               that starts a window also writes that window's E.
//   k_gen_loss_parts, k_gen_loss  the four terms and the weighted loss: 64
//               workgroups sum contiguous slices, one workgroup adds the 64
//               partial sums (a fixed summation order throughout).
//   k_gen_grad  one workgroup per row: dloss/dz_draft =
//               q (m ? cA : cB) + cP p + cX 1[v = x*].
#include "aal_device.h"
#include "aal_internal.h"
#include "aal_rowops.h"

#include <limits.h>

namespace aal {
namespace {

constexpr int kBlock = kRowBlock;
constexpr int kWaves = kRowWaves;
constexpr float kLn2 = 0.693147180559945309417f;

template <class TI, bool VEC, int U, bool NEED_T>
__global__ __launch_bounds__(kBlock) void k_gen_rows(const void* __restrict__ zd, const void* __restrict__ zt,
                                                     const int32_t* __restrict__ labels, int V, float scd,
                                                     float sct, int want_eal, int want_pq, int want_kl,
                                                     GenStats* __restrict__ stats) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  __shared__ LseState sh_lse[kWaves];
  __shared__ float sh_f[kWaves];
  __shared__ int sh_i[kWaves];

  const int64_t row = blockIdx.x;
  const int ng = V / E;
  const int64_t g0 = row * int64_t(ng);
  const int64_t e0 = row * int64_t(V);
  const bool argmax = NEED_T && want_eal && labels == nullptr;

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
        if constexpr (NEED_T) Gr::load(zt, g0, gi, xt[u]);
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
    if constexpr (NEED_T) {
      if (want_pq) {
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
      }
      if (argmax) {
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
  }

  sd = block_lse(sd, scd, sh_lse);
  const float l2sd = __log2f(sd.s);
  GenStats out{};
  out.msc_d = sd.msc;
  out.l2s_d = l2sd;
  out.xstar = -1;
  if (want_eal) {
    int x;
    if (labels != nullptr) {
      x = min(max(labels[row], 0), V - 1);  // out-of-range labels are clamped
    } else {
      x = block_argmax(best, bidx, sh_f, sh_i);
      if (x == INT_MAX) x = 0;  // no finite target logit: unspecified, stay in bounds
    }
    const float zx = TI::load1(zd, e0 + x);
    out.a_eal = ex2(__builtin_fmaf(zx, scd, -sd.msc) - l2sd);
    out.xstar = x;
  }
  if (NEED_T && want_pq) {
    st = block_lse(st, sct, sh_lse);
    const float l2st = __log2f(st.s);
    float smin = 0.f, qlt = 0.f, kl = 0.f;
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
      float am = 0.f, aq = 0.f, ak = 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float ld = __builtin_fmaf(xd[u][e], scd, -sd.msc) - l2sd;  // log2 q
          const float lt = __builtin_fmaf(xt[u][e], sct, -st.msc) - l2st;  // log2 p
          const float m = ex2(fminf(ld, lt));
          am += m;
          aq += (ld < lt) ? m : 0.f;
          if (want_kl) {
            const float pv = ex2(lt);
            ak += (pv > 0.f) ? pv * (lt - ld) : 0.f;  // p = 0 (masked) contributes nothing
          }
        }
      smin += am;
      qlt += aq;
      kl += ak;
    }
    smin = block_sum(smin, sh_f);
    qlt = block_sum(qlt, sh_f);
    if (want_kl) kl = block_sum(kl, sh_f);
    out.a_tv = smin;
    out.qlt = qlt;
    out.kl = kl * kLn2;
    out.msc_t = st.msc;
    out.l2s_t = l2st;
  }
  if (threadIdx.x == 0) stats[row] = out;
}

// dE/da of position j of the window whose rows start at `r0` (stride 1):
// prod_{i<j} a_i * (1 + a_{j+1} (1 + a_{j+2} (...))), in fp64.
__device__ double window_dE(const GenStats* __restrict__ st, int64_t r0, int K, int j, bool eal) {
  double P = 1.0;
  for (int i = 0; i < j; ++i) P *= double(eal ? st[r0 + i].a_eal : st[r0 + i].a_tv);
  double S = 1.0;
  for (int i = K - 1; i > j; --i) S = 1.0 + double(eal ? st[r0 + i].a_eal : st[r0 + i].a_tv) * S;
  return P * S;
}

__device__ double window_E(const GenStats* __restrict__ st, int64_t r0, int K, bool eal) {
  double p = 1.0, E = 0.0;
  for (int i = 0; i < K; ++i) {
    p *= double(eal ? st[r0 + i].a_eal : st[r0 + i].a_tv);
    E += p;
  }
  return E;
}

struct ScanParams {
  GenStats* stats;
  int layout;
  int64_t B;
  int S, K;
  int64_t R, W;
  float w_wtv, w_eal, w_kl, w_tv;
  float inv_t_d;
  const float* grad_scale;
  float* win_tv;  // [W] (workspace)
  float* win_eal; // [W] (workspace)
  float* e_tv;    // user outputs, may be null
  float* e_eal;
  float* accept_tv;
  float* accept_eal;
  int32_t* xstar;
};

__global__ __launch_bounds__(kBlock) void k_gen_scan(ScanParams p) {
  const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (r >= p.R) return;
  const int K = p.K;
  // windows containing row r: starts t0..t1 (in row units r0 = base + t), position j = s - t
  int64_t base;
  int s, t0, t1;
  int64_t wbase;  // window index of start t = 0 of this sequence / window
  if (p.layout == 0) {
    base = (r / K) * K;
    s = int(r - base);
    t0 = t1 = 0;
    wbase = r / K;
  } else {
    const int64_t b = r / p.S;
    base = b * p.S;
    s = int(r - base);
    t0 = max(0, s - K + 1);
    t1 = min(s, p.S - K);  // empty (t1 < t0) when S < K
    wbase = b * int64_t(max(0, p.S - K + 1));
  }
  const bool tv = p.w_wtv != 0.f || p.w_tv != 0.f;
  const bool eal = p.w_eal != 0.f;
  double dtv = 0.0, deal = 0.0, count = 0.0;
  for (int t = t0; t <= t1; ++t) {
    const int64_t r0 = base + (p.layout == 0 ? 0 : t);
    if (tv) dtv += window_dE(p.stats, r0, K, s - t, false);
    if (eal) deal += window_dE(p.stats, r0, K, s - t, true);
    count += 1.0;
  }
  GenStats& st = p.stats[r];
  const double W = double(p.W), R = double(p.R);
  const double scale = p.grad_scale ? double(*p.grad_scale) : 1.0;
  const double g_tv = p.W > 0 ? (-double(p.w_wtv) * dtv - double(p.w_tv) * count / K) / W : 0.0;
  const double g_eal = p.W > 0 ? -double(p.w_eal) * deal / W : 0.0;
  const double g_kl = double(p.w_kl) / R;
  const double f = scale * double(p.inv_t_d);
  const double c_tv = g_tv * f, c_eal = g_eal * double(st.a_eal) * f, c_kl = g_kl * f;
  st.cA = float(c_tv * (1.0 - double(st.qlt)) - c_eal + c_kl);
  st.cB = float(-c_tv * double(st.qlt) - c_eal + c_kl);
  st.cX = float(c_eal);
  st.cP = float(-c_kl);
  st.tv_w = float(count * (1.0 - double(st.a_tv)));  // this row's share of sum_w sum_j TV
  if (p.accept_tv) p.accept_tv[r] = st.a_tv;
  if (p.accept_eal) p.accept_eal[r] = st.a_eal;
  if (p.xstar) p.xstar[r] = st.xstar;
  // the window that starts at this row
  const bool starts = p.layout == 0 ? s == 0 : (s <= p.S - K);
  if (starts) {
    const int64_t w = wbase + (p.layout == 0 ? 0 : s);
    const float etv = tv || p.e_tv ? float(window_E(p.stats, r, K, false)) : 0.f;
    const float eeal = eal || p.e_eal ? float(window_E(p.stats, r, K, true)) : 0.f;
    p.win_tv[w] = etv;
    p.win_eal[w] = eeal;
    if (p.e_tv) p.e_tv[w] = etv;
    if (p.e_eal) p.e_eal[w] = eeal;
  }
}

__device__ double block_sum_d(double v, double* sh) {
  v = wave_sum_d(v);
  if ((threadIdx.x & (kWave - 1)) == 0) sh[threadIdx.x / kWave] = v;
  __syncthreads();
  double t = sh[0];
  for (int i = 1; i < kWaves; ++i) t += sh[i];
  __syncthreads();
  return t;
}

// Block b sums windows and rows of its contiguous slice.
__global__ __launch_bounds__(kBlock) void k_gen_loss_parts(const GenStats* __restrict__ stats,
                                                           const float* __restrict__ win_tv,
                                                           const float* __restrict__ win_eal, int64_t R, int64_t W,
                                                           double* __restrict__ parts) {
  __shared__ double sh[kWaves];
  const int64_t b = blockIdx.x;
  const int64_t w0 = W * b / kGenLossParts, w1 = W * (b + 1) / kGenLossParts;
  const int64_t r0 = R * b / kGenLossParts, r1 = R * (b + 1) / kGenLossParts;
  double etv = 0.0, eeal = 0.0, kl = 0.0, tvs = 0.0;
  for (int64_t i = w0 + threadIdx.x; i < w1; i += kBlock) {
    etv += double(win_tv[i]);
    eeal += double(win_eal[i]);
  }
  for (int64_t i = r0 + threadIdx.x; i < r1; i += kBlock) {
    kl += double(stats[i].kl);
    tvs += double(stats[i].tv_w);
  }
  etv = block_sum_d(etv, sh);
  eeal = block_sum_d(eeal, sh);
  kl = block_sum_d(kl, sh);
  tvs = block_sum_d(tvs, sh);
  if (threadIdx.x == 0) {
    parts[b * 4 + 0] = etv;
    parts[b * 4 + 1] = eeal;
    parts[b * 4 + 2] = kl;
    parts[b * 4 + 3] = tvs;
  }
}

__global__ void k_gen_loss(const double* __restrict__ parts, int64_t R, int64_t W, int K, float w_wtv, float w_eal,
                           float w_kl, float w_tv, float* __restrict__ loss, float* __restrict__ terms,
                           const unsigned* __restrict__ err) {
  if (threadIdx.x == 0) {
    double etv = 0.0, eeal = 0.0, kl = 0.0, tvs = 0.0;
    for (int b = 0; b < kGenLossParts; ++b) {
      etv += parts[b * 4 + 0];
      eeal += parts[b * 4 + 1];
      kl += parts[b * 4 + 2];
      tvs += parts[b * 4 + 3];
    }
    // a term whose weight is 0 is not evaluated (its inputs may not be)
    const double t0 = W > 0 && w_wtv != 0.f ? -etv / double(W) : 0.0;
    const double t1 = W > 0 && w_eal != 0.f ? -eeal / double(W) : 0.0;
    const double t2 = w_kl != 0.f ? kl / double(R) : 0.0;
    const double t3 = W > 0 && w_tv != 0.f ? tvs / (double(W) * K) : 0.0;
    // a set error word (a resident kernel's poll timed out): NaN
    loss[0] = (err != nullptr && *err != 0u) ? __builtin_nanf("")
                                             : float(double(w_wtv) * t0 + double(w_eal) * t1 + double(w_kl) * t2 +
                                                     double(w_tv) * t3);
    if (terms) {
      terms[0] = float(t0);
      terms[1] = float(t1);
      terms[2] = float(t2);
      terms[3] = float(t3);
    }
  }
}

template <class TI, class TG, bool VEC, int U, bool NEED_P>
__global__ __launch_bounds__(kBlock) void k_gen_grad(const void* __restrict__ zd, const void* __restrict__ zt, int V,
                                                     float scd, float sct, const GenStats* __restrict__ stats,
                                                     void* __restrict__ grad) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  const int64_t row = blockIdx.x;
  const int ng = V / E;
  const int64_t g0 = row * int64_t(ng);
  const GenStats s = stats[row];
  for (int base = threadIdx.x; base < ng; base += kBlock * U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int gi = base + u * kBlock;
      if (gi >= ng) break;
      float xd[E], g[E];
      Gr::load(zd, g0, gi, xd);
      if constexpr (NEED_P) {
        float xt[E];
        Gr::load(zt, g0, gi, xt);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float ld = __builtin_fmaf(xd[e], scd, -s.msc_d) - s.l2s_d;
          const float lt = __builtin_fmaf(xt[e], sct, -s.msc_t) - s.l2s_t;
          g[e] = ex2(ld) * ((ld < lt) ? s.cA : s.cB) + s.cP * ex2(lt);
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) g[e] = ex2(__builtin_fmaf(xd[e], scd, -s.msc_d) - s.l2s_d) * s.cB;
      }
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (gi * E + e == s.xstar) g[e] += s.cX;
      if constexpr (VEC) {
        store_vec<TG, E>(grad, (g0 + gi) * E, g);
      } else {
        TG::store1(grad, g0 + gi, g[0]);
      }
    }
  }
}

template <class TI, bool VEC, int U, bool NEED_T>
void rows_launch(const GenArgs& a, const GenStats* unused) {
  (void)unused;
  k_gen_rows<TI, VEC, U, NEED_T><<<dim3(unsigned(a.R)), kBlock, 0, a.stream>>>(
      a.zd, a.zt, a.labels, a.V, a.sc_d, a.sc_t, a.w_eal != 0.f, a.w_wtv != 0.f || a.w_tv != 0.f || a.w_kl != 0.f,
      a.w_kl != 0.f, a.stats);
}

template <class TI, class TG, bool VEC, int U>
void grad_launch(const GenArgs& a, bool need_p) {
  if (need_p)
    k_gen_grad<TI, TG, VEC, U, true><<<dim3(unsigned(a.R)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d, a.sc_t,
                                                                                  a.stats, a.grad);
  else
    k_gen_grad<TI, TG, VEC, U, false><<<dim3(unsigned(a.R)), kBlock, 0, a.stream>>>(a.zd, a.zt, a.V, a.sc_d, a.sc_t,
                                                                                   a.stats, a.grad);
}

template <class TI>
hipError_t launch_typed(const GenArgs& a) {
  const bool vec = (a.V % TI::kVec) == 0;
  const bool need_pq = a.w_wtv != 0.f || a.w_tv != 0.f || a.w_kl != 0.f;
  const bool need_t = need_pq || (a.w_eal != 0.f && a.labels == nullptr);
  if (vec) {
    if (need_t) rows_launch<TI, true, 4, true>(a, nullptr);
    else rows_launch<TI, true, 4, false>(a, nullptr);
  } else {
    if (need_t) rows_launch<TI, false, 8, true>(a, nullptr);
    else rows_launch<TI, false, 8, false>(a, nullptr);
  }
  ScanParams sp{};
  sp.stats = a.stats;
  sp.layout = a.layout;
  sp.B = a.B;
  sp.S = a.S;
  sp.K = a.K;
  sp.R = a.R;
  sp.W = a.W;
  sp.w_wtv = a.w_wtv;
  sp.w_eal = a.w_eal;
  sp.w_kl = a.w_kl;
  sp.w_tv = a.w_tv;
  sp.inv_t_d = a.inv_t_d;
  sp.grad_scale = a.grad_scale;
  sp.win_tv = a.win_tv;
  sp.win_eal = a.win_eal;
  sp.e_tv = a.e_tv;
  sp.e_eal = a.e_eal;
  sp.accept_tv = a.accept_tv;
  sp.accept_eal = a.accept_eal;
  sp.xstar = a.xstar;
  k_gen_scan<<<dim3(unsigned((a.R + kBlock - 1) / kBlock)), kBlock, 0, a.stream>>>(sp);
  if (hipError_t e = launch_general_loss(a); e != hipSuccess) return e;
  if (a.grad) {
    if (a.gd == DType::kBf16) {
      if (vec) grad_launch<TI, GBf16, true, 4>(a, need_pq);
      else grad_launch<TI, GBf16, false, 8>(a, need_pq);
    } else {
      if (vec) grad_launch<TI, GF32, true, 4>(a, need_pq);
      else grad_launch<TI, GF32, false, 8>(a, need_pq);
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_general_loss(const GenArgs& a, const unsigned* err) {
  k_gen_loss_parts<<<kGenLossParts, kBlock, 0, a.stream>>>(a.stats, a.win_tv, a.win_eal, a.R, a.W, a.loss_parts);
  k_gen_loss<<<1, 64, 0, a.stream>>>(a.loss_parts, a.R, a.W, a.K, a.w_wtv, a.w_eal, a.w_kl, a.w_tv, a.loss,
                                     a.terms, err);
  return hipGetLastError();
}

hipError_t launch_general_resident(const GenArgs& a, bool* used) {
  *used = false;
  const int E = a.in == DType::kBf16 ? Bf16::kVec : F32::kVec;
  if (a.V % E != 0 || a.zt == nullptr || a.res_slots == nullptr) return hipSuccess;
  return a.in == DType::kBf16 ? launch_general_resident_bf16(a, used) : launch_general_resident_f32(a, used);
}

hipError_t launch_general(const GenArgs& a) {
  if (!a.streaming) {
    bool used = false;
    if (hipError_t e = launch_general_resident(a, &used); e != hipSuccess) return e;
    if (used) {
      return launch_general_loss(a, a.res_err);  // NaN loss if a poll timed out
    }
  }
  return a.in == DType::kBf16 ? launch_typed<Bf16>(a) : launch_typed<F32>(a);
}

}  // namespace aal
