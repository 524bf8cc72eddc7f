// Vocabulary-parallel pieces of the EAL and WTV losses: what one rank of a
// tensor-parallel LM head computes on its contiguous slice of the vocabulary.
//
//   k_vp_partials  one workgroup per row of the slice: (max, sum-exp) of the
//                  tempered draft and, for WTV, target logits; for EAL the
//                  slice's greedy target candidate with the draft logit there.
//   k_vp_merge     one thread per row: the gathered partials of all slices
//                  merged in rank order into the row's normalisers and, for
//                  EAL, x* and a = q(x*)  (Eq. acc_greedy).
//   k_vp_accept    one workgroup per row (WTV): the slice's part of
//                  sum_v min(p, q) and of Q< with the merged normalisers
//                  (Eq. acc_sample).
//   k_vp_scan      one thread per window: WTV's partials summed in rank order,
//                  then prefix products, E = sum_k P_k (Eq. eal_generic) and
//                  the coefficients dloss/da_j = -P_j S_j / N (Eqs. loss_eal,
//                  loss_tv); the loss is reduced afterwards in fixed order.
//   k_vp_seq_scan  the same for sequences with windows sliding by one: one
//                  thread per row sums dE/da over the windows that contain it.
//   k_vp_grad      one workgroup per row: the slice of dloss/dz_draft.
//
// A slice is HBM-bound like the streaming schedule it mirrors: the partial
// pass reads both slices once, the acceptance pass (WTV) reads them again
// with the merged normalisers, the gradient pass reads them and writes the
// gradient.  The exchange between passes is a few bytes per row.
#include "aal_device.h"
#include "aal_rowops.h"
#include "aal_vp.h"

#include <limits.h>

namespace aal {
namespace {

constexpr int kBlock = kRowBlock;
constexpr int kWaves = kRowWaves;
constexpr int kMaxRowBlocks = 65536;  // rows beyond this are visited grid-stride

unsigned row_grid(int64_t rows) { return unsigned(rows < kMaxRowBlocks ? rows : kMaxRowBlocks); }

// LAB (EAL with labels): the label replaces the greedy token and the target
// slice is not read.
template <class TI, int MODE, bool VEC, int U, bool LAB>
__global__ __launch_bounds__(kBlock) void k_vp_partials(const void* __restrict__ zd, const void* __restrict__ zt,
                                                        const int32_t* __restrict__ labels, int64_t rows, int Vs,
                                                        int v0, int vtot, float scd, float sct,
                                                        aal_vp_part_t* __restrict__ parts) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  __shared__ LseState sh_lse[kWaves];
  __shared__ float sh_f[kWaves];
  __shared__ int sh_i[kWaves];
  const int ng = Vs / E;

  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const int64_t g0 = row * int64_t(ng);
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
          if constexpr (!LAB) Gr::load(zt, g0, gi, xt[u]);
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
      } else if constexpr (!LAB) {
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
    aal_vp_part_t out;
    out.zmax_d = sd.m;
    out.s_d = sd.s;
    out.reserved0 = 0;
    out.reserved1 = 0;
    if constexpr (LAB) {
      // the label clamped into the vocabulary [0, vtot), as the fused calls
      // clamp it, then in slice coordinates
      const int64_t xl = int64_t(min(max(labels[row], 0), vtot - 1)) - v0;
      if (xl >= 0 && xl < Vs) {
        out.zmax_t = 0.f;  // the only candidate of the row: its value decides nothing
        out.zd_at = TI::load1(zd, row * int64_t(Vs) + xl);
        out.t_idx = int(xl) + v0;
      } else {
        out.zmax_t = kNegInf;
        out.zd_at = 0.f;
        out.t_idx = INT_MAX;
      }
      out.s_t = 0.f;
    } else if constexpr (MODE == int(Mode::kEal)) {
      const int x = block_argmax(best, bidx, sh_f, sh_i);
      const int64_t e0 = row * int64_t(Vs);
      if (x == INT_MAX) {
        out.zmax_t = kNegInf;
        out.zd_at = 0.f;
        out.t_idx = INT_MAX;
      } else {
        out.zmax_t = TI::load1(zt, e0 + x);
        out.zd_at = TI::load1(zd, e0 + x);
        out.t_idx = v0 + x;
      }
      out.s_t = 0.f;
    } else {
      st = block_lse(st, sct, sh_lse);
      out.zmax_t = st.m;
      out.s_t = st.s;
      out.zd_at = 0.f;
      out.t_idx = -1;
    }
    if (threadIdx.x == 0) parts[row] = out;
  }
}

// Sum over slices of s_r 2^(fl(zmax_r sc) - fl(M sc)), M = max_r zmax_r, in
// rank order.  Returns fl(M sc) in *msc and log2 of the sum.
__device__ __forceinline__ float merge_lse(const aal_vp_part_t* __restrict__ parts, int R, int64_t rows, int64_t row,
                                           bool target, float sc, float* msc) {
  float M = kNegInf;
  for (int r = 0; r < R; ++r) {
    const aal_vp_part_t& p = parts[int64_t(r) * rows + row];
    M = fmaxf(M, target ? p.zmax_t : p.zmax_d);
  }
  const float mref = M * sc;
  float s = 0.f;
  for (int r = 0; r < R; ++r) {
    const aal_vp_part_t& p = parts[int64_t(r) * rows + row];
    const float zm = target ? p.zmax_t : p.zmax_d;
    const float sr = target ? p.s_t : p.s_d;
    if (zm != kNegInf) s += sr * ex2(zm * sc - mref);
  }
  *msc = mref;
  return __log2f(s);
}

__global__ __launch_bounds__(kBlock) void k_vp_merge(const aal_vp_part_t* __restrict__ parts, int R, int64_t rows,
                                                     int mode, float scd, float sct, aal_vp_row_t* __restrict__ out) {
  const int64_t row = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (row >= rows) return;
  aal_vp_row_t o;
  o.l2s_d = merge_lse(parts, R, rows, row, false, scd, &o.msc_d);
  o.qlt = 0.f;
  o.coef = 0.f;
  if (mode == int(Mode::kEal)) {
    // largest target logit, lowest global index among equal ones
    float bv = kNegInf, bz = 0.f;
    int bi = INT_MAX;
    for (int r = 0; r < R; ++r) {
      const aal_vp_part_t& p = parts[int64_t(r) * rows + row];
      if (p.t_idx != INT_MAX && (p.zmax_t > bv || (p.zmax_t == bv && p.t_idx < bi))) {
        bv = p.zmax_t;
        bi = p.t_idx;
        bz = p.zd_at;
      }
    }
    o.msc_t = 0.f;
    o.l2s_t = 0.f;
    if (bi == INT_MAX) {  // no finite target logit in the row: unspecified, stay in bounds
      o.xstar = 0;
      o.a = 0.f;
    } else {
      o.xstar = bi;
      o.a = ex2(__builtin_fmaf(bz, scd, -o.msc_d) - o.l2s_d);
    }
  } else {
    o.l2s_t = merge_lse(parts, R, rows, row, true, sct, &o.msc_t);
    o.a = 0.f;
    o.xstar = -1;
  }
  out[row] = o;
}

template <class TI, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void k_vp_accept(const void* __restrict__ zd, const void* __restrict__ zt,
                                                      int64_t rows, int Vs, float scd, float sct,
                                                      const aal_vp_row_t* __restrict__ rec,
                                                      aal_vp_acc_t* __restrict__ acc) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  __shared__ float sh_f[kWaves];
  const int ng = Vs / E;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const int64_t g0 = row * int64_t(ng);
    const aal_vp_row_t s = rec[row];
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
          const float ld = __builtin_fmaf(xd[u][e], scd, -s.msc_d) - s.l2s_d;
          const float lt = __builtin_fmaf(xt[u][e], sct, -s.msc_t) - s.l2s_t;
          const float m = ex2(fminf(ld, lt));
          am += m;
          aq += (ld < lt) ? m : 0.f;
        }
      smin += am;
      qlt += aq;
    }
    smin = block_sum(smin, sh_f);
    qlt = block_sum(qlt, sh_f);
    if (threadIdx.x == 0) acc[row] = aal_vp_acc_t{smin, qlt};
  }
}

// One thread per window.  P_j = prod_{i<j} a_i, E = sum_{k=1..K} P_k,
// S_{K-1} = 1, S_j = 1 + a_{j+1} S_{j+1};  dE/da_j = P_j S_j.
__global__ __launch_bounds__(kBlock) void k_vp_scan(aal_vp_row_t* __restrict__ rec,
                                                    const aal_vp_acc_t* __restrict__ acc, int R, int64_t N, int K,
                                                    int mode, float inv_t_d, const float* __restrict__ grad_scale,
                                                    float* __restrict__ window_e, float* __restrict__ accept,
                                                    int32_t* __restrict__ xstar) {
  const int64_t n = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (n >= N) return;
  const int64_t rows = N * K;
  aal_vp_row_t* s = rec + n * K;
  if (mode == int(Mode::kWtv)) {
    for (int j = 0; j < K; ++j) {
      float a = 0.f, q = 0.f;
      for (int r = 0; r < R; ++r) {
        const aal_vp_acc_t& p = acc[int64_t(r) * rows + n * K + j];
        a += p.smin;
        q += p.qlt;
      }
      s[j].a = a;
      s[j].qlt = q;
    }
  }
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

// WTV before a sequence scan: each row's acceptance partials summed in rank
// order (a row's coefficient needs its neighbours' sums).
__global__ __launch_bounds__(kBlock) void k_vp_merge_acc(aal_vp_row_t* __restrict__ rec,
                                                         const aal_vp_acc_t* __restrict__ acc, int R,
                                                         int64_t rows) {
  const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (r >= rows) return;
  float a = 0.f, q = 0.f;
  for (int k = 0; k < R; ++k) {
    const aal_vp_acc_t& p = acc[int64_t(k) * rows + r];
    a += p.smin;
    q += p.qlt;
  }
  rec[r].a = a;
  rec[r].qlt = q;
}

// dE/da_j of the window whose rows start at r0: P_j S_j with
// P_j = prod_{i<j} a_i, S_{K-1} = 1, S_i = 1 + a_{i+1} S_{i+1} (fp64).
__device__ double window_dE_vp(const aal_vp_row_t* __restrict__ rec, int64_t r0, int K, int j) {
  double P = 1.0;
  for (int i = 0; i < j; ++i) P *= double(rec[r0 + i].a);
  double S = 1.0;
  for (int i = K - 1; i > j; --i) S = 1.0 + double(rec[r0 + i].a) * S;
  return P * S;
}

// One thread per row of B sequences of S positions with windows of K
// positions sliding by one: the row's coefficient sums dE/da over the windows
// that contain it; the row that starts a window also writes that window's E.
__global__ __launch_bounds__(kBlock) void k_vp_seq_scan(aal_vp_row_t* __restrict__ rec, int64_t B, int S, int K,
                                                        int mode, float inv_t_d, const float* __restrict__ grad_scale,
                                                        float* __restrict__ window_e, float* __restrict__ accept,
                                                        int32_t* __restrict__ xstar) {
  const int64_t r = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (r >= B * S) return;
  const int64_t b = r / S;
  const int64_t base = b * S;
  const int s = int(r - base);
  const int t0 = s - K + 1 > 0 ? s - K + 1 : 0;
  const int t1 = s < S - K ? s : S - K;
  double d = 0.0;
  for (int t = t0; t <= t1; ++t) d += window_dE_vp(rec, base + t, K, s - t);
  const double W = double(B) * double(S - K + 1);
  const double scale = grad_scale ? double(*grad_scale) : 1.0;
  const float a = rec[r].a;
  const double factor = (mode == int(Mode::kEal)) ? double(a) * double(inv_t_d) : double(inv_t_d);
  if (s <= S - K) {  // this row starts window s of its sequence
    double p = 1.0, E = 0.0;
    for (int j = 0; j < K; ++j) {
      p *= double(rec[r + j].a);
      E += p;
    }
    window_e[b * (S - K + 1) + s] = float(E);
  }
  if (accept) accept[r] = a;
  if (xstar) xstar[r] = rec[r].xstar;
  // written last: other threads read only a of this row
  rec[r].coef = float(-d / W * scale * factor);
}

template <class TI, class TG, int MODE, bool VEC, int U>
__global__ __launch_bounds__(kBlock) void k_vp_grad(const void* __restrict__ zd, const void* __restrict__ zt,
                                                    int64_t rows, int Vs, int v0, float scd, float sct,
                                                    const aal_vp_row_t* __restrict__ rec, void* __restrict__ grad) {
  using Gr = Groups<TI, VEC>;
  constexpr int E = Gr::E;
  const int ng = Vs / E;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const int64_t g0 = row * int64_t(ng);
    const aal_vp_row_t s = rec[row];
    const float c = s.coef;
    const float cA = c * (1.f - s.qlt);  // WTV, entries with q < p
    const float cB = -c * s.qlt;         // WTV, the others
    const int64_t xl = int64_t(s.xstar) - v0;  // EAL: x* in slice coordinates (may lie outside)
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
            const float d = (int64_t(gi) * E + e == xl) ? 1.f : 0.f;
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
}

template <class TI, int MODE, bool LAB>
void partials_lab(const VpSlice& s, aal_vp_part_t* parts) {
  const unsigned grid = row_grid(s.rows);
  if (s.vs % TI::kVec == 0)
    k_vp_partials<TI, MODE, true, 4, LAB><<<grid, kBlock, 0, s.stream>>>(s.zd, s.zt, s.labels, s.rows, s.vs, s.v0, s.vtot,
                                                                          s.scd, s.sct, parts);
  else
    k_vp_partials<TI, MODE, false, 8, LAB><<<grid, kBlock, 0, s.stream>>>(s.zd, s.zt, s.labels, s.rows, s.vs, s.v0, s.vtot,
                                                                           s.scd, s.sct, parts);
}

template <class TI, int MODE>
void partials_typed(const VpSlice& s, aal_vp_part_t* parts) {
  if constexpr (MODE == int(Mode::kEal)) {
    if (s.labels) {
      partials_lab<TI, MODE, true>(s, parts);
      return;
    }
  }
  partials_lab<TI, MODE, false>(s, parts);
}

template <class TI>
void accept_typed(const VpSlice& s, const aal_vp_row_t* row, aal_vp_acc_t* acc) {
  const unsigned grid = row_grid(s.rows);
  if (s.vs % TI::kVec == 0)
    k_vp_accept<TI, true, 4><<<grid, kBlock, 0, s.stream>>>(s.zd, s.zt, s.rows, s.vs, s.scd, s.sct, row, acc);
  else
    k_vp_accept<TI, false, 8><<<grid, kBlock, 0, s.stream>>>(s.zd, s.zt, s.rows, s.vs, s.scd, s.sct, row, acc);
}

template <class TI, class TG, int MODE>
void grad_typed(const VpSlice& s, const aal_vp_row_t* row, void* grad) {
  const unsigned grid = row_grid(s.rows);
  if (s.vs % TI::kVec == 0)
    k_vp_grad<TI, TG, MODE, true, 4><<<grid, kBlock, 0, s.stream>>>(s.zd, s.zt, s.rows, s.vs, s.v0, s.scd, s.sct,
                                                                    row, grad);
  else
    k_vp_grad<TI, TG, MODE, false, 8><<<grid, kBlock, 0, s.stream>>>(s.zd, s.zt, s.rows, s.vs, s.v0, s.scd, s.sct,
                                                                     row, grad);
}

template <class TG>
void grad_by_input(const VpSlice& s, const aal_vp_row_t* row, void* grad) {
  const bool eal = s.mode == Mode::kEal;
  if (s.in == DType::kBf16)
    eal ? grad_typed<Bf16, TG, int(Mode::kEal)>(s, row, grad) : grad_typed<Bf16, TG, int(Mode::kWtv)>(s, row, grad);
  else
    eal ? grad_typed<F32, TG, int(Mode::kEal)>(s, row, grad) : grad_typed<F32, TG, int(Mode::kWtv)>(s, row, grad);
}

}  // namespace

hipError_t launch_vp_partials(const VpSlice& s, aal_vp_part_t* parts) {
  const bool eal = s.mode == Mode::kEal;
  if (s.in == DType::kBf16)
    eal ? partials_typed<Bf16, int(Mode::kEal)>(s, parts) : partials_typed<Bf16, int(Mode::kWtv)>(s, parts);
  else
    eal ? partials_typed<F32, int(Mode::kEal)>(s, parts) : partials_typed<F32, int(Mode::kWtv)>(s, parts);
  return hipGetLastError();
}

hipError_t launch_vp_merge(const aal_vp_part_t* parts_all, int32_t R, int64_t rows, Mode mode, float scd, float sct,
                           aal_vp_row_t* row, hipStream_t stream) {
  const unsigned blocks = unsigned((rows + kBlock - 1) / kBlock);
  k_vp_merge<<<blocks, kBlock, 0, stream>>>(parts_all, R, rows, int(mode), scd, sct, row);
  return hipGetLastError();
}

hipError_t launch_vp_accept(const VpSlice& s, const aal_vp_row_t* row, aal_vp_acc_t* acc) {
  if (s.in == DType::kBf16)
    accept_typed<Bf16>(s, row, acc);
  else
    accept_typed<F32>(s, row, acc);
  return hipGetLastError();
}

hipError_t launch_vp_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R, int64_t N, int32_t K, Mode mode,
                          float inv_t_d, const float* grad_scale, float* loss, float* window_e, float* accept,
                          int32_t* xstar, hipStream_t stream) {
  const unsigned blocks = unsigned((N + kBlock - 1) / kBlock);
  k_vp_scan<<<blocks, kBlock, 0, stream>>>(row, acc_all, R, N, K, int(mode), inv_t_d, grad_scale, window_e, accept,
                                           xstar);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LossArgs a{};
  a.window_e = window_e;
  a.N = N;
  a.loss = loss;
  a.stream = stream;
  return launch_loss_reduce(a);
}

hipError_t launch_vp_seq_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R, int64_t B, int32_t S,
                              int32_t K, Mode mode, float inv_t_d, const float* grad_scale, float* loss,
                              float* window_e, float* accept, int32_t* xstar, hipStream_t stream) {
  const int64_t rows = B * S;
  const unsigned blocks = unsigned((rows + kBlock - 1) / kBlock);
  if (mode == Mode::kWtv) k_vp_merge_acc<<<blocks, kBlock, 0, stream>>>(row, acc_all, R, rows);
  k_vp_seq_scan<<<blocks, kBlock, 0, stream>>>(row, B, S, K, int(mode), inv_t_d, grad_scale, window_e, accept,
                                               xstar);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LossArgs a{};
  a.window_e = window_e;
  a.N = B * int64_t(S - K + 1);
  a.loss = loss;
  a.stream = stream;
  return launch_loss_reduce(a);
}

hipError_t launch_vp_grad(const VpSlice& s, const aal_vp_row_t* row, void* grad, DType gd) {
  if (gd == DType::kBf16)
    grad_by_input<GBf16>(s, row, grad);
  else
    grad_by_input<GF32>(s, row, grad);
  return hipGetLastError();
}

}  // namespace aal
