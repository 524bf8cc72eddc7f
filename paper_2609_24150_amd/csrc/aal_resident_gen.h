// Register-resident schedule for the combined objectives (aal_loss_fwd_bwd):
// the weighted sum of the WTV, EAL, forward-KL and window-mean TV terms over
// disjoint windows or over sequences whose windows slide by one (Sections
// "Window TV Loss" and "Settings"), reading each logit once and writing the
// gradient once.
//
// The work items are chunks of K consecutive rows of a sequence (the windows
// layout is the special case S = K: one chunk, one window per sequence).  A
// chunk is split by vocabulary columns over a team of W workgroups, each
// keeping its columns of all K rows of both tensors in VGPRs, as in the
// EAL/WTV resident kernel:
//
//   phase A  per-row max / sum-exp partials of the tempered draft and target
//            and the target's greedy token with the draft logit there as a
//            payload; published, merged in member order (bit-identical row
//            constants in every member).  With labels, x* is the label and
//            both logits at it are read once per row.
//   phase B  (WTV or TV term) partial sums of min(p, q), of q over q < p,
//            and with a KL term of p (log p - log q); published, merged.
//            Without a WTV or TV term there is no phase B: the KL partials
//            are summed in phase C and merged one chunk later (the KL value
//            enters the loss, not the gradient).
//   scan     with windows sliding over a sequence, a row's coefficient needs
//            the acceptances of the K-1 rows on either side: one member per
//            team publishes the chunk's a values (tagged words, written once
//            per call) and every member reads the neighbouring chunks'.  A
//            chunk's neighbours are processed by the adjacent teams in the
//            same round (the next round's first team for the last one), and
//            publishing never waits for a neighbour, so the waits always end.
//            Then, per row, dE/da summed over the windows that contain it,
//            and the coefficients of g = q (m ? cA : cB) + cP p + cX 1[v=x*].
//   phase C  gradient from the registers, refill with the team's next chunk;
//            the entry at x* is rewritten with its cX term by the thread
//            that stored it.
//
// Variants with a phase B split the chunk's rows into two groups whose merges
// overlap the other group's arithmetic, as in the EAL/WTV kernel, and no
// barrier separates consecutive chunks (the staging buffer is per wave and
// the label data is double-buffered by chunk parity).  With a TV term and no
// KL term, phase B keeps the mask [q < p] as bits and phase C reads no
// target: the first group's target registers are refilled early and the
// freed staging slots take most of the next chunk's unstaged pairs, and
// (without the greedy token) that group's target partials of the next chunk
// are evaluated while a wait is in flight: the last team merge for disjoint
// windows, the neighbour exchange for sliding ones.
//
// Rows of a chunk past the end of its sequence (when K does not divide S)
// load as zeros and store nothing.  Polls are bounded; a timeout sets the
// error word and the loss becomes NaN.
#pragma once

#include "aal_device.h"
#include "aal_internal.h"
#include "aal_resident_common.h"

#include <limits.h>

#include <type_traits>

namespace aal {
namespace {

constexpr int kGenBlock = 512;
constexpr int kGenSlotWords = 16;  // per (row, member): 0-6 phase A, 8-10 phase B
constexpr int kGenClearBlock = 256;

struct GenResParams {
  const uint8_t* zd;
  const uint8_t* zt;
  const int32_t* labels;  // may be null
  uint8_t* grad;          // may be null
  int64_t NC;             // chunks
  int S;                  // positions per sequence (windows layout: K)
  int CS;                 // chunks per sequence
  int64_t Wn;             // windows
  double inv_wn, inv_r;   // 1 / Wn (0 without windows), 1 / R
  int64_t R;              // rows
  int V, ng, W, T;
  uint32_t row_bytes, grow_bytes;
  float scd, sct, inv_t_d;
  const float* grad_scale;
  float w_wtv, w_eal, w_kl, w_tv;
  int eal;                // an EAL term
  GenStats* stats;        // kl and tv_w of every row (for the loss reduction)
  float* win_tv;
  float* win_eal;
  float* e_tv;
  float* e_eal;
  float* accept_tv;
  float* accept_eal;
  int32_t* xstar;
  uint64_t* slots;        // [2][T][K][W][16]
  uint64_t* arow;         // [R][2]: a_tv, a_eal, tagged
  unsigned* err;
};

template <class TI, class TG, int K, int NV, int VAR>
__global__ __launch_bounds__(kGenBlock) void k_res_gen(GenResParams p) {
  // VAR bits: 1 the target's normaliser (a WTV, TV or KL term); 2 a KL term;
  // 4 the EAL term's x* is the target's greedy token; 8 sum min(p, q) and Q<
  // (a WTV or TV term, or the a_tv / E_tv outputs).
  constexpr bool PQ = (VAR & 1) != 0, KL = (VAR & 2) != 0, AM = (VAR & 4) != 0, TV = (VAR & 8) != 0;
  static_assert(PQ || !(KL || TV), "KL and TV need the target normaliser");
  // Without a WTV or TV term there is no phase B: the KL term's per-row
  // partials are accumulated in phase C from the two exponentials the
  // gradient evaluates anyway (the KL value enters the loss only, never the
  // gradient), and merged over the team one chunk later, inside the next
  // chunk's phase-A merge (the team's last chunk after the loop).
  constexpr bool KLC = KL && !TV;
  constexpr bool HB = TV;  // a phase B
  constexpr int kKlWord = 12;  // slot word of the KL partials (phase B is absent)
  constexpr int kBlock = kGenBlock;
  constexpr int kWaves = kBlock / kWave;
  constexpr int E = TI::kVec;
  constexpr int GS = sizeof(typename TG::storage);
  constexpr int kC = AM ? 7 : 4;  // phase-A words per (row, member)
  constexpr int kPairs = K * NV;
  constexpr int kLdsStage = 144 * 1024;
  constexpr int kPre = kPairs < kLdsStage / (2 * kBlock * 16) ? kPairs : kLdsStage / (2 * kBlock * 16);
  constexpr float kLn2 = 0.693147180559945309417f;
  static_assert(kC * K <= kBlock && 2 * K <= kWave && K * K <= kBlock, "thread-per-item steps");
  // Phase B, when present, splits the rows into two groups (K0 rows, then the
  // rest).  With a TV term and no KL term phase C needs the target only for
  // the mask [q < p], which phase B leaves in bits: the first group's target
  // registers then take the next chunk's staged copies after the second
  // phase-A merge, and the freed slots stage most of the next chunk's
  // unstaged pairs, as in the EAL/WTV kernel.
  constexpr int K0 = PQ && K > 1 ? (K + 1) / 2 : K;
  constexpr bool MB = TV && !KL;
  constexpr bool kEarly = MB && K0 < K && K0 * NV <= kPre;
  constexpr int kFree = kEarly ? K0 * NV : 0;
  constexpr int kUnst = kPairs - kPre;
  // Without the greedy token (which phase A takes from the same target
  // data), the first group's target partials of a chunk are evaluated during
  // the previous chunk's last team merge, with a first group of 4 rows.
  constexpr bool kAhead = kEarly && !AM && K0 == 4;
  // With a phase B and no early refill (a KL term with a TV term) the staged
  // copies stay in LDS until phase C: the first rows' target partials of the
  // next chunk are then evaluated from them during the last team merge, or,
  // for sliding windows, the neighbour exchange (KL + TV over 2048 x 7
  // windows of V = 128256: 1.2% faster).
  constexpr int kLtMax = kPre / NV < K0 ? kPre / NV : K0;
  constexpr int kLT = (PQ && !AM && HB && !kEarly && K0 < K) ? (kLtMax < 4 ? kLtMax : 4) : 0;
  // Cache policy of the logit loads and gradient stores: ordinary cached
  // accesses for the look-ahead variants (sliding WTV over 7 x 2048 rows of
  // V = 128256 0.8% faster than nontemporal ones; disjoint windows 1% slower,
  // a case the fused EAL/WTV kernel serves), nontemporal otherwise.
  constexpr int kCp = kAhead ? 0 : kNontemporal;
  constexpr int KE = kAhead ? K0 : (kLT > 0 ? kLT : 1);
  // Greedy-token variants without a phase B: between publishing a chunk's
  // phase-A partials and polling the team's, each wave takes, for the next
  // chunk's first (staged) rows, the target maximum over each thread's
  // columns (with its sum-exp partial when the target is normalised) and the
  // row's greedy token over the wave (value, lowest index, owning lane),
  // reading the staged target copies from LDS; phase A then skips that part
  // (the draft payload is read from the owning lane).  KL + 0.1 EAL over
  // 2048 x 7 windows of V = 128256: 3% faster; the same rows' draft partials
  // from the staged draft copies as well measured 5% slower.
  constexpr int kGA = (AM && !HB) ? (kPre / NV < 4 ? (kPre / NV < K ? kPre / NV : K) : (K < 4 ? K : 4)) : 0;
  constexpr int kGAR = kGA > 0 ? kGA : 1;
  constexpr int kPairsPerReg = 32 / E;
  constexpr int kMaskRegs = MB ? (kPairs + kPairsPerReg - 1) / kPairsPerReg : 1;
  __shared__ u32x4 sh_pre[kPre][2][kBlock];
  __shared__ float sh_w[kWaves][K][kC];
  __shared__ float sh_row[K][6];    // msc_d, l2s_d, msc_t, l2s_t, a_eal = q(x*), p(x*)
  __shared__ int sh_x[K];
  __shared__ int sh_labx[2][K];     // the label, by chunk parity
  __shared__ float sh_lab[2][K][2]; // draft and target logits at the label, by chunk parity
  __shared__ float sh_b[K][3];      // a_tv, Q<, KL of the chunk's rows
  __shared__ float sh_a[3 * K][2];  // a_tv, a_eal of rows row0 - K .. row0 + 2K - 1
  __shared__ float sh_coef[K][7];   // cA, cB, cP scaled by 2^-l2s_d; cX; cA, cB, cP unscaled
  __shared__ float sh_d[K][K][2];   // dE/da (WTV, EAL) of row k at place jj of a window
  __shared__ float sh_klw[2][kWaves][K];  // KLC: each wave's KL partials, by chunk parity

  const int b = blockIdx.x;
  int team, member;
  if ((p.T & 7) == 0) {
    const int j = b >> 3;
    team = (j / p.W) * 8 + (b & 7);
    member = j % p.W;
  } else {
    team = b / p.W;
    member = b % p.W;
  }
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;
  const bool last = member == p.W - 1;
  const bool eal = p.eal != 0;
  int col[NV];
  uint32_t coff[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    col[v] = member * (kBlock * NV) + v * kBlock + tid;
    coff[v] = uint32_t(min(col[v], p.ng - 1)) * 16u;
  }
  uint64_t* const slots_team = p.slots + (int64_t(team) * K * p.W) * kGenSlotWords;
  const int64_t slot_plane = int64_t(p.T) * K * p.W * kGenSlotWords;

  // Chunk c: sequence c / CS, rows row0 .. row0 + nvalid - 1 of it.
  auto chunk = [&](int64_t c, int64_t& row0, int& j, int& nvalid) {
    const int64_t s = c / p.CS;
    j = int(c - s * p.CS);
    row0 = s * p.S + int64_t(j) * K;
    nvalid = min(K, p.S - j * K);
  };

  u32x4 rd[K][NV], rt[K][NV];
  uint32_t mbits[kMaskRegs];
#pragma unroll
  for (int r = 0; r < kMaskRegs; ++r) mbits[r] = 0u;
  // bit position of element e of pair i once phase B is complete (pair i's
  // bits are pushed into register i / kPairsPerReg in pair order)
  auto mask_pos = [](int i, int e) {
    const int r = i / kPairsPerReg;
    const int n = (kPairs - r * kPairsPerReg < kPairsPerReg ? kPairs - r * kPairsPerReg : kPairsPerReg) * E;
    return n - 1 - ((i % kPairsPerReg) * E + e);
  };
  auto rslot_t = [](int i) { return (i - kPre) < kFree ? i - kPre : -1; };
  auto rslot_d = [](int i) { return kUnst + (i - kPre) < kFree ? kUnst + (i - kPre) : -1; };
  float em[KE], es[KE];
  float gmt[kGAR], gbest[kGAR], gst[kGAR];
  int gx[kGAR], gsrc[kGAR];
  // row k's greedy-token look-ahead from the target vectors tv (masked past the row end)
  auto greedy_ahead = [&](const u32x4 (&tv)[NV], int k) {
    float xs[NV][E];
#pragma unroll
    for (int v = 0; v < NV; ++v) unpackv<TI, E>(tv[v], xs[v]);
    float mt = kNegInf;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < E; ++e) mt = fmaxf(mt, xs[v][e]);
    int li = 0;
#pragma unroll
    for (int v = NV - 1; v >= 0; --v)
#pragma unroll
      for (int e = E - 1; e >= 0; --e)
        if (xs[v][e] == mt) li = v * E + e;
    const int idx = mt == kNegInf ? INT_MAX : col[0] * E + (li / E) * (kBlock * E) + li % E;
    if constexpr (PQ) {  // the sum-exp partial that phase A pairs with this maximum
      const float mtsc = mt * p.sct;
      float st = 0.f;
      if (mt != kNegInf) {
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const float xe = ex2(__builtin_fmaf(xs[v][e], p.sct, -mtsc));
            st = (v == 0 && e == 0) ? xe : st + xe;
          }
      }
      gst[k] = st;
    }
    float m[1] = {mt};
    wave_max_n(m);
    const int x = wave_min_i(mt == m[0] ? idx : INT_MAX);
    const uint64_t own = __builtin_amdgcn_ballot_w64(mt == m[0] && idx == x);
    gmt[k] = mt;
    gbest[k] = m[0];
    gx[k] = x;
    gsrc[k] = own != 0 ? __builtin_ctzll(own) : 0;
  };
  // the draft logit at element x of row k (wave-uniform x, held by lane src)
  auto draft_at = [&](int k, int x, int src) {
    if (x == INT_MAX) return kNegInf;
    const int c = x / E - member * (kBlock * NV);
    const int vv = c / kBlock, e = x % E;
    constexpr int EPW = E / 4;
    const int q = e / EPW;
    uint32_t wd = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        if (v == vv && qq == q) wd = __builtin_amdgcn_readlane(rd[k][v][qq], src);
    if constexpr (EPW == 2) {
      return __builtin_bit_cast(float, (e & 1) ? (wd & 0xffff0000u) : (wd << 16));
    } else {
      return __builtin_bit_cast(float, wd);
    }
  };
  // the target's (max, sum-exp) partial of a row over this thread's columns
  // (its vectors tv)
  auto target_partial_v = [&](const u32x4 (&tv)[NV], float& mo, float& so) {
    float xs[NV][E];
#pragma unroll
    for (int v = 0; v < NV; ++v) unpackv<TI, E>(tv[v], xs[v]);
    float mt = kNegInf;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < E; ++e) mt = fmaxf(mt, xs[v][e]);
    const float mtsc = mt * p.sct;
    float st = 0.f;
    if (mt != kNegInf) {
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float x = ex2(__builtin_fmaf(xs[v][e], p.sct, -mtsc));
          st = (v == 0 && e == 0) ? x : st + x;
        }
    }
    mo = mt == kNegInf ? kNegInf : mtsc;
    so = st;
  };
  auto target_partial = [&](int k, float& mo, float& so) { target_partial_v(rt[k], mo, so); };
  // kLT: the next chunk's first target partials from the staged copies
  auto staged_target_ahead = [&]() {
    wait_vmem_all();  // the next chunk's staging (issued in phase A) has landed
#pragma unroll
    for (int k = 0; k < kLT; ++k) {
      u32x4 tv[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        tv[v] = sh_pre[k * NV + v][1][tid];
        if (last && col[v] >= p.ng) tv[v] = neg_inf_vec(TI{});
      }
      target_partial_v(tv, em[k], es[k]);
    }
  };
  auto mask_tail = [&](u32x4 (&r)[K][NV], int k) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
      if (col[v] >= p.ng) r[k][v] = neg_inf_vec(TI{});
  };
  auto pin_all = [&]() {
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        pin(rd[k][v]);
        pin(rt[k][v]);
      }
  };

  int64_t c = team;
  if (c < p.NC) {
    int64_t row0;
    int j, nvalid;
    chunk(c, row0, j, nvalid);
    const uint32_t bytes = uint32_t(nvalid) * p.row_bytes;
    const rsrc_t bd = make_rsrc(p.zd + row0 * p.row_bytes, bytes);
    const rsrc_t bt = make_rsrc(p.zt + row0 * p.row_bytes, bytes);
    const int wbase = __builtin_amdgcn_readfirstlane(wv * kWave);
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int k = i / NV, v = i % NV;
      bld16_lds<kCp>(bd, &sh_pre[i][0][wbase], coff[v], k * p.row_bytes);
      bld16_lds<kCp>(bt, &sh_pre[i][1][wbase], coff[v], k * p.row_bytes);
    }
#pragma unroll
    for (int i = kPre; i < kPairs; ++i) {
      const int k = i / NV, v = i % NV;
      rd[k][v] = bld16<kCp>(bd, coff[v], k * p.row_bytes);
      rt[k][v] = bld16<kCp>(bt, coff[v], k * p.row_bytes);
    }
    wait_vmem_all();
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int k = i / NV, v = i % NV;
      rd[k][v] = sh_pre[i][0][tid];
      rt[k][v] = sh_pre[i][1][tid];
    }
    __syncthreads();
    if constexpr (kAhead) {
#pragma unroll
      for (int k = 0; k < K0; ++k) {
        if (last) mask_tail(rt, k);
        target_partial(k, em[k], es[k]);
      }
    }
    if constexpr (kGA > 0) {
#pragma unroll
      for (int k = 0; k < kGA; ++k) {
        u32x4 tv[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) tv[v] = col[v] >= p.ng ? neg_inf_vec(TI{}) : rt[k][v];
        greedy_ahead(tv, k);
      }
    }
    if constexpr (kLT > 0) {
#pragma unroll
      for (int k = 0; k < kLT; ++k) {
        u32x4 tv[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) tv[v] = col[v] >= p.ng ? neg_inf_vec(TI{}) : rt[k][v];
        target_partial_v(tv, em[k], es[k]);
      }
    }
  }
  // read once: a global load inside the scan would sit on every chunk's
  // critical path
  const double gscale = p.grad_scale ? double(*p.grad_scale) : 1.0;
  const double inv_k = 1.0 / double(K);
  uint32_t iter = 0;
  int64_t prev_row0 = 0;  // the previous chunk (KLC: its KL is merged one chunk later)
  int prev_nvalid = 0;
  for (; c < p.NC; c += p.T, ++iter) {
    const int parity = iter & 1;
    const uint32_t tagA = 2u * (iter + 1u), tagB = tagA + 1u;
    uint64_t* const slots = slots_team + parity * slot_plane;
    uint64_t* const prev_slots = slots_team + (parity ^ 1) * slot_plane;
    int64_t row0;
    int j, nvalid;
    chunk(c, row0, j, nvalid);

    const int64_t cn = c + p.T;
    const bool more = cn < p.NC;
    int64_t nrow0 = row0;
    int nj, nnvalid = 0;
    if (more) chunk(cn, nrow0, nj, nnvalid);
    const rsrc_t nd = make_rsrc(p.zd + nrow0 * p.row_bytes, uint32_t(nnvalid) * p.row_bytes);
    const rsrc_t nt = make_rsrc(p.zt + nrow0 * p.row_bytes, uint32_t(nnvalid) * p.row_bytes);
    const int wbase = __builtin_amdgcn_readfirstlane(wv * kWave);

    // With labels, x* and the two logits there are read once per row, by
    // the first K threads; they are needed only after merge A.
    int lab_x = 0;
    float lab_d = 0.f, lab_t = 0.f;
    const bool lab_thread = eal && !AM && tid < nvalid;
    if (lab_thread) {
      const int64_t r = row0 + tid;
      lab_x = min(max(p.labels[r], 0), p.V - 1);
      lab_d = TI::load1(p.zd + r * p.row_bytes, lab_x);
      lab_t = TI::load1(p.zt + r * p.row_bytes, lab_x);
    }

    // ------------------------------------------------------------ phase A
    pin_all();
    if (last) {
#pragma unroll
      for (int v = 0; v < NV; ++v)
        if (col[v] >= p.ng)
#pragma unroll
          for (int k = 0; k < K; ++k) {
            rd[k][v] = neg_inf_vec(TI{});
            rt[k][v] = neg_inf_vec(TI{});
          }
    }
    float m0[K], s0[K], m1[K], s1[K];
    // Phase A of rows [k0, k1): per-thread partials, wave reductions, the
    // fixed-order merge of the waves and the publication of one component
    // per thread.
    auto phase_a = [&](auto k0c, auto k1c) {
      constexpr int k0 = decltype(k0c)::value, k1 = decltype(k1c)::value, KG = k1 - k0;
#pragma unroll
      for (int k = k0; k < k1; ++k) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int i = k * NV + v;
          if (i < kPre) {
            bld16_lds<kCp>(nd, &sh_pre[i][0][wbase], coff[v], k * p.row_bytes);
            bld16_lds<kCp>(nt, &sh_pre[i][1][wbase], coff[v], k * p.row_bytes);
          }
        }
        float xs[NV][E];
#pragma unroll
        for (int v = 0; v < NV; ++v) unpackv<TI, E>(rd[k][v], xs[v]);
        float m = kNegInf;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int e = 0; e < E; ++e) m = fmaxf(m, xs[v][e]);
        const float msc = m * p.scd;
        float sum = 0.f;
        if (m != kNegInf) {
#pragma unroll
          for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int e = 0; e < E; ++e) {
              const float x = ex2(__builtin_fmaf(xs[v][e], p.scd, -msc));
              sum = (v == 0 && e == 0) ? x : sum + x;  // no add of the initial zero
            }
        }
        m0[k] = m == kNegInf ? kNegInf : msc;
        s0[k] = sum;
        m1[k] = kNegInf;
        s1[k] = 0.f;
        if constexpr (PQ && !AM) {
          if ((kAhead && k < K0) || k < kLT) {  // evaluated during the previous chunk's last merge
            m1[k] = em[k < KE ? k : 0];
            s1[k] = es[k < KE ? k : 0];
          } else {
            target_partial(k, m1[k], s1[k]);
          }
        }
        if constexpr (AM) {
#pragma unroll
          for (int v = 0; v < NV; ++v) unpackv<TI, E>(rt[k][v], xs[v]);
          float mt = kNegInf;  // the target's maximum (normaliser and greedy token)
          if (k < kGA) {
            mt = gmt[k < kGAR ? k : 0];  // taken during the previous chunk's merge
          } else {
#pragma unroll
            for (int v = 0; v < NV; ++v)
#pragma unroll
              for (int e = 0; e < E; ++e) mt = fmaxf(mt, xs[v][e]);
          }
          if constexpr (PQ) {
            const float mtsc = mt * p.sct;
            float st = 0.f;
            if (k < kGA) {
              st = gst[k < kGAR ? k : 0];
            } else if (mt != kNegInf) {
#pragma unroll
              for (int v = 0; v < NV; ++v)
#pragma unroll
                for (int e = 0; e < E; ++e) {
                  const float x = ex2(__builtin_fmaf(xs[v][e], p.sct, -mtsc));
                  st = (v == 0 && e == 0) ? x : st + x;
                }
            }
            m1[k] = mt == kNegInf ? kNegInf : mtsc;
            s1[k] = st;
          }
          float best = mt, bi, bz;
          if (k < kGA) {
            const int kk = k < kGAR ? k : 0;
            best = gbest[kk];
            bi = __builtin_bit_cast(float, gx[kk]);
            bz = draft_at(k, gx[kk], gsrc[kk]);
          } else {
            first_max<TI, NV, E, kBlock>(xs, rd[k], mt, col[0] * E, bi, bz);
            wave_argmax(best, bi, bz);
          }
          // wave-uniform from here: stored right away rather than kept live
          if (lane == 0) {
            sh_w[wv][k][4] = best;
            sh_w[wv][k][5] = bi;
            sh_w[wv][k][6] = bz;
          }
        }
      }
      {
        // (max, sum) pairs of the draft (and target) rows, reduced over the wave
        // together (transposed reduction; lanes 16q store what ends on row q)
        constexpr int NL = PQ ? 2 * KG : KG;
        constexpr int NP = (NL + 3) / 4 * 4;
        float mm[NP], ss[NP], tmp[NP];
#pragma unroll
        for (int jr = 0; jr < KG; ++jr) {
          mm[jr] = m0[k0 + jr];
          ss[jr] = s0[k0 + jr];
          if constexpr (PQ) {
            mm[KG + jr] = m1[k0 + jr];
            ss[KG + jr] = s1[k0 + jr];
          }
        }
#pragma unroll
        for (int i = NL; i < NP; ++i) {
          mm[i] = kNegInf;
          ss[i] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < NP; ++i) tmp[i] = mm[i];
        float mt[NP / 4], st[NP / 4];
        wave_reduce_t(tmp, mt, OpMax{});
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const float M = reduced_t(mt, i);
          ss[i] = (M == kNegInf) ? 0.f : ss[i] * ex2(mm[i] - M);
        }
        wave_reduce_t(ss, st, OpAdd{});
        if ((lane & 15) == 0) {
          const int q = lane >> 4;
#pragma unroll
          for (int jq = 0; jq < NP / 4; ++jq) {
            const int i = 4 * jq + q;
            if (i < NL) {
              const int k = k0 + i % KG, cc = 2 * (i / KG);
              sh_w[wv][k][cc] = mt[jq];
              sh_w[wv][k][cc + 1] = st[jq];
            }
          }
        }
        if (!PQ && lane == 0) {
#pragma unroll
          for (int k = k0; k < k1; ++k) {
            sh_w[wv][k][2] = kNegInf;
            sh_w[wv][k][3] = 0.f;
          }
        }
      }
      if constexpr (k0 == 0) {
        // the label data, double-buffered by parity: a slower wave may still
        // be in the previous chunk's phase C
        if (lab_thread) {
          sh_labx[parity][tid] = lab_x;
          sh_lab[parity][tid][0] = lab_d;
          sh_lab[parity][tid][1] = lab_t;
        }
      }
      lds_barrier();
      if constexpr (KLC && k0 == 0) {
        // the previous chunk's KL partials of this member: every wave finished
        // that chunk's phase C before this barrier; summed over the waves in
        // order and published with the previous chunk's tag
        if (iter > 0 && tid < K) {
          float r = sh_klw[parity ^ 1][0][tid];
#pragma unroll
          for (int i = 1; i < kWaves; ++i) r += sh_klw[parity ^ 1][i][tid];
          publish(prev_slots + (int64_t(tid) * p.W + member) * kGenSlotWords + kKlWord, r, 2u * iter);
        }
      }
      // merge the waves, publish one component each.  With pipelined merges
      // (a phase B) the last threads of the workgroup publish when the next
      // merge (polled by waves 0, 1, ...) leaves the last wave idle, so that
      // the polling waves start at once; with a single merge right after
      // phase A the publication itself is what every member waits for, and
      // the first wave (which the SIMDs favour) publishes it sooner.
      constexpr int kPolled = K0 < K ? K0 : K;
      constexpr int kPub0 = (HB && kPolled < kWaves) ? kBlock - kC * KG : 0;
      if (tid >= kPub0 && tid < kPub0 + kC * KG) {
        const int k = k0 + (tid - kPub0) / kC, cc = (tid - kPub0) % kC;
        float a0 = sh_w[0][k][0], a1 = sh_w[0][k][1], a2 = sh_w[0][k][2], a3 = sh_w[0][k][3];
        float a4 = 0.f, a5 = 0.f, a6 = 0.f;
        if constexpr (AM) {
          a4 = sh_w[0][k][4];
          a5 = sh_w[0][k][5];
          a6 = sh_w[0][k][6];
        }
#pragma unroll
        for (int i = 1; i < kWaves; ++i) {
          lse_fold(a0, a1, sh_w[i][k][0], sh_w[i][k][1]);
          lse_fold(a2, a3, sh_w[i][k][2], sh_w[i][k][3]);
          if constexpr (AM) argmax_fold(a4, a5, a6, sh_w[i][k][4], sh_w[i][k][5], sh_w[i][k][6]);
        }
        const float val = cc == 0 ? a0 : cc == 1 ? a1 : cc == 2 ? a2 : cc == 3 ? a3 : cc == 4 ? a4 : cc == 5 ? a5 : a6;
        publish(slots + (int64_t(k) * p.W + member) * kGenSlotWords + cc, val, tagA);
      }
    };

    // Row merges of phase A for rows [k0, k1): wave wv takes rows k0 + wv,
    // k0 + wv + kWaves, ...; lane j folds members j, j+64, ... in order, then
    // a fixed DPP tree: every member obtains bit-identical row constants.
    auto merge_a = [&](int k0, int k1) {
      for (int k = k0 + wv; k < k1; k += kWaves) {
        float a0[1] = {kNegInf}, a1[1] = {0.f}, a2[1] = {kNegInf}, a3[1] = {0.f};
        float a4 = kNegInf, a5 = __builtin_bit_cast(float, INT_MAX), a6 = kNegInf;
        for (int jm = lane; jm < p.W; jm += kWave) {
          float q[kC];
          collect<kC>(slots + (int64_t(k) * p.W + jm) * kGenSlotWords, tagA, p.err, q);
          lse_fold(a0[0], a1[0], q[0], q[1]);
          lse_fold(a2[0], a3[0], q[2], q[3]);
          if constexpr (AM) argmax_fold(a4, a5, a6, q[4], q[kC - 2], q[kC - 1]);
        }
        wave_lse_n(a0, a1);
        if constexpr (PQ) wave_lse_n(a2, a3);
        if constexpr (AM) wave_argmax(a4, a5, a6);
        if (lane == 0) {
          const float mscd = a0[0], l2sd = __log2f(a1[0]);
          const float msct = a2[0], l2st = PQ ? __log2f(a3[0]) : 0.f;
          sh_row[k][0] = mscd;
          sh_row[k][1] = l2sd;
          sh_row[k][2] = msct;
          sh_row[k][3] = l2st;
          float aq = 0.f, px = 0.f;
          int x = -1;
          if (eal) {
            float zdx, ztx;
            if constexpr (AM) {
              x = __builtin_bit_cast(int, a5);
              zdx = a6;
              ztx = a4;
              if (x == INT_MAX) {  // no finite target logit: unspecified, stay in bounds
                x = 0;
                zdx = k < nvalid ? TI::load1(p.zd + (row0 + k) * int64_t(p.row_bytes), 0) : 0.f;
                ztx = kNegInf;
              }
            } else {
              x = k < nvalid ? sh_labx[parity][k] : 0;
              zdx = k < nvalid ? sh_lab[parity][k][0] : 0.f;
              ztx = k < nvalid ? sh_lab[parity][k][1] : kNegInf;
            }
            aq = ex2(__builtin_fmaf(zdx, p.scd, -mscd) - l2sd);
            if constexpr (PQ) px = ex2(__builtin_fmaf(ztx, p.sct, -msct) - l2st);
          }
          sh_x[k] = x;
          sh_row[k][4] = aq;
          sh_row[k][5] = px;
        }
        if constexpr (KLC) {
          // the previous chunk's KL of row k: the members' partials in order,
          // then the wave; they were published before this chunk's phase-A
          // words, so the polls find them at once
          if (member == 0 && iter > 0) {
            float r[1] = {0.f};
            for (int jm = lane; jm < p.W; jm += kWave) {
              float q[1];
              collect<1>(prev_slots + (int64_t(k) * p.W + jm) * kGenSlotWords + kKlWord, 2u * iter, p.err, q);
              r[0] += q[0];
            }
            wave_sum_n(r);
            if (lane == 0 && k < prev_nvalid) p.stats[prev_row0 + k].kl = r[0];
          }
        }
      }
    };
    // Phase B of rows [k0, k1): the present sums (TV: sum min(p, q) and Q<;
    // KL), reduced over the workgroup and published.
    // hook(r) runs before the arithmetic of row k0 + r of the group (after
    // that row's constants are read, so that LDS reads the hook issues do not
    // hold it up) and, with r = KG, after the last row.
    auto phase_b = [&](auto k0c, auto k1c, auto hook) {
      constexpr int k0 = decltype(k0c)::value, k1 = decltype(k1c)::value, KG = k1 - k0;
      pin_all();
      float am[KG], aq[KG], ak[KG];
#pragma unroll
      for (int k = k0; k < k1; ++k) {
        const float mscd = sh_row[k][0];
        const float ct = sh_row[k][2] + (sh_row[k][3] - sh_row[k][1]);
        hook(k - k0);
        float sm = 0.f, sq = 0.f, sk = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          float xd[E], xt[E];
          unpackv<TI, E>(rd[k][v], xd);
          unpackv<TI, E>(rt[k][v], xt);
#pragma unroll
          for (int e = 0; e < E; ++e) {
            // log2 q = u - l2s_d, log2 p = t - l2s_d (as in the WTV kernel)
            const float u = __builtin_fmaf(xd[e], p.scd, -mscd);
            const float t = __builtin_fmaf(xt[e], p.sct, -ct);
            if constexpr (TV) {
              const float mn = ex2(fminf(u, t));
              sm += mn;
              sq += (u < t) ? mn : 0.f;
              if constexpr (MB) {
                // the compare above as a lane mask (one v_cmp serves both)
                push_bit(mbits[(k * NV + v) / kPairsPerReg], __builtin_amdgcn_fcmpf(u, t, 4 /* ordered less-than */));
              }
            }
            if constexpr (KL) {
              const float ep = ex2(t);  // p 2^l2s_d; p = 0 contributes nothing
              sk = __builtin_fmaf(ep, kl_diff(t, u), sk);
            }
          }
        }
        am[k - k0] = sm;
        aq[k - k0] = sq;
        ak[k - k0] = sk;
      }
      hook(KG);
      {
        constexpr int C0 = TV ? 0 : 2;  // first component present
        constexpr int NC = (TV ? 2 : 0) + (KL ? 1 : 0);
        constexpr int NB = NC * KG;
        constexpr int NP = (NB + 3) / 4 * 4;
        float vv[NP], vt[NP / 4];
#pragma unroll
        for (int jr = 0; jr < KG; ++jr) {
          if constexpr (TV) {
            vv[jr] = am[jr];
            vv[KG + jr] = aq[jr];
          }
          if constexpr (KL) vv[(TV ? 2 * KG : 0) + jr] = ak[jr];
        }
#pragma unroll
        for (int i = NB; i < NP; ++i) vv[i] = 0.f;
        wave_reduce_t(vv, vt, OpAdd{});
        if ((lane & 15) == 0) {
          const int q = lane >> 4;
#pragma unroll
          for (int jq = 0; jq < NP / 4; ++jq) {
            const int i = 4 * jq + q;
            if (i < NB) sh_w[wv][k0 + i % KG][C0 + i / KG] = vt[jq];
          }
        }
        if (lane == 0) {
#pragma unroll
          for (int k = k0; k < k1; ++k) {
            if constexpr (!TV) {
              sh_w[wv][k][0] = 0.f;
              sh_w[wv][k][1] = 0.f;
            }
            if constexpr (!KL) sh_w[wv][k][2] = 0.f;
          }
        }
      }
      lds_barrier();
      constexpr int kPolledB = k1 < K ? K - k1 : K;  // rows of the next merge
      constexpr int kPubB = kPolledB < kWaves ? kBlock - 3 * KG : 0;
      if (tid >= kPubB && tid < kPubB + 3 * KG) {
        const int k = k0 + (tid - kPubB) / 3, cc = (tid - kPubB) % 3;
        float r = sh_w[0][k][cc];
#pragma unroll
        for (int i = 1; i < kWaves; ++i) r += sh_w[i][k][cc];
        r *= ex2(-sh_row[k][1]);
        if (cc == 2) r *= kLn2;
        publish(slots + (int64_t(k) * p.W + member) * kGenSlotWords + 8 + cc, r, tagB);
      }
    };
    // Merges of phase B for rows [k0, k1), as for phase A.
    auto merge_b = [&](int k0, int k1) {
      for (int k = k0 + wv; k < k1; k += kWaves) {
        float r[3] = {0.f, 0.f, 0.f};
        for (int jm = lane; jm < p.W; jm += kWave) {
          float q[3];
          collect<3>(slots + (int64_t(k) * p.W + jm) * kGenSlotWords + 8, tagB, p.err, q);
          r[0] += q[0];
          r[1] += q[1];
          r[2] += q[2];
        }
        wave_sum_n(r);
        if (lane == 0) {
          sh_b[k][0] = r[0];
          sh_b[k][1] = r[1];
          sh_b[k][2] = r[2];
        }
      }
    };

    // With a phase B the rows are split into two groups and the team merges
    // pipelined: each group's partials are published as soon as they are
    // complete and a merge is polled only after the other group's
    // arithmetic, so three of the four merges of a chunk overlap arithmetic.
    using I0 = std::integral_constant<int, 0>;
    using IK0 = std::integral_constant<int, K0>;
    using IK = std::integral_constant<int, K>;
    phase_a(I0{}, IK0{});
    if constexpr (K0 < K) phase_a(IK0{}, IK{});

    // ------------------------------------------------------------ phase B
    // kGA: the next chunk's greedy tokens from the staged target copies
    auto staged_greedy_ahead = [&]() {
      wait_vmem_all();  // the next chunk's staging (issued in phase A) has landed
#pragma unroll
      for (int k = 0; k < kGA; ++k) {
        u32x4 tv[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          tv[v] = sh_pre[k * NV + v][1][tid];
          if (last && col[v] >= p.ng) tv[v] = neg_inf_vec(TI{});
        }
        greedy_ahead(tv, k);
      }
    };
    if constexpr (!HB) {
      // before the merge for disjoint windows; for sliding ones in the
      // neighbour exchange below, off the ring of neighbour dependencies
      if constexpr (kGA > 0) {
        if (p.CS == 1) staged_greedy_ahead();
      }
      merge_a(0, K);
      if (tid < K) {
        sh_b[tid][0] = 0.f;
        sh_b[tid][1] = 0.f;
        sh_b[tid][2] = 0.f;
      }
    } else if constexpr (K0 == K) {
      merge_a(0, K);
      lds_barrier();
      phase_b(I0{}, IK{}, [](int) {});
      merge_b(0, K);
    } else {
      merge_a(0, K0);
      lds_barrier();
      phase_b(I0{}, IK0{}, [](int) {});
      merge_a(K0, K);
      lds_barrier();
      // With kEarly the first group's target is dead: the next chunk's staged
      // copies go to its registers, then the freed slots are restaged.
      auto refill = [&]() {
        wait_vmem_all();  // this chunk's staging (issued in phase A) has landed
#pragma unroll
        for (int i = 0; i < kFree; ++i) rt[i / NV][i % NV] = sh_pre[i][1][tid];
      };
      auto restage = [&]() {
        if (last) {
#pragma unroll
          for (int k = 0; k < K0; ++k) mask_tail(rt, k);
        }
        wait_lds_all();  // the slots are read before the loads below rewrite them
#pragma unroll
        for (int s = 0; s < kFree; ++s) {
          const int i = kPre + (s < kUnst ? s : s - kUnst);
          if (i < kPairs)
            bld16_lds<kCp>(s < kUnst ? nt : nd, &sh_pre[s][1][wbase], coff[i % NV], (i / NV) * p.row_bytes);
        }
      };
      if constexpr (kAhead) {
        // the reads land while the second group's first row is evaluated
        phase_b(IK0{}, IK{}, [&](int r) {
          if (r == 0) refill();
          if (r == 1) restage();
        });
      } else {
        if constexpr (kEarly) {
          refill();
          restage();
        }
        phase_b(IK0{}, IK{}, [](int) {});
      }
      if constexpr (kAhead) {
        // the next chunk's first-group target partials while the other
        // members' last partials are on their way (past the team's last chunk
        // the registers hold zeros and the results go unused); with windows
        // sliding over sequences they wait for the neighbour exchange below
        // instead, whose wait sits on the cycle that paces the teams
        if (p.CS == 1) {
#pragma unroll
          for (int k = 0; k < K0; ++k) target_partial(k, em[k], es[k]);
        }
      }
      if constexpr (kLT > 0) {
        if (p.CS == 1) staged_target_ahead();
      }
      merge_b(0, K);
    }
    lds_barrier();

    // --------------------------------------------------------------- scan
    // a values of the rows row0 - K .. row0 + 2K - 1 (own chunk in the middle)
    if (tid < K) {
      sh_a[K + tid][0] = sh_b[tid][0];
      sh_a[K + tid][1] = sh_row[tid][4];
    }
    if (p.CS > 1) {
      if (member == 0 && tid < nvalid) {
        uint64_t* const ar = p.arow + (row0 + tid) * 2;
        publish(ar, sh_b[tid][0], 1u);
        publish(ar + 1, sh_row[tid][4], 1u);
      }
      if constexpr (kAhead) {
#pragma unroll
        for (int k = 0; k < K0; ++k) target_partial(k, em[k], es[k]);
      }
      if constexpr (kLT > 0) staged_target_ahead();
      if constexpr (kGA > 0) staged_greedy_ahead();
      if (wv == 0 && lane < 2 * K) {
        const int o = lane < K ? lane - K : lane;  // offset from row0: -K..-1, K..2K-1
        const int pos = j * K + o;                 // position in the sequence
        if (pos >= 0 && pos < p.S) {
          float q[2];
          collect<2>(p.arow + (row0 + o) * 2, 1u, p.err, q);
          sh_a[K + o][0] = q[0];
          sh_a[K + o][1] = q[1];
        }
      }
    }
    lds_barrier();
    // dE/da of row k as the jj-th row of the window that starts at position
    // s - jj (s = the row's position), one thread per (k, jj); the thread with
    // jj = 0 also evaluates E of the window that starts at the row.
    if (tid < K * K) {
      const int k = tid / K, jj = tid % K;
      const int s = j * K + k, t = s - jj;
      float dt = 0.f, de = 0.f;
      if (k < nvalid && t >= 0 && t <= p.S - K) {
        const int o0 = K + (t - j * K);  // the window's first row in sh_a
        // The window's acceptances are read up front and the recurrences are
        // straight-line: a factor outside the product enters as 1.0 and a step
        // outside the nesting keeps the previous value, which gives the same
        // bits as skipping them (a branch per factor made this one-wave step
        // wait for each LDS read in turn, with every other wave at the barrier).
        float xa[K], xe[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
          xa[i] = sh_a[o0 + i][0];
          xe[i] = sh_a[o0 + i][1];
        }
        double ptv = 1.0, peal = 1.0, stv = 1.0, seal = 1.0, etv = 0.0, eeal = 0.0;
#pragma unroll
        for (int i = 0; i < K; ++i) {
          ptv *= i < jj ? double(xa[i]) : 1.0;
          peal *= i < jj ? double(xe[i]) : 1.0;
        }
#pragma unroll
        for (int i = K - 1; i > 0; --i) {
          const double nt = 1.0 + double(xa[i]) * stv, ne = 1.0 + double(xe[i]) * seal;
          stv = i > jj ? nt : stv;
          seal = i > jj ? ne : seal;
        }
        dt = float(ptv * stv);
        de = float(peal * seal);
        if (jj == 0 && member == 0) {
          double pt = 1.0, pe = 1.0;
#pragma unroll
          for (int q = 0; q < K; ++q) {
            pt *= double(xa[q]);
            pe *= double(xe[q]);
            etv += pt;
            eeal += pe;
          }
          const int64_t w = (row0 - int64_t(j) * K) / p.S * int64_t(p.S - K + 1) + t;
          p.win_tv[w] = float(etv);
          p.win_eal[w] = float(eeal);
          if (p.e_tv) p.e_tv[w] = float(etv);
          if (p.e_eal) p.e_eal[w] = float(eeal);
        }
      }
      sh_d[k][jj][0] = dt;
      sh_d[k][jj][1] = de;
    }
    lds_barrier();
    if (tid < nvalid) {
      const int k = tid;
      const int s = j * K + k;
      double dtv = 0.0, deal = 0.0;
#pragma unroll
      for (int jj = 0; jj < K; ++jj) {
        dtv += double(sh_d[k][jj][0]);
        deal += double(sh_d[k][jj][1]);
      }
      const int lo = max(0, s - K + 1), hi = min(s, p.S - K);
      const double count = hi >= lo ? double(hi - lo + 1) : 0.0;
      const double f = gscale * double(p.inv_t_d);
      const double a_tv = double(sh_b[k][0]), qlt = double(sh_b[k][1]), a_eal = double(sh_row[k][4]);
      const double g_tv = (-double(p.w_wtv) * dtv - double(p.w_tv) * count * inv_k) * p.inv_wn;
      const double g_eal = -double(p.w_eal) * deal * p.inv_wn;
      const double g_kl = double(p.w_kl) * p.inv_r;
      const double c_tv = g_tv * f, c_eal = g_eal * a_eal * f, c_kl = g_kl * f;
      const float cA = float(c_tv * (1.0 - qlt) - c_eal + c_kl);
      const float cB = float(-c_tv * qlt - c_eal + c_kl);
      const float cP = float(-c_kl);
      const float rs = ex2(-sh_row[k][1]);
      sh_coef[k][0] = cA * rs;
      sh_coef[k][1] = cB * rs;
      sh_coef[k][2] = cP * rs;
      sh_coef[k][3] = float(c_eal);
      sh_coef[k][4] = cA;
      sh_coef[k][5] = cB;
      sh_coef[k][6] = cP;
      if (member == 0) {
        const int64_t r = row0 + k;
        if constexpr (!KLC) p.stats[r].kl = sh_b[k][2];
        p.stats[r].tv_w = float(count * (1.0 - a_tv));
        if (p.accept_tv) p.accept_tv[r] = sh_b[k][0];
        if (p.accept_eal) p.accept_eal[r] = sh_row[k][4];
        if (p.xstar) p.xstar[r] = eal ? sh_x[k] : -1;
      }
    }
    lds_barrier();

    // ------------------------------------------------------------ phase C
    uint8_t* const gw = p.grad ? p.grad + row0 * int64_t(p.grow_bytes) : nullptr;
    // KLC: this thread's sum of 2^t (t - u) over row k's entries
    // (p (log2 p - log2 q) 2^l2s_d), reduced over the wave as soon as the
    // row's last pair is done, so at most two of them are live
    float klp[K];
#pragma unroll
    for (int k = 0; k < K; ++k) klp[k] = 0.f;
    wait_vmem_all();  // staging has landed
    pin_all();
    float mscd = 0.f, ct = 0.f, cA = 0.f, cB = 0.f, cP = 0.f;
#pragma unroll
    for (int jp = 0; jp < kPairs; ++jp) {
      const int i = (jp + kPre) % kPairs;
      const int k = i / NV, v = i % NV;
      if (jp == 0 || v == 0) {  // a new row: its constants, once per row
        mscd = sh_row[k][0];
        ct = sh_row[k][2] + (sh_row[k][3] - sh_row[k][1]);
        cA = sh_coef[k][0];
        cB = sh_coef[k][1];
        if constexpr (!MB) asm volatile("" : "+v"(cA), "+v"(cB));
        cP = sh_coef[k][2];
      }
      const rsrc_t gr = make_rsrc(gw + k * p.grow_bytes, gw != nullptr && k < nvalid ? p.grow_bytes : 0u);
      float xd[E], g[E];
      unpackv<TI, E>(rd[k][v], xd);
      if constexpr (MB) {
        // the mask [q < p] from phase B selects the coefficient
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float u = __builtin_fmaf(xd[e], p.scd, -mscd);
          g[e] = ex2(u) * select_bit(mbits[i / kPairsPerReg], mask_pos(i, e), cA, cB);
        }
      } else if constexpr (PQ) {
        float xt[E];
        unpackv<TI, E>(rt[k][v], xt);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float u = __builtin_fmaf(xd[e], p.scd, -mscd);
          const float t = __builtin_fmaf(xt[e], p.sct, -ct);
          if constexpr (TV) {
            g[e] = ex2(u) * ((u < t) ? cA : cB);
          } else {
            g[e] = ex2(u) * cA;  // no mask without a TV term: cA = cB
          }
          if constexpr (KL) {
            const float ep = ex2(t);  // p 2^l2s_d; p = 0 contributes nothing
            g[e] = __builtin_fmaf(cP, ep, g[e]);
            if constexpr (KLC) klp[k] = __builtin_fmaf(ep, kl_diff(t, u), klp[k]);
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) g[e] = cA * ex2(__builtin_fmaf(xd[e], p.scd, -mscd));
      }
      store_g<TG, E, kCp>(gr, uint32_t(col[v]) * uint32_t(E * GS), g);
      asm volatile("" ::: "memory");
      if (i < kPre) {
        rd[k][v] = sh_pre[i][0][tid];
        if (i >= kFree) rt[k][v] = sh_pre[i][1][tid];  // pairs below kFree were refilled after merge A
      } else {
        const int sd = kEarly ? rslot_d(i) : -1, st = kEarly ? rslot_t(i) : -1;
        rd[k][v] = sd >= 0 ? sh_pre[sd][1][tid] : bld16<kCp>(nd, coff[v], k * p.row_bytes);
        rt[k][v] = st >= 0 ? sh_pre[st][1][tid] : bld16<kCp>(nt, coff[v], k * p.row_bytes);
      }
      if constexpr (KLC) {
        // the last pair of row k in this order: (jp + kPre) % kPairs runs
        // through the pairs from kPre, wrapping round, so a row that pair kPre
        // cuts (kPre not a multiple of NV) ends at pair kPre - 1
        constexpr int kCut = kPre % NV != 0 ? (kPre - 1) / NV : -1;
        const bool row_done = k == kCut ? i == kPre - 1 : v == NV - 1;
        if (row_done) {
          const float r = wave_sum(klp[k]);  // this wave's partial of row k (uniform)
          if (lane == 0) sh_klw[parity][wv][k] = r * ex2(-sh_row[k][1]) * kLn2;
        }
      }
    }
    if (eal && gw != nullptr) {
      // the entry at x*: q (m ? cA : cB) + cP p + cX, rewritten by the thread
      // whose vector store covered it (same thread, so it lands last)
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int xk = sh_x[k];
        bool own = false;
#pragma unroll
        for (int v = 0; v < NV; ++v) own = own || (col[v] == xk / E);
        if (own && k < nvalid) {
          const float qx = sh_row[k][4], px = sh_row[k][5];
          float gx = qx * ((TV && qx < px) ? sh_coef[k][4] : sh_coef[k][5]) + sh_coef[k][3];
          if constexpr (KL) gx = __builtin_fmaf(sh_coef[k][6], px, gx);
          const rsrc_t gr = make_rsrc(gw + k * p.grow_bytes, p.grow_bytes);
          store_one<TG>(gr, uint32_t(xk) * GS, gx);
        }
      }
    }
    prev_row0 = row0;
    prev_nvalid = nvalid;
    // No barrier before the next chunk: a wave only reads and restages its
    // own slice of the staging buffer (after its reads above have completed),
    // the label data and the KL partials are double-buffered, and the shared
    // row constants are rewritten only after the barrier closing the next
    // chunk's first phase-A group, which every wave reaches after finishing
    // this phase C.
    wait_lds_all();
  }
  if constexpr (KLC) {
    // the team's last chunk: its KL partials, published and merged as above
    if (iter > 0) {
      const int pp = int((iter - 1) & 1);
      uint64_t* const last_slots = slots_team + pp * slot_plane;
      lds_barrier();
      if (tid < K) {
        float r = sh_klw[pp][0][tid];
#pragma unroll
        for (int i = 1; i < kWaves; ++i) r += sh_klw[pp][i][tid];
        publish(last_slots + (int64_t(tid) * p.W + member) * kGenSlotWords + kKlWord, r, 2u * iter);
      }
      if (member == 0) {
        for (int k = wv; k < K; k += kWaves) {
          float r[1] = {0.f};
          for (int jm = lane; jm < p.W; jm += kWave) {
            float q[1];
            collect<1>(last_slots + (int64_t(k) * p.W + jm) * kGenSlotWords + kKlWord, 2u * iter, p.err, q);
            r[0] += q[0];
          }
          wave_sum_n(r);
          if (lane == 0 && k < prev_nvalid) p.stats[prev_row0 + k].kl = r[0];
        }
      }
    }
  }
  wait_vmem_all();
}

// Zeroes the slot words and the acceptance words of windows sliding over
// sequences (n1 = 0 without), and sets the error word to `err`, in one launch.
__global__ void k_gen_clear(uint64_t* p0, int64_t n0, uint64_t* p1, int64_t n1, uint64_t* err_word,
                            uint64_t err) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (int64_t i = t; i < n0; i += stride) p0[i] = 0;
  for (int64_t i = t; i < n1; i += stride) p1[i] = 0;
  if (t == 0) *err_word = err;
}

template <class TI, class TG, int K, int VAR>
hipError_t launch_kg(const GenArgs& a, bool* used) {
  constexpr int NV = (16 / K) > 0 ? (16 / K) : 1;
  constexpr int E = TI::kVec;
  constexpr int kBlock = kGenBlock;
  auto kern = k_res_gen<TI, TG, K, NV, VAR>;
  const DevInfo di = device_info();
  if ((a.coop && !di.coop) || di.cus == 0) return hipSuccess;
  const int ng = a.V / E;
  const int W = (ng + kBlock * NV - 1) / (kBlock * NV);
  const int64_t row_bytes = int64_t(a.V) * (a.in == DType::kBf16 ? 2 : 4);
  const int64_t grow_bytes = int64_t(a.V) * (a.gd == DType::kBf16 ? 2 : 4);
  if (int64_t(K) * grow_bytes >= (int64_t(1) << 31) || int64_t(K) * row_bytes >= (int64_t(1) << 31))
    return hipSuccess;
  const int S = a.layout == 0 ? K : a.S;
  const int CS = (S + K - 1) / K;
  const int64_t NC = a.B * CS;
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kBlock, 0);
  if (e != hipSuccess) return e;
  int64_t T = int64_t(per_cu) * di.cus / W;
  // every co-resident team runs (members span XCDs unless the team count is a
  // multiple of 8)
  if (T > NC) T = NC;
  if (T < 1) return hipSuccess;
  // a chunk waits for its neighbours' acceptances, which must come from
  // another team
  if (CS > 1 && T < 2) return hipSuccess;
  auto words = [&](int64_t t) { return int64_t(2) * t * K * W * kGenSlotWords; };
  while (T > 8 && size_t(words(T)) * 8 > a.res_slot_bytes) T -= 8;
  if (size_t(words(T)) * 8 > a.res_slot_bytes) return hipSuccess;
  GenResParams p{};
  p.zd = static_cast<const uint8_t*>(a.zd);
  p.zt = static_cast<const uint8_t*>(a.zt);
  p.labels = a.labels;
  p.grad = static_cast<uint8_t*>(a.grad);
  p.NC = NC;
  p.S = S;
  p.CS = CS;
  p.Wn = a.W;
  p.R = a.R;
  p.inv_wn = a.W > 0 ? 1.0 / double(a.W) : 0.0;
  p.inv_r = 1.0 / double(a.R);
  p.V = a.V;
  p.ng = ng;
  p.W = W;
  p.T = int(T);
  p.row_bytes = uint32_t(row_bytes);
  p.grow_bytes = uint32_t(grow_bytes);
  p.scd = a.sc_d;
  p.sct = a.sc_t;
  p.inv_t_d = a.inv_t_d;
  p.grad_scale = a.grad_scale;
  p.w_wtv = a.w_wtv;
  p.w_eal = a.w_eal;
  p.w_kl = a.w_kl;
  p.w_tv = a.w_tv;
  p.eal = a.w_eal != 0.f ? 1 : 0;
  p.stats = a.stats;
  p.win_tv = a.win_tv;
  p.win_eal = a.win_eal;
  p.e_tv = a.e_tv;
  p.e_eal = a.e_eal;
  p.accept_tv = a.accept_tv;
  p.accept_eal = a.accept_eal;
  p.xstar = a.xstar;
  p.slots = a.res_slots;
  p.arow = a.arow;
  p.err = a.res_err;
  k_gen_clear<<<CS > 1 ? 256 : 64, kGenClearBlock, 0, a.stream>>>(p.slots, words(T), p.arow, CS > 1 ? a.R * 2 : 0,
                                                                  reinterpret_cast<uint64_t*>(p.err),
                                                                  initial_error_word());
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.coop) {
    void* args[] = {&p};
    e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kern), dim3(unsigned(T * W)), dim3(kBlock), args, 0,
                                   a.stream);
  } else {
    // the grid fits the device at once (see the occupancy bound above)
    kern<<<dim3(unsigned(T * W)), dim3(kBlock), 0, a.stream>>>(p);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  *used = true;
  return hipSuccess;
}

template <class TI, class TG, int VAR>
hipError_t launch_kl(const GenArgs& a, bool* used) {
  switch (a.K) {
    case 1: return launch_kg<TI, TG, 1, VAR>(a, used);
    case 2: return launch_kg<TI, TG, 2, VAR>(a, used);
    case 3: return launch_kg<TI, TG, 3, VAR>(a, used);
    case 4: return launch_kg<TI, TG, 4, VAR>(a, used);
    case 5: return launch_kg<TI, TG, 5, VAR>(a, used);
    case 6: return launch_kg<TI, TG, 6, VAR>(a, used);
    case 7: return launch_kg<TI, TG, 7, VAR>(a, used);
    case 8: return launch_kg<TI, TG, 8, VAR>(a, used);
    case 16: return launch_kg<TI, TG, 16, VAR>(a, used);
    default: return hipSuccess;
  }
}

template <class TI, class TG>
hipError_t launch_tg(const GenArgs& a, bool* used) {
  // sum min(p, q) is needed by the WTV and TV terms and by the a_tv / E_tv
  // outputs (which the KL term alone would otherwise leave unevaluated)
  const bool tv = a.w_wtv != 0.f || a.w_tv != 0.f || (a.w_kl != 0.f && (a.accept_tv || a.e_tv));
  const bool kl = a.w_kl != 0.f;
  const bool am = a.w_eal != 0.f && a.labels == nullptr;
  if (!tv && !kl) return am ? launch_kl<TI, TG, 4>(a, used) : hipSuccess;  // EAL with labels: streaming
  if (kl && tv) return am ? launch_kl<TI, TG, 15>(a, used) : launch_kl<TI, TG, 11>(a, used);
  if (kl) return am ? launch_kl<TI, TG, 7>(a, used) : launch_kl<TI, TG, 3>(a, used);
  return am ? launch_kl<TI, TG, 13>(a, used) : launch_kl<TI, TG, 9>(a, used);
}

template <class TI>
hipError_t launch_ti(const GenArgs& a, bool* used) {
  if (a.gd == DType::kF32) return launch_tg<TI, GF32>(a, used);
  if constexpr (std::is_same_v<TI, Bf16>) return launch_tg<TI, GBf16>(a, used);
  return hipSuccess;  // fp32 logits with a bf16 gradient: streaming schedule
}

}  // namespace
}  // namespace aal
