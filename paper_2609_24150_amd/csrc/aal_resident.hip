// Register-resident schedule for the EAL and WTV losses: one kernel that reads
// each logit once and writes the gradient once.
//
// A window (K logit rows) is split by vocabulary columns over a team of W
// workgroups.  Each workgroup loads its column chunk of all K rows of both
// logit tensors into VGPRs (16-byte nontemporal loads) and keeps them there:
//
//   phase A  per-row max / sum-exp partials of the tempered draft and target
//            (EAL: the target's greedy token, with the draft logit there as
//            a payload, instead of the target sum); published to the team.
//   merge A  every member merges the W partials in member order (so every
//            member holds bit-identical row normalisers; EAL's a = q(x*)
//            follows from the payload).
//   phase B  (WTV) per-row partial sums of min(p, q) and Q< = sum_{q<p} q,
//            published, merged in member order; the mask [q < p] of every
//            element is kept as one bit per element for phase C.
//   scan     prefix products / suffix sums over the K rows give E and the
//            gradient coefficients (Eqs. eal_generic, loss_eal, loss_tv).
//   phase C  gradient from the registers, 16-byte nontemporal stores; each
//            register slot is refilled with the team's next window as soon
//            as its gradient is written.
//
// WTV splits the rows into two groups and publishes each group's partials as
// soon as they are complete, so that a merge is polled only after the other
// group's arithmetic: of the four merges of a window only the last one waits.
// The first pairs of the next window are staged into LDS during phase A and
// copied to the registers in phase C; each wave stages and reads back only
// its own threads' slots, so no barrier separates consecutive windows.  For
// WTV the first row group's target is dead once its phase-B partials are
// summed (phase C needs only the mask bits): its registers take their staged
// next-window copies after the second phase-A merge, and the freed slots
// stage most of the next window's remaining pairs, so phase C issues few HBM
// loads besides its gradient stores.
//
// The grid is persistent and no larger than the device holds at once, so
// every member of a team becomes resident (work already on the device can
// delay the placement of some members, never prevent it; a launch through the
// runtime's cooperative launch, on request, has the runtime place the whole
// grid first, at about 20 us per call).  Partials travel as 64-bit words {value, tag}: a reader
// polls the words it needs until every tag names the current window and
// phase, so publishing doubles as the team barrier and no separate counter
// round trip is needed.  Slots are double-buffered by window parity, which
// keeps a fast member from overwriting a partial a slow member has not read.
// Polls are bounded (a timeout sets an error word and the loss becomes NaN;
// the kernel always exits).  With a multiple of 8 teams, team members share
// blockIdx % 8, i.e. one XCD; otherwise they span XCDs.
#include "aal_device.h"
#include "aal_internal.h"
#include "aal_resident_common.h"

#include <limits.h>

#include <type_traits>

namespace aal {
namespace {

constexpr int kClearBlock = 256;
#ifndef AAL_SLOT_BUDGET
#define AAL_SLOT_BUDGET 16
#endif
// 16-byte vectors of each logit tensor a thread keeps per window (K * NV).
constexpr int kSlotBudget = AAL_SLOT_BUDGET;

struct ResParams {
  const uint8_t* zd;
  const uint8_t* zt;
  uint8_t* grad;
  int64_t N;
  int ng;              // 16-byte vectors per row
  int W;               // workgroups per team
  int T;               // teams
  uint32_t row_bytes;  // bytes per logit row
  uint32_t grow_bytes; // bytes per gradient row
  float scd, sct, inv_t_d;
  const float* grad_scale;
  float* window_e;
  float* accept;
  int32_t* xstar;
  uint64_t* slots;     // [parity 2][T][K][W][8] words {value bits, tag}: 0-4 phase A, 4-5 phase B
  unsigned* err;       // [1]
};

template <class TI, class TG, int MODE, int K, int NV, int kBlock>
__global__ __launch_bounds__(kBlock) void k_resident(ResParams p) {
  constexpr int kWaves = kBlock / kWave;
  constexpr int E = TI::kVec;
  constexpr bool kWtv = MODE == int(Mode::kWtv);
  constexpr int GS = sizeof(typename TG::storage);  // gradient element bytes
  // Phase-A components per row: draft (max, sum), target (max, sum) for WTV;
  // draft (max, sum), target (max, argmax), draft logit at the argmax for EAL.
  constexpr int kC = kWtv ? 4 : 5;
  static_assert(kC * K <= kBlock, "one publishing thread per row component");
  // LDS staging of the team's next window: the first kPre (row, vector) pairs
  // of both tensors are fetched into LDS at the start of a window and copied
  // to the registers in phase C, so most of the refill traffic overlaps the
  // compute phases instead of all of it queueing behind phase C.
  constexpr int kPairs = K * NV;
  constexpr int kLdsStage = kBlock >= 512 ? 144 * 1024 : 72 * 1024;  // one or two workgroups per CU
  constexpr int kPre = kPairs < kLdsStage / (2 * kBlock * 16) ? kPairs : kLdsStage / (2 * kBlock * 16);
  static_assert(kPre >= 1, "staging holds at least one pair");
  // WTV splits the rows into two groups (K0 rows, then the rest).  Phase C
  // reads no target (the mask bits replace it), so the target registers of
  // the first group are refilled with the next window as soon as the second
  // group's normalisers are merged, from their staged copies, and those
  // staging slots then take the next window's unstaged target pairs and, as
  // far as they go, its unstaged draft pairs: phase C, which carries the
  // gradient stores, is left with few or no HBM loads.
  constexpr int K0 = kWtv && K > 1 ? (K + 1) / 2 : K;
  // EAL: the target is dead after phase A, so between publishing a window's
  // partials and polling the team's, each wave takes the greedy token of the
  // next window's wholly staged rows (up to 4) over its own columns: the
  // largest value and its lowest index, the same fold as phase A, without
  // the draft payload, which phase A then reads from the lane that holds it.
#ifndef AAL_EAL_AHEAD
#define AAL_EAL_AHEAD 1
#endif
  constexpr int kEA = (!kWtv && AAL_EAL_AHEAD) ? (kPre / NV < 4 ? (kPre / NV < K ? kPre / NV : K) : (K < 4 ? K : 4)) : 0;
  constexpr int kEAPairs = kEA * NV;
  // Target slots refilled early (WTV: the first row group after the second
  // phase-A merge; EAL: the look-ahead rows before the merge); the freed
  // slots then stage the next window's unstaged pairs.
  constexpr bool kEarly = (kWtv && K0 < K && K0 * NV <= kPre) || (kEA > 0 && kPairs > kPre);
  constexpr int kFree = kEarly ? (kWtv ? K0 * NV : kEAPairs) : 0;
  constexpr int kUnst = kPairs - kPre;                                 // unstaged pairs per tensor
  // Restaging slot of unstaged pair i (i >= kPre) of the target / draft, or
  // -1 when it still comes from HBM in phase C.
  auto rslot_t = [](int i) { return (i - kPre) < kFree ? i - kPre : -1; };
  auto rslot_d = [](int i) { return kUnst + (i - kPre) < kFree ? kUnst + (i - kPre) : -1; };
  // staging slots of the draft and of the target, as separate arrays so that
  // reads of draft slots are visibly independent of loads into target slots
  __shared__ u32x4 sh_pre_d[kPre][kBlock];
  __shared__ u32x4 sh_pre_t[kPre][kBlock];
  __shared__ float sh_w[kWaves][K][kC];  // per-wave partials
  __shared__ float sh_row[K][4];        // merged row constants
  __shared__ float sh_coef[K][2];       // gradient coefficients
  __shared__ int sh_x[K];

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
  const bool last = member == p.W - 1;  // the only member whose chunk can pass the row end
  int col[NV];
  uint32_t coff[NV];  // clamped byte offsets of the slots within a row: always in bounds
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    col[v] = member * (kBlock * NV) + v * kBlock + tid;
    coff[v] = uint32_t(min(col[v], p.ng - 1)) * 16u;
  }
  const int64_t stride_w = int64_t(K) * p.row_bytes;
  // Tagged slots: 8 words per (row, member), one 64-byte line; planes by parity.
  uint64_t* const slots_team = p.slots + (int64_t(team) * K * p.W) * 8;
  const int64_t slot_plane = int64_t(p.T) * K * p.W * 8;

  u32x4 rd[K][NV], rt[K][NV];
  // WTV: phase B leaves [q < p] of every element in these bits for phase C,
  // which then needs neither the target nor a compare.  Pair i = k NV + v
  // holds bits in register i / kPairsPerReg, pushed in pair order.
  constexpr int kPairsPerReg = 32 / E;
  constexpr int kMaskRegs = kWtv ? (kPairs + kPairsPerReg - 1) / kPairsPerReg : 1;
  uint32_t mbits[kMaskRegs];
#pragma unroll
  for (int r = 0; r < kMaskRegs; ++r) mbits[r] = 0u;
  // bit position of element e of pair i once phase B is complete
  auto mask_pos = [](int i, int e) {
    const int r = i / kPairsPerReg;
    const int n = (kPairs - r * kPairsPerReg < kPairsPerReg ? kPairs - r * kPairsPerReg : kPairsPerReg) * E;
    return n - 1 - ((i % kPairsPerReg) * E + e);
  };

  const uint32_t win_bytes = uint32_t(stride_w);
  auto pin_all = [&]() {
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        pin(rd[k][v]);
        pin(rt[k][v]);
      }
  };

  // WTV: the first group's target (max, sum-exp) partials of a window are
  // evaluated one window ahead, while the previous window's last team merge
  // is in flight (the registers hold the next window's target by then), so
  // that wait is spent on arithmetic phase A would otherwise do.
  // Used with a first group of 4 rows (K = 7, 8), where the partials fit
  // beside the resident data: at K = 5 (3 rows, 13-member teams) it measured
  // slower, and larger groups spill.
#ifndef AAL_AHEAD_MIN_ROWS
#define AAL_AHEAD_MIN_ROWS 4
#endif
#ifndef AAL_AHEAD_MAX_ROWS
#define AAL_AHEAD_MAX_ROWS 4
#endif
  constexpr bool kAhead = kWtv && kEarly && K0 >= AAL_AHEAD_MIN_ROWS && K0 <= AAL_AHEAD_MAX_ROWS;
  // Cache policy of the logit loads and gradient stores: nontemporal, except
  // for WTV with the look-ahead, whose ordinary cached accesses measured 1%
  // faster at K = 7, V = 128256 (nontemporal is faster for EAL, by 2-5%, and
  // for WTV at K = 5 and 16, by 1-2%).
  constexpr int kCp = kAhead ? 0 : kNontemporal;
  constexpr int KE = kAhead ? K0 : 1;
  float em[KE], es[KE];
  auto target_partial = [&](int k, float& mo, float& so) {
    float xs[NV][E];
#pragma unroll
    for (int v = 0; v < NV; ++v) unpackv<TI, E>(rt[k][v], xs[v]);
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
          st = (v == 0 && e == 0) ? x : st + x;  // no add of the initial zero
        }
    }
    mo = mt == kNegInf ? kNegInf : mtsc;
    so = st;
  };
  // slots past the row end (last member only) hold copies of the row's last
  // vector: mask them
  auto mask_tail = [&](u32x4 (&r)[K][NV], int k) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
      if (col[v] >= p.ng) r[k][v] = neg_inf_vec(TI{});
  };

  // EAL look-ahead (see kEA above): per row the wave's largest target value,
  // its lowest index and the lane holding it
  constexpr int kEAR = kEA > 0 ? kEA : 1;
  float eab[kEAR];
  int eax[kEAR], eas[kEAR];
  // and, once those registers are free again, the same rows' draft (max,
  // sum-exp) partials from the draft's staged copies: with 4 such rows
  // (K = 7: 1.7% faster); with 3 (K = 5, 13-member teams) it measured 2%
  // slower
  constexpr bool kEAD = kEA >= 4;
  float edm[kEAR], eds[kEAR];
  auto argmax_ahead = [&](int k, float& bo, int& xo, int& so) {
    float xs[NV][E];
#pragma unroll
    for (int v = 0; v < NV; ++v) unpackv<TI, E>(rt[k][v], xs[v]);
    float best = kNegInf;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < E; ++e) best = fmaxf(best, xs[v][e]);
    int li = 0;
#pragma unroll
    for (int v = NV - 1; v >= 0; --v)
#pragma unroll
      for (int e = E - 1; e >= 0; --e)
        if (xs[v][e] == best) li = v * E + e;
    const int idx = best == kNegInf ? INT_MAX : col[0] * E + (li / E) * (kBlock * E) + li % E;
    float m[1] = {best};
    wave_max_n(m);
    const int x = wave_min_i(best == m[0] ? idx : INT_MAX);
    const uint64_t own = __builtin_amdgcn_ballot_w64(best == m[0] && idx == x);
    bo = m[0];
    xo = x;
    so = own != 0 ? __builtin_ctzll(own) : 0;
  };
  // the draft's (max, sum-exp) partial of row k from registers r, as phase A
  // evaluates it
  auto draft_partial = [&](const u32x4 (&r)[K][NV], int k, float& mo, float& so) {
    float xs[NV][E];
#pragma unroll
    for (int v = 0; v < NV; ++v) unpackv<TI, E>(r[k][v], xs[v]);
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
    mo = m == kNegInf ? kNegInf : msc;
    so = sum;
  };
  // the draft logit at element x of row k (wave-uniform x, held by lane src)
  auto payload = [&](int k, int x, int src) {
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

  int64_t w = team;
  if (w < p.N) {
    // The first window arrives the way later windows do (staged pairs through
    // LDS, the rest straight to registers), so the loop sees one wait pattern.
    const rsrc_t bd = make_rsrc(p.zd + w * stride_w, win_bytes);
    const rsrc_t bt = make_rsrc(p.zt + w * stride_w, win_bytes);
    const int wbase = __builtin_amdgcn_readfirstlane(wv * kWave);
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int k = i / NV, v = i % NV;
      bld16_lds<kCp>(bd, &sh_pre_d[i][wbase], coff[v], k * p.row_bytes);
      bld16_lds<kCp>(bt, &sh_pre_t[i][wbase], coff[v], k * p.row_bytes);
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
      rd[k][v] = sh_pre_d[i][tid];
      rt[k][v] = sh_pre_t[i][tid];
    }
    __syncthreads();  // staging is read before the loop restages it
    if constexpr (kAhead) {
#pragma unroll
      for (int k = 0; k < K0; ++k) {
        if (last) mask_tail(rt, k);
        target_partial(k, em[k], es[k]);
      }
    }
    if constexpr (kEA > 0) {
#pragma unroll
      for (int k = 0; k < kEA; ++k) {
        if (last) {
          mask_tail(rt, k);
          mask_tail(rd, k);
        }
        argmax_ahead(k, eab[k], eax[k], eas[k]);
        if constexpr (kEAD) draft_partial(rd, k, edm[k], eds[k]);
      }
    }
  }
  // read once: a global load inside the scan would sit on every window's
  // critical path
  const double gscale = p.grad_scale ? double(*p.grad_scale) : 1.0;
  uint32_t iter = 0;
  for (; w < p.N; w += p.T, ++iter) {
    const int parity = iter & 1;
    const uint32_t tagA = 2u * (iter + 1u), tagB = tagA + 1u;
    uint64_t* const slots = slots_team + parity * slot_plane;

    const int64_t wn = w + p.T;
    const bool more = wn < p.N;
    // Past the team's last window the next-window resources are empty: the
    // staging and refill loads still issue (so every iteration has the same
    // memory-counter pattern) but read nothing.
    const rsrc_t nd = make_rsrc(p.zd + (more ? wn : w) * stride_w, more ? win_bytes : 0u);
    const rsrc_t nt = make_rsrc(p.zt + (more ? wn : w) * stride_w, more ? win_bytes : 0u);
    // The first kPre pairs of the next window are staged into LDS during
    // phase A (each wave stages and later reads back only its own threads'
    // slots, so no barrier guards the buffer between windows).
    const int wbase = __builtin_amdgcn_readfirstlane(wv * kWave);
    auto stage_row = [&](int k) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int i = k * NV + v;
        if (i < kPre) {
          bld16_lds<kCp>(nd, &sh_pre_d[i][wbase], coff[v], k * p.row_bytes);
          bld16_lds<kCp>(nt, &sh_pre_t[i][wbase], coff[v], k * p.row_bytes);
        }
      }
    };
    // The kFree target slots refilled early stage the next window's unstaged
    // pairs: its targets first, then as many of its drafts as remain.
    auto restage_freed = [&]() {
      wait_lds_all();  // the slots are read before the loads below rewrite them
#pragma unroll
      for (int s = 0; s < kFree; ++s) {
        const int i = kPre + (s < kUnst ? s : s - kUnst);
        if (i < kPairs)
          bld16_lds<kCp>(s < kUnst ? nt : nd, &sh_pre_t[s][wbase], coff[i % NV], (i / NV) * p.row_bytes);
      }
    };

    // ------------------------------------------------------------ phase A
    pin_all();
    if (last) {  // slots past the row end hold copies of its last vector: mask them
#pragma unroll
      for (int v = 0; v < NV; ++v)
        if (col[v] >= p.ng)
#pragma unroll
          for (int k = 0; k < K; ++k) {
            rd[k][v] = neg_inf_vec(TI{});
            rt[k][v] = neg_inf_vec(TI{});
          }
    }
    float m0[K], s0[K], m1[K], s1[K], z1[K];
    // Phase A of rows [k0, k1): per-thread partials, wave reductions, the
    // fixed-order merge of the waves and the publication of one component
    // per thread.
    auto phase_a = [&](auto k0c, auto k1c) {
      constexpr int k0 = decltype(k0c)::value, k1 = decltype(k1c)::value, KG = k1 - k0;
#pragma unroll
      for (int k = k0; k < k1; ++k) {
        stage_row(k);  // issued between the rows' arithmetic, the loads do not stall the wave
        float xs[NV][E];
        if (kEAD && k < kEA) {  // evaluated during the previous window's merge
          m0[k] = edm[k < kEAR ? k : 0];
          s0[k] = eds[k < kEAR ? k : 0];
        } else {
          draft_partial(rd, k, m0[k], s0[k]);
        }
        if constexpr (kWtv) {
          if (kAhead && k < K0) {  // evaluated during the previous window's last merge
            m1[k] = em[k < KE ? k : 0];
            s1[k] = es[k < KE ? k : 0];
          } else {
            target_partial(k, m1[k], s1[k]);
          }
        } else if (k < kEA) {  // evaluated during the previous window's merge
          m1[k] = eab[k < kEAR ? k : 0];
          s1[k] = __builtin_bit_cast(float, eax[k < kEAR ? k : 0]);
          z1[k] = payload(k, eax[k < kEAR ? k : 0], eas[k < kEAR ? k : 0]);
        } else {
#pragma unroll
          for (int v = 0; v < NV; ++v) unpackv<TI, E>(rt[k][v], xs[v]);
          float best = kNegInf, bi, bz;
#pragma unroll
          for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int e = 0; e < E; ++e) best = fmaxf(best, xs[v][e]);
          first_max<TI, NV, E, kBlock>(xs, rd[k], best, col[0] * E, bi, bz);
          // reduced over the wave right away: the results are wave-uniform, so
          // the per-lane payloads are short-lived
          wave_argmax(best, bi, bz);
          m1[k] = best;
          s1[k] = bi;
          z1[k] = bz;
        }
      }
      {
        // (max, sum) pairs of the draft (and target) rows, reduced over the
        // wave together: the maxima first, every lane's sum rescaled to them,
        // then the sums; lanes 16q store the values that end on row q.
        constexpr int NL = kWtv ? 2 * KG : KG;
        constexpr int NP = (NL + 3) / 4 * 4;
        float mm[NP], ss[NP], tmp[NP];
#pragma unroll
        for (int j = 0; j < KG; ++j) {
          mm[j] = m0[k0 + j];
          ss[j] = s0[k0 + j];
          if constexpr (kWtv) {
            mm[KG + j] = m1[k0 + j];
            ss[KG + j] = s1[k0 + j];
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
              const int k = k0 + i % KG, c = 2 * (i / KG);
              sh_w[wv][k][c] = mt[jq];
              sh_w[wv][k][c + 1] = st[jq];
            }
          }
        }
      }
      if constexpr (!kWtv) {
        if (lane == 0) {
#pragma unroll
          for (int k = k0; k < k1; ++k) {
            sh_w[wv][k][2] = m1[k];
            sh_w[wv][k][3] = s1[k];
            sh_w[wv][k][4] = z1[k];
          }
        }
      }
      lds_barrier();
      // merge the waves (fixed order), publish one component each: the last
      // threads of the workgroup when the next merge (of the first group's
      // rows, polled by waves 0, 1, ...) leaves the last wave idle, so that
      // the polling waves start at once; otherwise the first threads
      constexpr int kPolled = K0 < K ? K0 : K;
      constexpr int kPub0 = kPolled < kWaves ? kBlock - kC * KG : 0;
      if (tid >= kPub0 && tid < kPub0 + kC * KG) {
        const int pt = tid - kPub0;
        const int k = k0 + pt / kC, c = pt % kC;
        float a0 = sh_w[0][k][0], a1 = sh_w[0][k][1], a2 = sh_w[0][k][2], a3 = sh_w[0][k][3];
        float a4 = kWtv ? 0.f : sh_w[0][k][kC - 1];
#pragma unroll
        for (int i = 1; i < kWaves; ++i) {
          lse_fold(a0, a1, sh_w[i][k][0], sh_w[i][k][1]);
          if constexpr (kWtv) {
            lse_fold(a2, a3, sh_w[i][k][2], sh_w[i][k][3]);
          } else {
            argmax_fold(a2, a3, a4, sh_w[i][k][2], sh_w[i][k][3], sh_w[i][k][kC - 1]);
          }
        }
        const float val = c == 0 ? a0 : c == 1 ? a1 : c == 2 ? a2 : c == 3 ? a3 : a4;
        publish(slots + (int64_t(k) * p.W + member) * 8 + c, val, tagA);
      }
    };

    // Row merges of phase A for rows [k0, k1): wave wv takes rows k0 + wv,
    // k0 + wv + kWaves, ...; lane j folds members j, j+64, ... in order, then a
    // fixed DPP tree: every member of the team obtains bit-identical row
    // constants.
    auto merge_a = [&](int k0, int k1) {
      for (int k = k0 + wv; k < k1; k += kWaves) {
        float a0[1] = {kNegInf}, a1[1] = {0.f}, a2[1] = {kNegInf}, a3[1], a4 = kNegInf;
        a3[0] = kWtv ? 0.f : __builtin_bit_cast(float, INT_MAX);
        for (int j = lane; j < p.W; j += kWave) {
          float q[kC];
          collect<kC>(slots + (int64_t(k) * p.W + j) * 8, tagA, p.err, q);
          lse_fold(a0[0], a1[0], q[0], q[1]);
          if constexpr (kWtv) {
            lse_fold(a2[0], a3[0], q[2], q[3]);
          } else {
            argmax_fold(a2[0], a3[0], a4, q[2], q[3], q[kC - 1]);
          }
        }
        wave_lse_n(a0, a1);
        if constexpr (kWtv) {
          wave_lse_n(a2, a3);
          if (lane == 0) {
            sh_row[k][0] = a0[0];
            sh_row[k][1] = __log2f(a1[0]);
            sh_row[k][2] = a2[0];
            sh_row[k][3] = __log2f(a3[0]);
          }
        } else {
          wave_argmax(a2[0], a3[0], a4);
          int x = __builtin_bit_cast(int, a3[0]);
          if (lane == 0) {
            float zx = a4;  // the draft logit at x, carried through the merges
            if (x == INT_MAX) {  // no finite target logit: unspecified, stay in bounds
              x = 0;
              zx = TI::load1(p.zd + (w * K + k) * int64_t(p.row_bytes), 0);
            }
            const float l2s = __log2f(a1[0]);
            sh_x[k] = x;
            sh_row[k][0] = a0[0];
            sh_row[k][1] = l2s;
            sh_row[k][2] = ex2(__builtin_fmaf(zx, p.scd, -a0[0]) - l2s);  // a = q(x*)
          }
        }
      }
    };
    // Phase B (WTV) of rows [k0, k1): partial sums of min(p, q) and Q<,
    // reduced over the workgroup and published.
    // hook(r) runs before the arithmetic of row k0 + r of the group (after
    // that row's constants are read, so that LDS reads the hook issues do not
    // hold it up) and, with r = KG, after the last row.  With the look-ahead
    // (4-row first groups) every group's row constants are read before its
    // first row (0.8% faster at K = 7, V = 128256); at K = 5 and 16 that
    // raised the register count and measured slower.
    auto phase_b = [&](auto k0c, auto k1c, auto hook) {
      constexpr int k0 = decltype(k0c)::value, k1 = decltype(k1c)::value, KG = k1 - k0;
      pin_all();
      float am[KG], aq[KG];
      // With u = x_d sc_d - msc_d and t = x_t sc_t - (msc_t + dl), each one
      // fma, log2 q = u - l2sd and log2 p = t - l2sd for dl = l2st - l2sd, so
      // min(p, q) = 2^-l2sd 2^min(u, t) and [q < p] = [u < t]: the common
      // factor is applied once per row after the reductions.
      constexpr bool kPreload = kAhead;
      float rmscd[kPreload ? KG : 1], rct[kPreload ? KG : 1];
      if constexpr (kPreload) {
#pragma unroll
        for (int k = k0; k < k1; ++k) {
          rmscd[k - k0] = sh_row[k][0];
          rct[k - k0] = sh_row[k][2] + (sh_row[k][3] - sh_row[k][1]);
        }
      }
#pragma unroll
      for (int k = k0; k < k1; ++k) {
        float mscd, ct;
        if constexpr (kPreload) {
          mscd = rmscd[k - k0];
          ct = rct[k - k0];
        } else {
          mscd = sh_row[k][0];
          ct = sh_row[k][2] + (sh_row[k][3] - sh_row[k][1]);
        }
        hook(k - k0);
        float sm = 0.f, sq = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          float xd[E], xt[E];
          unpackv<TI, E>(rd[k][v], xd);
          unpackv<TI, E>(rt[k][v], xt);
#pragma unroll
          for (int e = 0; e < E; ++e) {
            const float u = __builtin_fmaf(xd[e], p.scd, -mscd);
            const float t = __builtin_fmaf(xt[e], p.sct, -ct);
            const float mn = ex2(fminf(u, t));
            // the compare below, as a lane mask (the compiler emits one v_cmp for both)
            const uint64_t lt = __builtin_amdgcn_fcmpf(u, t, 4 /* ordered less-than */);
            if (v == 0 && e == 0) {
              sm = mn;
              sq = (u < t) ? mn : 0.f;
            } else {
              sm += mn;
              sq += (u < t) ? mn : 0.f;
            }
            push_bit(mbits[(k * NV + v) / kPairsPerReg], lt);
          }
        }
        am[k - k0] = sm;
        aq[k - k0] = sq;
      }
      hook(KG);
      {
        constexpr int NP = (2 * KG + 3) / 4 * 4;
        float vv[NP], vt[NP / 4];
#pragma unroll
        for (int j = 0; j < KG; ++j) {
          vv[j] = am[j];
          vv[KG + j] = aq[j];
        }
#pragma unroll
        for (int i = 2 * KG; i < NP; ++i) vv[i] = 0.f;
        wave_reduce_t(vv, vt, OpAdd{});
        if ((lane & 15) == 0) {
          const int q = lane >> 4;
#pragma unroll
          for (int jq = 0; jq < NP / 4; ++jq) {
            const int i = 4 * jq + q;
            if (i < 2 * KG) sh_w[wv][k0 + i % KG][i / KG] = vt[jq];
          }
        }
      }
      lds_barrier();
      // the last threads when the next merge (of rows [k1 < K ? k1 : 0, K))
      // leaves the last wave idle, as in phase A
      constexpr int kPolled = k1 < K ? K - k1 : K;
      constexpr int kPub0 = kPolled < kWaves ? kBlock - 2 * KG : 0;
      if (tid >= kPub0 && tid < kPub0 + 2 * KG) {
        const int pt = tid - kPub0;
        const int k = k0 + (pt >> 1), c = pt & 1;
        float r = sh_w[0][k][c];
#pragma unroll
        for (int i = 1; i < kWaves; ++i) r += sh_w[i][k][c];
        publish(slots + (int64_t(k) * p.W + member) * 8 + 4 + c, r * ex2(-sh_row[k][1]), tagB);
      }
    };
    // Merges of phase B for rows [k0, k1), as for phase A.
    auto merge_b = [&](int k0, int k1) {
      for (int k = k0 + wv; k < k1; k += kWaves) {
        float r[2] = {0.f, 0.f};
        for (int j = lane; j < p.W; j += kWave) {
          float q[2];
          collect<2>(slots + (int64_t(k) * p.W + j) * 8 + 4, tagB, p.err, q);
          r[0] += q[0];
          r[1] += q[1];
        }
        wave_sum_n(r);
        if (lane == 0) {
          sh_coef[k][0] = r[0];  // a_k, until the scan below
          sh_coef[k][1] = r[1];  // Q<_k
        }
      }
    };

    // WTV splits the rows into two groups and pipelines the team merges: each
    // group's partials are published as soon as they are complete, and a
    // merge is only polled once the other group's arithmetic has given the
    // slower members time to publish, so three of the four merges of a
    // window overlap arithmetic and only the last one waits.  EAL has one
    // merge per window and keeps a single group.
    using I0 = std::integral_constant<int, 0>;
    using IK0 = std::integral_constant<int, K0>;
    using IK = std::integral_constant<int, K>;
    phase_a(I0{}, IK0{});
    if constexpr (K0 < K) phase_a(IK0{}, IK{});

    // ------------------------------------------------------------ phase B
    if constexpr (!kWtv) {
      if constexpr (kEA > 0) {
        wait_vmem_all();  // the next window's staging (issued in phase A) has landed
#pragma unroll
        for (int i = 0; i < kEAPairs; ++i) rt[i / NV][i % NV] = sh_pre_t[i][tid];
#pragma unroll
        for (int k = 0; k < kEA; ++k) {
          if (last) mask_tail(rt, k);
          argmax_ahead(k, eab[k], eax[k], eas[k]);
        }
        if constexpr (kEAD) {
          // the target registers of these rows are free again: the next
          // window's staged draft copies, for its draft partials
#pragma unroll
          for (int i = 0; i < kEAPairs; ++i) rt[i / NV][i % NV] = sh_pre_d[i][tid];
#pragma unroll
          for (int k = 0; k < kEA; ++k) {
            if (last) mask_tail(rt, k);
            draft_partial(rt, k, edm[k], eds[k]);
          }
        }
      }
      merge_a(0, K);
      lds_barrier();
      // issued after the polls, which would otherwise wait for these loads
      // (vector-memory instructions complete in issue order)
      if constexpr (kEarly) restage_freed();
    } else if constexpr (K0 == K) {
      merge_a(0, K);
      lds_barrier();
      phase_b(I0{}, IK{}, [](int) {});
      merge_b(0, K);
      lds_barrier();
    } else {
      merge_a(0, K0);
      lds_barrier();
      phase_b(I0{}, IK0{}, [](int) {});
      merge_a(K0, K);
      lds_barrier();
      // The first group's target is dead: the next window's staged copies go
      // to its registers, then the freed slots are restaged.
      auto refill = [&]() {
        wait_vmem_all();  // this window's staging (issued in phase A) has landed
#pragma unroll
        for (int i = 0; i < kFree; ++i) rt[i / NV][i % NV] = sh_pre_t[i][tid];
      };
      auto restage = [&]() {
        if (last) {
#pragma unroll
          for (int k = 0; k < K0; ++k) mask_tail(rt, k);
        }
        restage_freed();
      };
      if constexpr (kAhead) {
        // the reads land while the second group's first row is evaluated
        phase_b(IK0{}, IK{}, [&](int r) {
          if (r == 0) refill();
          if (r == 1) restage();
        });
      } else {
        refill();
        restage();
        phase_b(IK0{}, IK{}, [](int) {});
      }
      // the next window's first-group target partials, while the other
      // members' last partials are on their way (past the team's last window
      // the registers hold zeros and the results go unused)
      if constexpr (kAhead) {
#pragma unroll
        for (int k = 0; k < K0; ++k) target_partial(k, em[k], es[k]);
      }
      merge_b(0, K);
      lds_barrier();
    }

    // --------------------------------------------------------------- scan
    // Lane k of wave 0 evaluates row k's coefficient: every lane reads the
    // K acceptances and forms P_k = prod_{j<k} a_j and S_k = 1 + a_{k+1} S_{k+1}
    // in the order of the serial recurrences, so the results equal the
    // one-thread form; lane 0 also sums E.
    if (wv == 0) {
      float a[K];
#pragma unroll
      for (int j = 0; j < K; ++j) a[j] = kWtv ? sh_coef[j][0] : sh_row[j][2];
      const int k = lane;
      const bool own = k < K;
      const float ak = own ? (kWtv ? sh_coef[k][0] : sh_row[k][2]) : 0.f;
      const float qlt = (kWtv && own) ? sh_coef[k][1] : 0.f;
      double P = 1.0, S = 1.0;
#pragma unroll
      for (int j = 0; j < K; ++j)
        if (j < k) P *= double(a[j]);
#pragma unroll
      for (int j = K - 1; j > 0; --j)
        if (j > k) S = 1.0 + double(a[j]) * S;
      const double inv_n = 1.0 / double(p.N);
      const double g = -P * S * inv_n;
      const double factor = kWtv ? double(p.inv_t_d) : double(ak) * double(p.inv_t_d);
      const float c = float(g * gscale * factor);
      if (own) {
        if constexpr (kWtv) {
          sh_coef[k][0] = c * (1.f - qlt);
          sh_coef[k][1] = -c * qlt;
        } else {
          sh_coef[k][0] = c;
        }
      }
      if (member == 0) {
        if (lane == 0) {
          double pr = 1.0, Ew = 0.0;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            pr *= double(a[j]);
            Ew += pr;
          }
          p.window_e[w] = float(Ew);
        }
        if (own) {
          if (p.accept) p.accept[w * K + k] = ak;
          if constexpr (!kWtv) {
            if (p.xstar) p.xstar[w * K + k] = sh_x[k];
          }
        }
      }
    }
    lds_barrier();

    // ------------------------------------------------------------ phase C
    // Gradient from the registers; each pair of slots is refilled with the
    // team's next window right after its gradient is stored: the unstaged
    // pairs first from HBM (the longest time to land), then the staged pairs
    // from LDS.
    // without a gradient output the stores go to an empty resource (dropped)
    uint8_t* const gw = p.grad ? p.grad + w * int64_t(K) * p.grow_bytes : nullptr;
    const uint32_t grow = gw != nullptr ? p.grow_bytes : 0u;
    // Order of the pairs.  Without restaging: the unstaged pairs first, from
    // HBM (the longest time to land), then the staged ones.  With restaging:
    //   C0  the pairs whose draft still comes from HBM (issued first: the
    //       next window's phase A waits for them);
    //   C1  the pairs staged in phase A, whose loads were issued before the
    //       restaging loads: a wave that did not poll the last merge may still
    //       have those in flight (the polls drained the others'), so waiting
    //       down to that many suffices;
    //   then one wait bounded by the stores and loads issued since the
    //   restaging, the target refills that read restaged slots (or staged
    //   slots beyond the first group), and
    //   C2  the pairs whose draft was restaged.
    constexpr int kStoresPerPair = (GS == 4 && E == 8) ? 2 : 1;
    constexpr int kRestOps = kEarly ? (kFree < 2 * kUnst ? kFree : 2 * kUnst) : 0;
    constexpr int kRD = kEarly ? (kFree - kUnst < 0 ? 0 : (kFree - kUnst < kUnst ? kFree - kUnst : kUnst)) : 0;
    constexpr int kC0 = kEarly ? kUnst - kRD : 0;  // pairs kPre + kRD .. kPairs - 1
    auto c_order = [](int j) {
      if constexpr (!kEarly) {
        return (j + kPre) % kPairs;
      } else {
        return j < kC0 ? kPre + kRD + j : j < kC0 + kPre ? j - kC0 : kPre + (j - kC0 - kPre);
      }
    };
    // loads of a C0 pair: the draft, and the target when its slot was not restaged
    auto c0_ops = []() {
      int n = 0;
      for (int i = kPre + kRD; i < kPairs; ++i) n += kStoresPerPair + 1 + ((i - kPre) >= kFree ? 1 : 0);
      return n;
    };
    constexpr int kOpsAfterRestage = kEarly ? c0_ops() + kPre * kStoresPerPair : 0;
    static_assert(kOpsAfterRestage < 64, "vmcnt range");
    auto restaged_reads = [&]() {
      wait_vmem_le<kOpsAfterRestage>();  // the restaging loads have landed
#pragma unroll
      for (int i2 = kFree; i2 < kPre; ++i2) rt[i2 / NV][i2 % NV] = sh_pre_t[i2][tid];
#pragma unroll
      for (int i2 = kPre + kRD; i2 < kPairs; ++i2)
        if (i2 - kPre < kFree) rt[i2 / NV][i2 % NV] = sh_pre_t[i2 - kPre][tid];
    };
    if constexpr (kEarly) {
      wait_vmem_le<kRestOps>();
    } else {
      wait_vmem_all();  // staging has landed (issued a whole phase A and B earlier)
    }
    pin_all();
    float mscd = 0.f, cA = 0.f, cB = 0.f;
#pragma unroll
    for (int j = 0; j < kPairs; ++j) {
      const int i = c_order(j);
      if (kEarly && j == kC0 + kPre) restaged_reads();
      const int k = i / NV, v = i % NV;
      if (j == 0 || v == 0 || j == kC0) {  // a new row: its constants, once per row
        // q = 2^-l2sd 2^u: the row factor 2^-l2sd is folded into the coefficients
        const float rs = ex2(-sh_row[k][1]);
        mscd = sh_row[k][0];
        if constexpr (kWtv) {
          cA = sh_coef[k][0] * rs;
          cB = sh_coef[k][1] * rs;
        } else {
          cA = -sh_coef[k][0] * rs;
        }
      }
      const rsrc_t gr = make_rsrc(gw + k * grow, grow);  // slots past the row end are dropped
      float xd[E], g[E];
      unpackv<TI, E>(rd[k][v], xd);
      if constexpr (kWtv) {
        // the mask [q < p] from phase B selects the coefficient
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float u = __builtin_fmaf(xd[e], p.scd, -mscd);
          g[e] = ex2(u) * select_bit(mbits[i / kPairsPerReg], mask_pos(i, e), cA, cB);
        }
      } else {
        // -c q everywhere; the greedy token's entry is fixed up after the loop
#pragma unroll
        for (int e = 0; e < E; ++e) g[e] = cA * ex2(__builtin_fmaf(xd[e], p.scd, -mscd));
      }
      store_g<TG, E, kCp>(gr, uint32_t(col[v]) * uint32_t(E * GS), g);
      asm volatile("" ::: "memory");  // keep the refill below this slot's store
      if (i < kPre) {
        rd[k][v] = sh_pre_d[i][tid];
        // target pairs below kFree were refilled after merge A (EAL: below
        // kEAPairs, before it); with restaging the others are read after the
        // wait above
        if (!kEarly && i >= kEAPairs) rt[k][v] = sh_pre_t[i][tid];
      } else {
        const int sd = kEarly ? rslot_d(i) : -1, st = kEarly ? rslot_t(i) : -1;
        rd[k][v] = sd >= 0 ? sh_pre_t[sd][tid] : bld16<kCp>(nd, coff[v], k * p.row_bytes);
        if (st < 0) {
          rt[k][v] = bld16<kCp>(nt, coff[v], k * p.row_bytes);
        } else if (j >= kC0 + kPre) {  // C2 (a C0 pair's restaged target is read after the wait)
          rt[k][v] = sh_pre_t[st][tid];
        }
      }
    }
    if constexpr (kEarly && kRD == 0) restaged_reads();  // no C2: the wait closes the phase
    if constexpr (!kWtv) {
      // EAL: the greedy token's entry is c (1 - q(x*)) = c (1 - a), written by
      // the thread whose vector store covered it (same thread, so it lands last)
      if (gw != nullptr) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int xk = sh_x[k];
          bool own = false;
#pragma unroll
          for (int v = 0; v < NV; ++v) own = own || (col[v] == xk / E);
          if (own) {
            const rsrc_t gr = make_rsrc(gw + k * p.grow_bytes, p.grow_bytes);
            store_one<TG>(gr, uint32_t(xk) * GS, sh_coef[k][0] * (1.f - sh_row[k][2]));
          }
        }
      }
    }
    // No barrier before the next window: a wave only reads and restages its
    // own slice of the staging buffer (after its reads above have completed),
    // and the next window rewrites sh_w, sh_row, sh_coef and sh_x only after
    // the barrier that closes its first phase-A group, which every wave
    // reaches after finishing this phase C.
    wait_lds_all();
  }
  wait_vmem_all();  // the last (empty) staging loads retire before the workgroup ends
}

// Zeroes the tag words (tag 0 never matches) and the error word.
// Zeroes the slot words p[0 .. n-2]; the error word p[n-1] takes `err`.
__global__ void k_clear(uint64_t* p, int64_t n, uint64_t err) {
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
    p[i] = i == n - 1 ? err : 0;
}

// -------------------------------------------------------------- dispatch
// Workgroup size per mode: one 512-thread workgroup per CU, which keeps the
// teams small (less skew at each team synchronisation) and gives the LDS
// staging the whole 144 KiB.
#ifndef AAL_WTV_BLOCK
#define AAL_WTV_BLOCK 512
#endif
#ifndef AAL_EAL_BLOCK
#define AAL_EAL_BLOCK 512
#endif
template <int MODE>
constexpr int block_for() {
  return MODE == int(Mode::kWtv) ? AAL_WTV_BLOCK : AAL_EAL_BLOCK;
}

template <class TI, class TG, int MODE, int K>
hipError_t launch_k(const LossArgs& a, bool* used) {
  constexpr int NV = (kSlotBudget / K) > 0 ? (kSlotBudget / K) : 1;
  constexpr int E = TI::kVec;
  constexpr int kBlock = block_for<MODE>();
  auto kern = k_resident<TI, TG, MODE, K, NV, kBlock>;
  const DevInfo di = device_info();
  if ((a.coop && !di.coop) || di.cus == 0) return hipSuccess;
  const int ng = a.V / E;
  const int W = (ng + kBlock * NV - 1) / (kBlock * NV);
  const int64_t row_bytes = int64_t(a.V) * (a.in == DType::kBf16 ? 2 : 4);
  const int64_t grow_bytes = int64_t(a.V) * (a.gd == DType::kBf16 ? 2 : 4);
  if (int64_t(K) * grow_bytes >= (int64_t(1) << 31) || int64_t(K) * row_bytes >= (int64_t(1) << 31))
    return hipSuccess;  // 32-bit in-window offsets
  int per_cu = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kBlock, 0);
  if (e != hipSuccess) return e;
  const int64_t resident = int64_t(per_cu) * di.cus;
  int64_t T = resident / W;
  // every co-resident team runs; with a multiple of 8 teams the members of a
  // team share an XCD, otherwise they span XCDs (measured: no slower than the
  // XCD-local exchange, and rounding the team count down idled up to 19% of
  // the CUs)
  if (T > a.N) T = a.N;
  if (T < 1) return hipSuccess;  // a window does not fit: streaming schedule
  auto words = [&](int64_t t) { return int64_t(2) * t * K * W * 8; };
  while (T > 8 && size_t(words(T) + 1) * 8 > a.ws.resident_bytes) T -= 8;
  if (size_t(words(T) + 1) * 8 > a.ws.resident_bytes) return hipSuccess;
  ResParams p{};
  p.zd = static_cast<const uint8_t*>(a.zd);
  p.zt = static_cast<const uint8_t*>(a.zt);
  p.grad = static_cast<uint8_t*>(a.grad);
  p.N = a.N;
  p.ng = ng;
  p.W = W;
  p.T = int(T);
  p.row_bytes = uint32_t(row_bytes);
  p.grow_bytes = uint32_t(grow_bytes);
  p.scd = a.sc_d;
  p.sct = a.sc_t;
  p.inv_t_d = a.inv_t_d;
  p.grad_scale = a.grad_scale;
  p.window_e = a.window_e;
  p.accept = a.accept;
  p.xstar = a.xstar;
  p.slots = reinterpret_cast<uint64_t*>(a.ws.resident);
  p.err = reinterpret_cast<unsigned*>(p.slots + words(T));
  const int64_t nclear = words(T) + 1;
  k_clear<<<64, kClearBlock, 0, a.stream>>>(p.slots, nclear, initial_error_word());
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
  return launch_loss_reduce(a, p.err);  // NaN loss if a poll timed out
}

template <class TI, class TG, int MODE>
hipError_t launch_mode(const LossArgs& a, bool* used) {
  switch (a.K) {
    case 1: return launch_k<TI, TG, MODE, 1>(a, used);
    case 2: return launch_k<TI, TG, MODE, 2>(a, used);
    case 3: return launch_k<TI, TG, MODE, 3>(a, used);
    case 4: return launch_k<TI, TG, MODE, 4>(a, used);
    case 5: return launch_k<TI, TG, MODE, 5>(a, used);
    case 6: return launch_k<TI, TG, MODE, 6>(a, used);
    case 7: return launch_k<TI, TG, MODE, 7>(a, used);
    case 8: return launch_k<TI, TG, MODE, 8>(a, used);
    case 16: return launch_k<TI, TG, MODE, 16>(a, used);
    default: return hipSuccess;
  }
}

template <class TI>
hipError_t launch_in(const LossArgs& a, bool* used) {
  const bool bf_grad = a.gd == DType::kBf16;
  if (a.mode == Mode::kEal)
    return bf_grad ? launch_mode<TI, GBf16, int(Mode::kEal)>(a, used) : launch_mode<TI, GF32, int(Mode::kEal)>(a, used);
  return bf_grad ? launch_mode<TI, GBf16, int(Mode::kWtv)>(a, used) : launch_mode<TI, GF32, int(Mode::kWtv)>(a, used);
}

}  // namespace

hipError_t launch_resident(const LossArgs& a, bool* used) {
  *used = false;
  const int E = a.in == DType::kBf16 ? Bf16::kVec : F32::kVec;
  if (a.V % E != 0) return hipSuccess;
  return a.in == DType::kBf16 ? launch_in<Bf16>(a, used) : launch_in<F32>(a, used);
}

}  // namespace aal
