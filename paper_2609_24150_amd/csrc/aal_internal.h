// Host-side interfaces between the C-ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace aal {

enum class Mode : int { kEal = 0, kWtv = 1 };
enum class DType : int { kBf16 = 0, kF32 = 1 };

// Per-row statistics written by the row pass and read by the window scan and
// the gradient pass.  32 bytes.
//   msc_*: fl(max_v z_v * sc) with sc = log2(e)/T, the reference of the sums
//   l2s_*: log2 of sum_v 2^(z_v*sc - msc)
// so that log2 q(v) = (z_v*sc - msc) - l2s.
struct RowStats {
  float msc_d, l2s_d;
  float msc_t, l2s_t;
  float a;      // per-position acceptance
  float qlt;    // WTV: sum of q over entries with q < p
  float coef;   // gradient coefficient (window scan output)
  int32_t xstar;  // EAL: greedy target token
};
static_assert(sizeof(RowStats) == 32, "RowStats layout");

// Workspace carve-up (all offsets 256-byte aligned).
struct Workspace {
  RowStats* stats;   // rows
  float* window_e;   // windows
  uint8_t* resident; // fixed region for the resident schedule
  size_t resident_bytes;
};

constexpr size_t kResidentRegionBytes = size_t(4) << 20;

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

inline size_t workspace_bytes(int64_t rows, int64_t windows) {
  return align256(size_t(rows) * sizeof(RowStats)) + align256(size_t(windows) * sizeof(float)) +
         kResidentRegionBytes;
}

inline Workspace carve(void* base, int64_t rows, int64_t windows) {
  uint8_t* p = static_cast<uint8_t*>(base);
  Workspace w;
  w.stats = reinterpret_cast<RowStats*>(p);
  p += align256(size_t(rows) * sizeof(RowStats));
  w.window_e = reinterpret_cast<float*>(p);
  p += align256(size_t(windows) * sizeof(float));
  w.resident = p;
  w.resident_bytes = kResidentRegionBytes;
  return w;
}

// Arguments of one EAL/WTV call after validation.
struct LossArgs {
  Mode mode;
  DType in;
  DType gd;
  const void* zd;
  const void* zt;
  int64_t N;
  int K;
  int V;
  float sc_d;      // log2(e)/T_draft
  float sc_t;      // log2(e)/T_target (WTV)
  float inv_t_d;   // 1/T_draft
  float* loss;
  float* window_e;  // user array or workspace
  float* accept;    // may be null
  int32_t* xstar;   // may be null
  void* grad;       // may be null
  const float* grad_scale;  // may be null
  Workspace ws;
  bool coop;       // resident schedule: the runtime's cooperative launch
  hipStream_t stream;
};

// Multi-kernel streaming schedule: row pass, window scan, loss reduction,
// gradient pass.  Handles every shape.
hipError_t launch_streaming(const LossArgs& a);

// loss = -(1/N) sum_n window_e[n], one workgroup, fixed summation order.
// err: the error word of a resident kernel (NaN loss when set), or null
hipError_t launch_loss_reduce(const LossArgs& a, const unsigned* err = nullptr);

// Register-resident single-kernel schedule.  Sets *used = false (and enqueues
// nothing) when the shape is outside what it supports: V not a multiple of the 16-byte vector, K outside {1..8, 16}, a window too
// wide for the co-resident grid, or (with a.coop) no cooperative launch on
// the device.
hipError_t launch_resident(const LossArgs& a, bool* used);

// Per-row statistics of the combined-objective schedule.  64 bytes.
struct GenStats {
  float msc_d, l2s_d;  // draft: fl(max * sc), log2 of the sum (as RowStats)
  float msc_t, l2s_t;  // target, when a TV or KL term is asked for
  float a_tv;          // sum_v min(p, q)
  float qlt;           // sum of q over entries with q < p
  float a_eal;         // q(x*)
  float kl;            // KL(p || q) in nats
  int32_t xstar;       // greedy target token or label (-1: no EAL term)
  float cA, cB;        // gradient: q (m ? cA : cB) + cP p + cX 1[v = x*]
  float cX, cP;
  float tv_w;          // (windows containing the row) * (1 - a_tv)
  float pad[2];
};
static_assert(sizeof(GenStats) == 64, "GenStats layout");

// Tagged partial slots of the combined-objective resident schedule (teams *
// members <= the co-resident workgroups; 16 words per row and member).
constexpr size_t kGenResidentSlotBytes = size_t(2) << 20;

// Blocks of the first stage of the combined objective's loss reduction.
constexpr int kGenLossParts = 64;

inline size_t general_workspace_bytes(int64_t rows, int64_t windows) {
  return align256(size_t(rows) * sizeof(GenStats)) + 2 * align256(size_t(windows) * sizeof(float)) +
         kGenResidentSlotBytes + align256(size_t(rows) * 2 * sizeof(uint64_t)) + 256 +
         align256(size_t(kGenLossParts) * 4 * sizeof(double));
}

struct GenArgs {
  DType in;
  DType gd;
  const void* zd;
  const void* zt;          // may be null when no term needs the target
  const int32_t* labels;   // may be null
  int layout;              // 0 windows, 1 sequences
  int64_t B;
  int S, K, V;
  int64_t R, W;            // rows, windows
  float sc_d, sc_t, inv_t_d;
  float w_wtv, w_eal, w_kl, w_tv;
  float* loss;
  float* terms;            // may be null
  float* e_tv;             // may be null
  float* e_eal;            // may be null
  float* accept_tv;        // may be null
  float* accept_eal;       // may be null
  int32_t* xstar;          // may be null
  void* grad;              // may be null
  const float* grad_scale; // may be null
  GenStats* stats;         // workspace [R]
  float* win_tv;           // workspace [W]
  float* win_eal;          // workspace [W]
  uint64_t* res_slots;     // workspace: resident schedule's tagged partials
  size_t res_slot_bytes;
  uint64_t* arow;          // workspace [R][2]: tagged acceptances of sliding-window chunks
  unsigned* res_err;       // workspace: poll time-out flag
  double* loss_parts;      // workspace [kGenLossParts][4]: first-stage sums of the loss
  bool streaming;          // force the multi-kernel schedule
  bool coop;               // resident schedule: the runtime's cooperative launch
  hipStream_t stream;
};

// The combined objective: the register-resident schedule when the shape
// allows it (V a multiple of the 16-byte vector, K in {1..8, 16}, target
// logits given, cooperative launch), else the row pass, window scan, loss and
// gradient pass of the streaming schedule, which handles every shape.
hipError_t launch_general(const GenArgs& a);

// Register-resident schedule of the combined objective; sets *used = false
// (enqueuing nothing) when the shape is outside what it supports.  The loss
// reduction and the time-out check are left to the caller.
hipError_t launch_general_resident(const GenArgs& a, bool* used);
hipError_t launch_general_resident_bf16(const GenArgs& a, bool* used);  // bf16 logits
hipError_t launch_general_resident_bf16_g32(const GenArgs& a, bool* used);  // bf16 logits, fp32 gradient
hipError_t launch_general_resident_f32(const GenArgs& a, bool* used);   // fp32 logits
// Loss reduction of the combined objective over the per-row and per-window
// values in the workspace.
// err: the error word of the resident kernel (NaN loss when set), or null
hipError_t launch_general_loss(const GenArgs& a, const unsigned* err = nullptr);

// Per-row quantities of the GRPO schedule.  32 bytes.
struct GrpoRow {
  int32_t s_theta;  // greedy token of the current draft
  int32_t s_ref;    // greedy token of the reference draft
  int32_t xstar;    // the target's greedy token or the label
  float lp_theta;   // log pi_theta(s_theta), natural log
  float lp_ref;     // log pi_ref(s_theta)
  float msc, l2s;   // current draft: fl(max * sc), log2 of the sum
  float pad;
};
static_assert(sizeof(GrpoRow) == 32, "GrpoRow layout");

inline size_t grpo_workspace_bytes(int64_t rows, int64_t groups, int64_t windows) {
  return align256(size_t(rows) * sizeof(GrpoRow)) + align256(size_t(windows) * sizeof(float)) +
         align256(size_t(groups) * sizeof(float));
}

struct GrpoArgs {
  DType in;
  DType gd;
  const void* zth;
  const void* zrf;
  const void* zt;          // null when labels are given
  const int32_t* labels;   // may be null
  int layout;
  int64_t B;
  int S, G, m, K, V;
  int64_t R;               // rows
  int64_t n_groups;
  const int32_t* anchors;  // sequences layout
  float sc, inv_t;
  float eps, adv_clip, eps_clip, rho_min, rho_max;
  float* loss;
  int32_t* tau_theta;      // optional [n_groups * m]
  int32_t* tau_ref;
  float* advantage;
  float* log_rho;
  void* grad;              // may be null
  const float* grad_scale; // may be null
  GrpoRow* rows;           // workspace
  float* win_coef;         // workspace [n_groups * m]
  float* group_loss;       // workspace [n_groups]
  hipStream_t stream;
};

hipError_t launch_grpo(const GrpoArgs& a);

// The streaming probe behind aal_stream_probe: n_src (1..3) sources of `bytes`
// bytes each (a multiple of 16), summed into dst when dst is not null.
hipError_t launch_stream_probe(const void* const src[3], int n_src, void* dst, size_t bytes, uint32_t* flag,
                               hipStream_t stream);

struct SimArgs {
  DType in;
  const void* zd;
  const void* zt;
  int P, G, K, V;
  float sc;
  const float* u1;
  const float* u2;
  int32_t* token;   // rows (user or workspace)
  int32_t* accept;  // rows (user or workspace)
  int32_t* reward;
  float* advantage;
  float eps;
  int ddof;
  float clip;
  hipStream_t stream;
};

hipError_t launch_sim(const SimArgs& a);

}  // namespace aal
