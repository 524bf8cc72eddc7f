// Host-side interface of the vocabulary-parallel kernels (aal_vp.hip): the
// C-ABI layer validates the arguments and calls these launchers.
#pragma once

#include "aal.h"
#include "aal_internal.h"

namespace aal {

// One vocabulary slice of `rows` rows, row stride V_slice elements.
struct VpSlice {
  const void* zd;
  const void* zt;
  const int32_t* labels;  // EAL: [rows] global token ids replacing the greedy token, or null
  DType in;
  int64_t rows;
  int32_t vs;    // V_slice
  int32_t v0;    // global index of the slice's first entry
  int32_t vtot;  // the whole vocabulary (labels are clamped into [0, vtot))
  Mode mode;
  float scd, sct;  // log2(e)/T of draft and target
  hipStream_t stream;
};

hipError_t launch_vp_partials(const VpSlice& s, aal_vp_part_t* parts);
hipError_t launch_vp_merge(const aal_vp_part_t* parts_all, int32_t R, int64_t rows, Mode mode, float scd, float sct,
                           aal_vp_row_t* row, hipStream_t stream);
hipError_t launch_vp_accept(const VpSlice& s, const aal_vp_row_t* row, aal_vp_acc_t* acc);
hipError_t launch_vp_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R, int64_t N, int32_t K, Mode mode,
                          float inv_t_d, const float* grad_scale, float* loss, float* window_e, float* accept,
                          int32_t* xstar, hipStream_t stream);
hipError_t launch_vp_seq_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R, int64_t B, int32_t S,
                              int32_t K, Mode mode, float inv_t_d, const float* grad_scale, float* loss,
                              float* window_e, float* accept, int32_t* xstar, hipStream_t stream);
hipError_t launch_vp_grad(const VpSlice& s, const aal_vp_row_t* row, void* grad, DType gd);

}  // namespace aal
