// Host-only stand-ins for libaal's kernel launchers, for the sanitizer build
// of the C-ABI layer (csrc/aal_api.hip).  Each stand-in writes every byte of
// the workspace regions its kernels would use, so that AddressSanitizer checks
// the workspace carve-up against a host buffer of exactly the advertised
// size; it never touches the (fake) device pointers of logits and outputs.
#include <string.h>

#include "aal_internal.h"
#include "aal_vp.h"

namespace aal {

int g_stub_calls = 0;  // launches that reached a stand-in (read by the driver)

namespace {
void touch(void* p, size_t n) {
  if (p && n) memset(p, 0xA5, n);
}
}  // namespace

hipError_t launch_resident(const LossArgs& a, bool* used) {
  touch(a.ws.resident, a.ws.resident_bytes);
  *used = false;  // fall through to the streaming stand-in, as for an unsupported shape
  return hipSuccess;
}

hipError_t launch_streaming(const LossArgs& a) {
  ++g_stub_calls;
  touch(a.ws.stats, size_t(a.N) * a.K * sizeof(RowStats));
  if (a.window_e == a.ws.window_e) touch(a.ws.window_e, size_t(a.N) * sizeof(float));
  return hipSuccess;
}

hipError_t launch_general(const GenArgs& a) {
  ++g_stub_calls;
  touch(a.stats, size_t(a.R) * sizeof(GenStats));
  touch(a.win_tv, size_t(a.W) * sizeof(float));
  touch(a.win_eal, size_t(a.W) * sizeof(float));
  touch(a.res_slots, a.res_slot_bytes);
  touch(a.arow, size_t(a.R) * 2 * sizeof(uint64_t));
  touch(a.res_err, sizeof(unsigned));
  touch(a.loss_parts, size_t(kGenLossParts) * 4 * sizeof(double));
  return hipSuccess;
}

hipError_t launch_grpo(const GrpoArgs& a) {
  ++g_stub_calls;
  touch(a.rows, size_t(a.R) * sizeof(GrpoRow));
  touch(a.win_coef, size_t(a.n_groups) * a.m * sizeof(float));
  touch(a.group_loss, size_t(a.n_groups) * sizeof(float));
  return hipSuccess;
}

hipError_t launch_sim(const SimArgs& a) {
  ++g_stub_calls;
  // token and accept fall back to the workspace when the caller passes none;
  // the driver passes none, so both are host memory here
  const size_t rows = size_t(a.P) * a.G * a.K;
  touch(a.token, rows * sizeof(int32_t));
  touch(a.accept, rows * sizeof(int32_t));
  return hipSuccess;
}

hipError_t launch_vp_partials(const VpSlice&, aal_vp_part_t*) { ++g_stub_calls; return hipSuccess; }
hipError_t launch_vp_merge(const aal_vp_part_t*, int32_t, int64_t, Mode, float, float, aal_vp_row_t*, hipStream_t) {
  ++g_stub_calls;
  return hipSuccess;
}
hipError_t launch_vp_accept(const VpSlice&, const aal_vp_row_t*, aal_vp_acc_t*) { ++g_stub_calls; return hipSuccess; }
hipError_t launch_vp_scan(aal_vp_row_t*, const aal_vp_acc_t*, int32_t, int64_t, int32_t, Mode, float, const float*, float*,
                          float*, float*, int32_t*, hipStream_t) {
  ++g_stub_calls;
  return hipSuccess;
}
hipError_t launch_vp_seq_scan(aal_vp_row_t*, const aal_vp_acc_t*, int32_t, int64_t, int32_t, int32_t, Mode, float,
                              const float*, float*, float*, float*, int32_t*, hipStream_t) {
  ++g_stub_calls;
  return hipSuccess;
}
hipError_t launch_vp_grad(const VpSlice&, const aal_vp_row_t*, void*, DType) { ++g_stub_calls; return hipSuccess; }

hipError_t launch_stream_probe(const void* const*, int, void*, size_t, uint32_t*, hipStream_t) {
  ++g_stub_calls;
  return hipSuccess;
}

}  // namespace aal
