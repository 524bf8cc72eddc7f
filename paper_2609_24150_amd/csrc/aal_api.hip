// C ABI of libaal: argument validation, workspace carve-up and dispatch.
// Declarations and the contract of every entry point are in include/aal.h.
#include "aal.h"
#include "aal_internal.h"
#include "aal_vp.h"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>

// Device scratch of aal_wtv_fwd_bwd_noalloc: a file-scope array in the code
// object, so that entry point never allocates.  Each GPU holds its own copy
// at its own address until the process ends.  Host code never uses the name
// as an address: it takes the per-device address from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[AAL_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr uint32_t kKnownFlags = AAL_FLAG_STREAMING | AAL_FLAG_COOPERATIVE;

// A plain per-thread buffer: nothing to construct or destroy at thread or
// process exit.
thread_local char g_last_error[512];

void clear_error() { g_last_error[0] = '\0'; }

aal_status_t fail(aal_status_t s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return s;
}

// Finite and > 0, checked on the bit pattern so that no floating-point
// compilation mode can fold the test away.
bool positive_finite(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  const bool sign = (u >> 31) != 0;
  const uint32_t expo = (u >> 23) & 0xffu;
  return !sign && expo != 0xffu && (u & 0x7fffffffu) != 0;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// The integer held by an enum argument, read without loading it as the enum
// type: a C caller may pass any int, and values outside the enumerators are
// validated here rather than assumed away.
template <class E>
int raw(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "enum arguments are int-sized");
  int v;
  memcpy(&v, &e, sizeof v);
  return v;
}

bool valid_dtype(int d) { return d == AAL_BF16 || d == AAL_F32; }

aal::DType to_dtype(int d) { return d == AAL_BF16 ? aal::DType::kBf16 : aal::DType::kF32; }

constexpr double kLog2e = 1.4426950408889634073599246810019;

// log2(e)/T as a finite positive float, or 0 if it is not representable.
float scale_for(float T) {
  const double s = kLog2e / double(T);
  if (!(s < 3.0e38)) return 0.f;
  const float f = float(s);
  return positive_finite(f) ? f : 0.f;
}

struct CommonIn {
  const void* zd;
  const void* zt;
  int in_dtype;
  int64_t N;
  int32_t K;
  int32_t V;
  float* loss;
  void* grad;
  int grad_dtype;
  void* workspace;
  size_t workspace_bytes;
};

aal_status_t validate_common(const CommonIn& c) {
  if (!c.zd || !c.zt) return fail(AAL_ERR_ARG, "z_draft and z_target must be non-NULL");
  if (!c.loss) return fail(AAL_ERR_ARG, "loss must be non-NULL");
  if (c.N < 1) return fail(AAL_ERR_ARG, "N must be >= 1 (got %lld)", (long long)c.N);
  if (c.K < 1 || c.K > 64) return fail(AAL_ERR_ARG, "K must be in [1, 64] (got %d)", c.K);
  if (c.V < 1) return fail(AAL_ERR_ARG, "V must be >= 1 (got %d)", c.V);
  if (c.N > (int64_t(1) << 31) / c.K) return fail(AAL_ERR_ARG, "N*K must be < 2^31");
  if (c.N * c.K > (int64_t(1) << 62) / c.V) return fail(AAL_ERR_ARG, "N*K*V must be < 2^62");
  if (!valid_dtype(c.in_dtype)) return fail(AAL_ERR_DTYPE, "unknown in_dtype %d", c.in_dtype);
  if (c.grad && !valid_dtype(c.grad_dtype)) return fail(AAL_ERR_DTYPE, "unknown grad_dtype %d", c.grad_dtype);
  if (!aligned(c.zd, 16) || !aligned(c.zt, 16)) return fail(AAL_ERR_ALIGN, "logit pointers must be 16-byte aligned");
  if (c.grad && !aligned(c.grad, 16)) return fail(AAL_ERR_ALIGN, "grad_draft must be 16-byte aligned");
  if (!c.workspace) return fail(AAL_ERR_WORKSPACE, "workspace must be non-NULL");
  if (!aligned(c.workspace, 256)) return fail(AAL_ERR_ALIGN, "workspace must be 256-byte aligned");
  const size_t need = aal::workspace_bytes(c.N * c.K, c.N);
  if (c.workspace_bytes < need)
    return fail(AAL_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", c.workspace_bytes, need);
  return AAL_OK;
}

aal_status_t run_loss(aal::LossArgs& a, uint32_t flags) {
  a.coop = (flags & AAL_FLAG_COOPERATIVE) != 0;
  bool used = false;
  hipError_t e = hipSuccess;
  if (!(flags & AAL_FLAG_STREAMING)) e = aal::launch_resident(a, &used);
  if (e == hipSuccess && !used) e = aal::launch_streaming(a);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

// Shared checks of the vocabulary-parallel slice calls.
aal_status_t validate_vp_slice(const void* zd, const void* zt, bool need_zt, int in_dtype, int64_t rows,
                               int32_t vs, int32_t v0) {
  if (!zd || (need_zt && !zt)) return fail(AAL_ERR_ARG, "z_draft and z_target must be non-NULL");
  if (rows < 1) return fail(AAL_ERR_ARG, "rows must be >= 1 (got %lld)", (long long)rows);
  if (vs < 1) return fail(AAL_ERR_ARG, "V_slice must be >= 1 (got %d)", vs);
  if (v0 < 0 || int64_t(v0) + vs > int64_t(INT32_MAX))
    return fail(AAL_ERR_ARG, "v0 must be >= 0 with v0 + V_slice < 2^31 (got v0 = %d)", v0);
  if (rows > (int64_t(1) << 62) / vs) return fail(AAL_ERR_ARG, "rows*V_slice must be < 2^62");
  if (!valid_dtype(in_dtype)) return fail(AAL_ERR_DTYPE, "unknown in_dtype %d", in_dtype);
  if (!aligned(zd, 16) || (zt && !aligned(zt, 16))) return fail(AAL_ERR_ALIGN, "logit pointers must be 16-byte aligned");
  return AAL_OK;
}

bool valid_vp_mode(int m) { return m == AAL_VP_EAL || m == AAL_VP_WTV; }

aal_status_t vp_scales(int mode, float temp_draft, float temp_target, float* scd, float* sct) {
  *scd = scale_for(temp_draft);
  if (!positive_finite(temp_draft) || *scd == 0.f)
    return fail(AAL_ERR_ARG, "temp_draft must be finite, > 0 and >= 1e-37");
  *sct = 0.f;
  if (mode == AAL_VP_WTV) {
    *sct = scale_for(temp_target);
    if (!positive_finite(temp_target) || *sct == 0.f)
      return fail(AAL_ERR_ARG, "temp_target must be finite, > 0 and >= 1e-37");
  }
  return AAL_OK;
}

aal::Mode vp_mode(int m) { return m == AAL_VP_EAL ? aal::Mode::kEal : aal::Mode::kWtv; }

// Per-device address of `scratch`, looked up once per device with that device
// current (0 = not yet looked up).  Atomics: nothing to destroy at exit.
constexpr int kMaxScratchDevices = 64;
std::atomic<uintptr_t> g_scratch_addr[kMaxScratchDevices];

aal_status_t scratch_for_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(AAL_ERR_ARG, "device %d is beyond the %d devices the static scratch serves", dev,
                kMaxScratchDevices);
  uintptr_t a = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (a == 0) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(AAL_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(e));
    a = reinterpret_cast<uintptr_t>(p);
    g_scratch_addr[dev].store(a, std::memory_order_release);
  }
  *out = reinterpret_cast<void*>(a);
  return AAL_OK;
}

}  // namespace

extern "C" {

int aal_version(void) { return 100; }

size_t aal_workspace_bytes(int64_t rows, int64_t windows) {
  if (rows < 0 || windows < 0) return 0;
  return aal::workspace_bytes(rows, windows);
}

const char* aal_status_string(aal_status_t status) {
  switch (raw(status)) {
    case AAL_OK: return "AAL_OK";
    case AAL_ERR_ARG: return "AAL_ERR_ARG: invalid argument";
    case AAL_ERR_DTYPE: return "AAL_ERR_DTYPE: unsupported element type";
    case AAL_ERR_ALIGN: return "AAL_ERR_ALIGN: misaligned pointer";
    case AAL_ERR_WORKSPACE: return "AAL_ERR_WORKSPACE: workspace missing or too small";
    case AAL_ERR_HIP: return "AAL_ERR_HIP: HIP runtime error";
    default: return "unknown status";
  }
}

const char* aal_last_error(void) { return g_last_error; }

}  // extern "C"

namespace {

// The bodies of the EAL, WTV and simulation entry points, with the element
// types as the integers the caller passed.
aal_status_t eal_impl(const void* z_draft, const void* z_target, int in_dtype, int64_t N, int32_t K, int32_t V,
                      float temp_draft, float* loss, float* eal_per_window, float* accept, int32_t* target_argmax,
                      void* grad_draft, int grad_dtype, const float* grad_scale, uint32_t flags, void* workspace,
                      size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  const CommonIn c{z_draft, z_target, raw(in_dtype), N, K, V, loss, grad_draft, raw(grad_dtype),
                   workspace, workspace_bytes};
  aal_status_t s = validate_common(c);
  if (s != AAL_OK) return s;
  const float scd = scale_for(temp_draft);
  if (!positive_finite(temp_draft) || scd == 0.f)
    return fail(AAL_ERR_ARG, "temp_draft must be finite, > 0 and >= 1e-37");
  if (flags & ~kKnownFlags) return fail(AAL_ERR_ARG, "unknown flags 0x%x", flags);
  aal::LossArgs a{};
  a.mode = aal::Mode::kEal;
  a.in = to_dtype(raw(in_dtype));
  a.gd = to_dtype(raw(grad_dtype));
  a.zd = z_draft;
  a.zt = z_target;
  a.N = N;
  a.K = K;
  a.V = V;
  a.sc_d = scd;
  a.sc_t = 0.f;
  a.inv_t_d = 1.0f / temp_draft;
  a.loss = loss;
  a.ws = aal::carve(workspace, N * K, N);
  a.window_e = eal_per_window ? eal_per_window : a.ws.window_e;
  a.accept = accept;
  a.xstar = target_argmax;
  a.grad = grad_draft;
  a.grad_scale = grad_scale;
  a.stream = stream;
  return run_loss(a, flags);
}

aal_status_t wtv_impl(const void* z_draft, const void* z_target, int in_dtype, int64_t N, int32_t K, int32_t V,
                      float temp_draft, float temp_target, float* loss, float* eal_per_window, float* accept,
                      void* grad_draft, int grad_dtype, const float* grad_scale, uint32_t flags, void* workspace,
                      size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  const CommonIn c{z_draft, z_target, raw(in_dtype), N, K, V, loss, grad_draft, raw(grad_dtype),
                   workspace, workspace_bytes};
  aal_status_t s = validate_common(c);
  if (s != AAL_OK) return s;
  const float scd = scale_for(temp_draft);
  const float sct = scale_for(temp_target);
  if (!positive_finite(temp_draft) || scd == 0.f)
    return fail(AAL_ERR_ARG, "temp_draft must be finite, > 0 and >= 1e-37");
  if (!positive_finite(temp_target) || sct == 0.f)
    return fail(AAL_ERR_ARG, "temp_target must be finite, > 0 and >= 1e-37");
  if (flags & ~kKnownFlags) return fail(AAL_ERR_ARG, "unknown flags 0x%x", flags);
  aal::LossArgs a{};
  a.mode = aal::Mode::kWtv;
  a.in = to_dtype(raw(in_dtype));
  a.gd = to_dtype(raw(grad_dtype));
  a.zd = z_draft;
  a.zt = z_target;
  a.N = N;
  a.K = K;
  a.V = V;
  a.sc_d = scd;
  a.sc_t = sct;
  a.inv_t_d = 1.0f / temp_draft;
  a.loss = loss;
  a.ws = aal::carve(workspace, N * K, N);
  a.window_e = eal_per_window ? eal_per_window : a.ws.window_e;
  a.accept = accept;
  a.xstar = nullptr;
  a.grad = grad_draft;
  a.grad_scale = grad_scale;
  a.stream = stream;
  return run_loss(a, flags);
}

aal_status_t sim_impl(const void* z_draft, const void* z_target, int in_dtype, int32_t P, int32_t G, int32_t K,
                      int32_t V, float temperature, const float* u1, const float* u2, int32_t* draft_token,
                      int32_t* accept, int32_t* reward, float* advantage, float eps, int32_t std_ddof,
                      float adv_clip, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  if (!z_draft || !z_target || !u1 || !u2) return fail(AAL_ERR_ARG, "z_draft, z_target, u1, u2 must be non-NULL");
  if (!reward || !advantage) return fail(AAL_ERR_ARG, "reward and advantage must be non-NULL");
  if (P < 1 || G < 1 || K < 1 || V < 1) return fail(AAL_ERR_ARG, "P, G, K, V must be >= 1");
  if (V > (1 << 21)) return fail(AAL_ERR_ARG, "V must be <= 2^21 (got %d)", V);
  if (std_ddof < 0 || G <= std_ddof) return fail(AAL_ERR_ARG, "need 0 <= std_ddof < G");
  const int64_t rows = int64_t(P) * G * K;
  if (rows >= (int64_t(1) << 31)) return fail(AAL_ERR_ARG, "P*G*K must be < 2^31");
  if (!valid_dtype(raw(in_dtype))) return fail(AAL_ERR_DTYPE, "unknown in_dtype %d", raw(in_dtype));
  const float sc = scale_for(temperature);
  if (!positive_finite(temperature) || sc == 0.f)
    return fail(AAL_ERR_ARG, "temperature must be finite, > 0 and >= 1e-37");
  uint32_t eb;
  memcpy(&eb, &eps, sizeof eb);
  if ((eb >> 31) || ((eb >> 23) & 0xffu) == 0xffu) return fail(AAL_ERR_ARG, "eps must be finite and >= 0");
  if (!aligned(z_draft, 16) || !aligned(z_target, 16)) return fail(AAL_ERR_ALIGN, "logit pointers must be 16-byte aligned");
  if (!workspace) return fail(AAL_ERR_WORKSPACE, "workspace must be non-NULL");
  if (!aligned(workspace, 256)) return fail(AAL_ERR_ALIGN, "workspace must be 256-byte aligned");
  const size_t need = aal::workspace_bytes(rows, int64_t(P) * G);
  if (workspace_bytes < need) return fail(AAL_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  aal::Workspace ws = aal::carve(workspace, rows, int64_t(P) * G);
  int32_t* scratch = reinterpret_cast<int32_t*>(ws.stats);  // rows * 32 bytes >= 2 int32 per row
  aal::SimArgs a{};
  a.in = to_dtype(raw(in_dtype));
  a.zd = z_draft;
  a.zt = z_target;
  a.P = P;
  a.G = G;
  a.K = K;
  a.V = V;
  a.sc = sc;
  a.u1 = u1;
  a.u2 = u2;
  a.token = draft_token ? draft_token : scratch;
  a.accept = accept ? accept : scratch + rows;
  a.reward = reward;
  a.advantage = advantage;
  a.eps = eps;
  a.ddof = std_ddof;
  a.clip = adv_clip;
  a.stream = stream;
  hipError_t e = aal::launch_sim(a);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

}  // namespace

extern "C" {

aal_status_t aal_eal_fwd_bwd_ex(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t N,
                                int32_t K, int32_t V, float temp_draft, float* loss, float* eal_per_window,
                                float* accept, int32_t* target_argmax, void* grad_draft, aal_dtype_t grad_dtype,
                                const float* grad_scale, uint32_t flags, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  return eal_impl(z_draft, z_target, raw(in_dtype), N, K, V, temp_draft, loss, eal_per_window, accept, target_argmax,
                  grad_draft, raw(grad_dtype), grad_scale, flags, workspace, workspace_bytes, stream);
}

aal_status_t aal_eal_fwd_bwd(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t N, int32_t K,
                             int32_t V, float temp_draft, float* loss, float* eal_per_window, float* accept,
                             int32_t* target_argmax, void* grad_draft, aal_dtype_t grad_dtype,
                             const float* grad_scale, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return eal_impl(z_draft, z_target, raw(in_dtype), N, K, V, temp_draft, loss, eal_per_window, accept, target_argmax,
                  grad_draft, raw(grad_dtype), grad_scale, 0u, workspace, workspace_bytes, stream);
}

aal_status_t aal_wtv_fwd_bwd_ex(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t N,
                                int32_t K, int32_t V, float temp_draft, float temp_target, float* loss,
                                float* eal_per_window, float* accept, void* grad_draft, aal_dtype_t grad_dtype,
                                const float* grad_scale, uint32_t flags, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  return wtv_impl(z_draft, z_target, raw(in_dtype), N, K, V, temp_draft, temp_target, loss, eal_per_window, accept,
                  grad_draft, raw(grad_dtype), grad_scale, flags, workspace, workspace_bytes, stream);
}

aal_status_t aal_sim_accept_grpo_ex(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int32_t P,
                                    int32_t G, int32_t K, int32_t V, float temperature, const float* u1,
                                    const float* u2, int32_t* draft_token, int32_t* accept, int32_t* reward,
                                    float* advantage, float eps, int32_t std_ddof, float adv_clip, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
  return sim_impl(z_draft, z_target, raw(in_dtype), P, G, K, V, temperature, u1, u2, draft_token, accept, reward,
                  advantage, eps, std_ddof, adv_clip, workspace, workspace_bytes, stream);
}

aal_status_t aal_wtv_fwd_bwd(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t N, int32_t K,
                             int32_t V, float temp_draft, float temp_target, float* loss, float* eal_per_window,
                             float* accept, void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return wtv_impl(z_draft, z_target, raw(in_dtype), N, K, V, temp_draft, temp_target, loss, eal_per_window, accept,
                  grad_draft, raw(grad_dtype), grad_scale, 0u, workspace, workspace_bytes, stream);
}

aal_status_t aal_sim_accept_grpo(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int32_t P,
                                 int32_t G, int32_t K, int32_t V, float temperature, const float* u1,
                                 const float* u2, int32_t* draft_token, int32_t* reward, float* advantage, float eps,
                                 int32_t std_ddof, float adv_clip, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
  return sim_impl(z_draft, z_target, raw(in_dtype), P, G, K, V, temperature, u1, u2, draft_token, nullptr, reward,
                  advantage, eps, std_ddof, adv_clip, workspace, workspace_bytes, stream);
}

aal_status_t aal_wtv_fwd_bwd_noalloc(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t N,
                                     int32_t K, int32_t V, float temp_draft, float temp_target, float* loss,
                                     float* eal_per_window, float* accept, void* grad_draft, aal_dtype_t grad_dtype,
                                     const float* grad_scale, hipStream_t stream) {
  clear_error();
  if (N < 1) return fail(AAL_ERR_ARG, "N must be >= 1 (got %lld)", (long long)N);
  if (K < 1 || K > 64) return fail(AAL_ERR_ARG, "K must be in [1, 64] (got %d)", K);
  if (N > (int64_t(1) << 31) / K) return fail(AAL_ERR_ARG, "N*K must be < 2^31");
  const size_t need = aal::workspace_bytes(N * K, N);
  if (need > size_t(AAL_NOALLOC_SCRATCH_BYTES))
    return fail(AAL_ERR_WORKSPACE,
                "aal_wtv_fwd_bwd_noalloc: N=%lld, K=%d needs %zu bytes of scratch, more than the %zu bytes of "
                "the static scratch buffer",
                (long long)N, K, need, size_t(AAL_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  const aal_status_t st = scratch_for_current_device(&ws);
  if (st != AAL_OK) return st;
  return wtv_impl(z_draft, z_target, raw(in_dtype), N, K, V, temp_draft, temp_target, loss, eal_per_window, accept,
                  grad_draft, raw(grad_dtype), grad_scale, 0u, ws, size_t(AAL_NOALLOC_SCRATCH_BYTES), stream);
}

size_t aal_loss_workspace_bytes(aal_layout_t layout, int64_t B, int32_t S, int32_t K) {
  if (B < 1 || K < 1 || (raw(layout) == AAL_LAYOUT_SEQUENCES && S < 1)) return 0;
  if (raw(layout) != AAL_LAYOUT_WINDOWS && raw(layout) != AAL_LAYOUT_SEQUENCES) return 0;
  const int64_t rows = raw(layout) == AAL_LAYOUT_WINDOWS ? B * K : B * S;
  const int64_t windows = raw(layout) == AAL_LAYOUT_WINDOWS ? B : B * int64_t(S >= K ? S - K + 1 : 0);
  return aal::general_workspace_bytes(rows, windows);
}

aal_status_t aal_loss_fwd_bwd(const void* z_draft, const void* z_target, const int32_t* labels, aal_dtype_t in_dtype,
                              aal_layout_t layout, int64_t B, int32_t S, int32_t K, int32_t V, float temp_draft,
                              float temp_target, aal_loss_weights_t weights, float* loss, float* terms, float* e_tv,
                              float* e_eal, float* accept_tv, float* accept_eal, int32_t* xstar, void* grad_draft,
                              aal_dtype_t grad_dtype, const float* grad_scale, uint32_t flags, void* workspace,
                              size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  if (raw(layout) != AAL_LAYOUT_WINDOWS && raw(layout) != AAL_LAYOUT_SEQUENCES)
    return fail(AAL_ERR_ARG, "unknown layout %d", raw(layout));
  if (B < 1) return fail(AAL_ERR_ARG, "B must be >= 1 (got %lld)", (long long)B);
  if (K < 1 || K > 64) return fail(AAL_ERR_ARG, "K must be in [1, 64] (got %d)", K);
  if (V < 1) return fail(AAL_ERR_ARG, "V must be >= 1 (got %d)", V);
  if (raw(layout) == AAL_LAYOUT_SEQUENCES && S < 1) return fail(AAL_ERR_ARG, "S must be >= 1 (got %d)", S);
  const int64_t per = raw(layout) == AAL_LAYOUT_WINDOWS ? K : S;
  if (B > ((int64_t(1) << 31) - 1) / per) return fail(AAL_ERR_ARG, "the number of rows must be < 2^31");
  const int64_t R = B * per;
  if (R > (int64_t(1) << 62) / V) return fail(AAL_ERR_ARG, "rows*V must be < 2^62");
  const int64_t W = raw(layout) == AAL_LAYOUT_WINDOWS ? B : B * int64_t(S >= K ? S - K + 1 : 0);
  auto finite = [](float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    return ((u >> 23) & 0xffu) != 0xffu;
  };
  if (!finite(weights.wtv) || !finite(weights.eal) || !finite(weights.kl) || !finite(weights.tv))
    return fail(AAL_ERR_ARG, "weights must be finite");
  if (flags & ~kKnownFlags) return fail(AAL_ERR_ARG, "unknown flags 0x%x", flags);
  const bool need_pq = weights.wtv != 0.f || weights.tv != 0.f || weights.kl != 0.f;
  const bool need_t = need_pq || (weights.eal != 0.f && labels == nullptr);
  if (!z_draft) return fail(AAL_ERR_ARG, "z_draft must be non-NULL");
  if (need_t && !z_target)
    return fail(AAL_ERR_ARG, "z_target must be non-NULL unless only the EAL term is asked for with labels");
  if (!loss) return fail(AAL_ERR_ARG, "loss must be non-NULL");
  if (!valid_dtype(raw(in_dtype))) return fail(AAL_ERR_DTYPE, "unknown in_dtype %d", raw(in_dtype));
  if (grad_draft && !valid_dtype(raw(grad_dtype))) return fail(AAL_ERR_DTYPE, "unknown grad_dtype %d", raw(grad_dtype));
  if (!aligned(z_draft, 16) || (z_target && !aligned(z_target, 16)))
    return fail(AAL_ERR_ALIGN, "logit pointers must be 16-byte aligned");
  if (grad_draft && !aligned(grad_draft, 16)) return fail(AAL_ERR_ALIGN, "grad_draft must be 16-byte aligned");
  const float scd = scale_for(temp_draft);
  const float sct = scale_for(temp_target);
  if (!positive_finite(temp_draft) || scd == 0.f)
    return fail(AAL_ERR_ARG, "temp_draft must be finite, > 0 and >= 1e-37");
  if (!positive_finite(temp_target) || sct == 0.f)
    return fail(AAL_ERR_ARG, "temp_target must be finite, > 0 and >= 1e-37");
  if (!workspace) return fail(AAL_ERR_WORKSPACE, "workspace must be non-NULL");
  if (!aligned(workspace, 256)) return fail(AAL_ERR_ALIGN, "workspace must be 256-byte aligned");
  const size_t need = aal::general_workspace_bytes(R, W);
  if (workspace_bytes < need)
    return fail(AAL_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  uint8_t* wp = static_cast<uint8_t*>(workspace);
  aal::GenArgs a{};
  a.in = to_dtype(raw(in_dtype));
  a.gd = to_dtype(raw(grad_dtype));
  a.zd = z_draft;
  a.zt = need_t ? z_target : nullptr;
  a.labels = labels;
  a.layout = raw(layout);
  a.B = B;
  a.S = raw(layout) == AAL_LAYOUT_WINDOWS ? K : S;
  a.K = K;
  a.V = V;
  a.R = R;
  a.W = W;
  a.sc_d = scd;
  a.sc_t = sct;
  a.inv_t_d = 1.0f / temp_draft;
  a.w_wtv = weights.wtv;
  a.w_eal = weights.eal;
  a.w_kl = weights.kl;
  a.w_tv = weights.tv;
  a.loss = loss;
  a.terms = terms;
  a.e_tv = e_tv;
  a.e_eal = e_eal;
  a.accept_tv = accept_tv;
  a.accept_eal = accept_eal;
  a.xstar = xstar;
  a.grad = grad_draft;
  a.grad_scale = grad_scale;
  a.stats = reinterpret_cast<aal::GenStats*>(wp);
  wp += aal::align256(size_t(R) * sizeof(aal::GenStats));
  a.win_tv = reinterpret_cast<float*>(wp);
  wp += aal::align256(size_t(W) * sizeof(float));
  a.win_eal = reinterpret_cast<float*>(wp);
  wp += aal::align256(size_t(W) * sizeof(float));
  a.res_slots = reinterpret_cast<uint64_t*>(wp);
  a.res_slot_bytes = aal::kGenResidentSlotBytes;
  wp += aal::kGenResidentSlotBytes;
  a.arow = reinterpret_cast<uint64_t*>(wp);
  wp += aal::align256(size_t(R) * 2 * sizeof(uint64_t));
  a.res_err = reinterpret_cast<unsigned*>(wp);
  wp += 256;
  a.loss_parts = reinterpret_cast<double*>(wp);
  a.streaming = (flags & AAL_FLAG_STREAMING) != 0;
  a.coop = (flags & AAL_FLAG_COOPERATIVE) != 0;
  a.stream = stream;
  hipError_t e = aal::launch_general(a);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

size_t aal_grpo_workspace_bytes(aal_layout_t layout, int64_t B, int32_t S, int32_t G, int32_t m, int32_t K) {
  if (B < 1 || K < 1 || m < 1) return 0;
  if (raw(layout) != AAL_LAYOUT_WINDOWS && raw(layout) != AAL_LAYOUT_SEQUENCES) return 0;
  if (raw(layout) == AAL_LAYOUT_SEQUENCES && (G < 1 || S < 1)) return 0;
  const int64_t groups = raw(layout) == AAL_LAYOUT_WINDOWS ? B : B * G;
  const int64_t rows = raw(layout) == AAL_LAYOUT_WINDOWS ? B * m * K : B * S;
  return aal::grpo_workspace_bytes(rows, groups, groups * m);
}

aal_status_t aal_grpo_fwd_bwd(const void* z_theta, const void* z_ref, const void* z_target, const int32_t* labels,
                              aal_dtype_t in_dtype, aal_layout_t layout, int64_t B, int32_t S, int32_t G, int32_t m,
                              int32_t K, int32_t V, const int32_t* anchors, float temperature,
                              aal_grpo_params_t params, float* loss, int32_t* tau_theta, int32_t* tau_ref,
                              float* advantage, float* log_rho, void* grad_theta, aal_dtype_t grad_dtype,
                              const float* grad_scale, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  clear_error();
  if (raw(layout) != AAL_LAYOUT_WINDOWS && raw(layout) != AAL_LAYOUT_SEQUENCES)
    return fail(AAL_ERR_ARG, "unknown layout %d", raw(layout));
  if (B < 1) return fail(AAL_ERR_ARG, "B must be >= 1 (got %lld)", (long long)B);
  if (K < 1 || K > 64) return fail(AAL_ERR_ARG, "K must be in [1, 64] (got %d)", K);
  if (m < 1 || m > 64) return fail(AAL_ERR_ARG, "m must be in [1, 64] (got %d)", m);
  if (V < 1) return fail(AAL_ERR_ARG, "V must be >= 1 (got %d)", V);
  const bool seq = raw(layout) == AAL_LAYOUT_SEQUENCES;
  if (seq) {
    if (G < 1) return fail(AAL_ERR_ARG, "G must be >= 1 (got %d)", G);
    if (S < m + K - 1) return fail(AAL_ERR_ARG, "S must be >= m + K - 1 (got S=%d, m=%d, K=%d)", S, m, K);
    if (!anchors) return fail(AAL_ERR_ARG, "anchors must be non-NULL for the sequences layout");
  }
  const int64_t per = seq ? int64_t(S) : int64_t(m) * K;
  if (B > ((int64_t(1) << 31) - 1) / per) return fail(AAL_ERR_ARG, "the number of rows must be < 2^31");
  const int64_t R = B * per;
  if (R > (int64_t(1) << 62) / V) return fail(AAL_ERR_ARG, "rows*V must be < 2^62");
  const int64_t groups = seq ? B * G : B;
  if (groups > (int64_t(1) << 31) / m) return fail(AAL_ERR_ARG, "groups*m must be < 2^31");
  if (!z_theta || !z_ref) return fail(AAL_ERR_ARG, "z_theta and z_ref must be non-NULL");
  if (!z_target && !labels) return fail(AAL_ERR_ARG, "z_target or labels must be given");
  if (!loss) return fail(AAL_ERR_ARG, "loss must be non-NULL");
  if (!valid_dtype(raw(in_dtype))) return fail(AAL_ERR_DTYPE, "unknown in_dtype %d", raw(in_dtype));
  if (grad_theta && !valid_dtype(raw(grad_dtype))) return fail(AAL_ERR_DTYPE, "unknown grad_dtype %d", raw(grad_dtype));
  if (!aligned(z_theta, 16) || !aligned(z_ref, 16) || (z_target && !aligned(z_target, 16)))
    return fail(AAL_ERR_ALIGN, "logit pointers must be 16-byte aligned");
  if (grad_theta && !aligned(grad_theta, 16)) return fail(AAL_ERR_ALIGN, "grad_theta must be 16-byte aligned");
  const float sc = scale_for(temperature);
  if (!positive_finite(temperature) || sc == 0.f)
    return fail(AAL_ERR_ARG, "temperature must be finite, > 0 and >= 1e-37");
  auto finite_nonneg = [](float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    return (u >> 31) == 0 && ((u >> 23) & 0xffu) != 0xffu;
  };
  auto nonneg = [](float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    return (u >> 31) == 0 && !(((u >> 23) & 0xffu) == 0xffu && (u & 0x7fffffu) != 0);  // +inf allowed, NaN not
  };
  uint32_t ac;
  memcpy(&ac, &params.adv_clip, sizeof ac);
  if (!finite_nonneg(params.eps)) return fail(AAL_ERR_ARG, "eps must be finite and >= 0");
  if (((ac >> 23) & 0xffu) == 0xffu) return fail(AAL_ERR_ARG, "adv_clip must be finite");
  if (!finite_nonneg(params.eps_clip)) return fail(AAL_ERR_ARG, "eps_clip must be finite and >= 0");
  if (!finite_nonneg(params.rho_min) || !nonneg(params.rho_max) || params.rho_max < params.rho_min)
    return fail(AAL_ERR_ARG, "need 0 <= rho_min <= rho_max (rho_min finite)");
  if (!workspace) return fail(AAL_ERR_WORKSPACE, "workspace must be non-NULL");
  if (!aligned(workspace, 256)) return fail(AAL_ERR_ALIGN, "workspace must be 256-byte aligned");
  const size_t need = aal::grpo_workspace_bytes(R, groups, groups * m);
  if (workspace_bytes < need)
    return fail(AAL_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  uint8_t* wp = static_cast<uint8_t*>(workspace);
  aal::GrpoArgs a{};
  a.in = to_dtype(raw(in_dtype));
  a.gd = to_dtype(raw(grad_dtype));
  a.zth = z_theta;
  a.zrf = z_ref;
  a.zt = labels ? nullptr : z_target;
  a.labels = labels;
  a.layout = raw(layout);
  a.B = B;
  a.S = seq ? S : m * K;
  a.G = seq ? G : 1;
  a.m = m;
  a.K = K;
  a.V = V;
  a.R = R;
  a.n_groups = groups;
  a.anchors = seq ? anchors : nullptr;
  a.sc = sc;
  a.inv_t = 1.0f / temperature;
  a.eps = params.eps;
  a.adv_clip = params.adv_clip;
  a.eps_clip = params.eps_clip;
  a.rho_min = params.rho_min;
  a.rho_max = params.rho_max;
  a.loss = loss;
  a.tau_theta = tau_theta;
  a.tau_ref = tau_ref;
  a.advantage = advantage;
  a.log_rho = log_rho;
  a.grad = grad_theta;
  a.grad_scale = grad_scale;
  a.rows = reinterpret_cast<aal::GrpoRow*>(wp);
  wp += aal::align256(size_t(R) * sizeof(aal::GrpoRow));
  a.win_coef = reinterpret_cast<float*>(wp);
  wp += aal::align256(size_t(groups * m) * sizeof(float));
  a.group_loss = reinterpret_cast<float*>(wp);
  a.stream = stream;
  hipError_t e = aal::launch_grpo(a);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}


aal_status_t aal_vp_row_partials(const void* z_draft, const void* z_target, const int32_t* labels,
                                 aal_dtype_t in_dtype, int64_t rows, int32_t V_slice, int32_t v0, int32_t V_total,
                                 aal_vp_mode_t mode, float temp_draft, float temp_target, aal_vp_part_t* parts,
                                 hipStream_t stream) {
  clear_error();
  if (!valid_vp_mode(raw(mode))) return fail(AAL_ERR_ARG, "unknown mode %d", raw(mode));
  if (labels && raw(mode) != AAL_VP_EAL) return fail(AAL_ERR_ARG, "labels are for EAL mode only");
  if (labels && !aligned(labels, 4)) return fail(AAL_ERR_ALIGN, "labels must be 4-byte aligned");
  aal_status_t st = validate_vp_slice(z_draft, labels ? nullptr : z_target, !labels, raw(in_dtype), rows, V_slice,
                                      v0);
  if (st != AAL_OK) return st;
  if (V_total < 1 || int64_t(v0) + V_slice > V_total)
    return fail(AAL_ERR_ARG, "V_total must hold the slice: v0 + V_slice <= V_total (got %d + %d > %d)", v0, V_slice,
                V_total);
  if (!parts) return fail(AAL_ERR_ARG, "parts must be non-NULL");
  if (!aligned(parts, 4)) return fail(AAL_ERR_ALIGN, "parts must be 4-byte aligned");
  aal::VpSlice s{};
  if ((st = vp_scales(raw(mode), temp_draft, temp_target, &s.scd, &s.sct)) != AAL_OK) return st;
  s.zd = z_draft;
  s.zt = labels ? nullptr : z_target;
  s.labels = labels;
  s.in = to_dtype(raw(in_dtype));
  s.rows = rows;
  s.vs = V_slice;
  s.v0 = v0;
  s.vtot = V_total;
  s.mode = vp_mode(raw(mode));
  s.stream = stream;
  const hipError_t e = aal::launch_vp_partials(s, parts);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

aal_status_t aal_vp_merge_rows(const aal_vp_part_t* parts_all, int32_t R, int64_t rows, aal_vp_mode_t mode,
                               float temp_draft, float temp_target, aal_vp_row_t* row, hipStream_t stream) {
  clear_error();
  if (!valid_vp_mode(raw(mode))) return fail(AAL_ERR_ARG, "unknown mode %d", raw(mode));
  if (!parts_all || !row) return fail(AAL_ERR_ARG, "parts_all and row must be non-NULL");
  if (R < 1) return fail(AAL_ERR_ARG, "R must be >= 1 (got %d)", R);
  if (rows < 1) return fail(AAL_ERR_ARG, "rows must be >= 1 (got %lld)", (long long)rows);
  if (rows > (int64_t(1) << 56) / R) return fail(AAL_ERR_ARG, "R*rows must be < 2^56");
  if (!aligned(parts_all, 4) || !aligned(row, 4)) return fail(AAL_ERR_ALIGN, "records must be 4-byte aligned");
  float scd, sct;
  aal_status_t st = vp_scales(raw(mode), temp_draft, temp_target, &scd, &sct);
  if (st != AAL_OK) return st;
  const hipError_t e =
      aal::launch_vp_merge(parts_all, R, rows, vp_mode(raw(mode)), scd, sct, row, stream);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

aal_status_t aal_vp_accept_partials(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t rows,
                                    int32_t V_slice, float temp_draft, float temp_target, const aal_vp_row_t* row,
                                    aal_vp_acc_t* acc, hipStream_t stream) {
  clear_error();
  aal_status_t st = validate_vp_slice(z_draft, z_target, true, raw(in_dtype), rows, V_slice, 0);
  if (st != AAL_OK) return st;
  if (!row || !acc) return fail(AAL_ERR_ARG, "row and acc must be non-NULL");
  if (!aligned(row, 4) || !aligned(acc, 4)) return fail(AAL_ERR_ALIGN, "records must be 4-byte aligned");
  aal::VpSlice s{};
  if ((st = vp_scales(AAL_VP_WTV, temp_draft, temp_target, &s.scd, &s.sct)) != AAL_OK) return st;
  s.zd = z_draft;
  s.zt = z_target;
  s.in = to_dtype(raw(in_dtype));
  s.rows = rows;
  s.vs = V_slice;
  s.v0 = 0;
  s.mode = aal::Mode::kWtv;
  s.stream = stream;
  const hipError_t e = aal::launch_vp_accept(s, row, acc);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

aal_status_t aal_vp_window_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R, int64_t N, int32_t K,
                                aal_vp_mode_t mode, float temp_draft, const float* grad_scale, float* loss,
                                float* eal_per_window, float* accept, int32_t* target_argmax, hipStream_t stream) {
  clear_error();
  if (!valid_vp_mode(raw(mode))) return fail(AAL_ERR_ARG, "unknown mode %d", raw(mode));
  if (!row || !loss || !eal_per_window) return fail(AAL_ERR_ARG, "row, loss and eal_per_window must be non-NULL");
  if (N < 1) return fail(AAL_ERR_ARG, "N must be >= 1 (got %lld)", (long long)N);
  if (K < 1 || K > 64) return fail(AAL_ERR_ARG, "K must be in [1, 64] (got %d)", K);
  if (N > (int64_t(1) << 31) / K) return fail(AAL_ERR_ARG, "N*K must be < 2^31");
  const bool wtv = raw(mode) == AAL_VP_WTV;
  if (wtv && !acc_all) return fail(AAL_ERR_ARG, "acc_all must be non-NULL in WTV mode");
  if (wtv && R < 1) return fail(AAL_ERR_ARG, "R must be >= 1 (got %d)", R);
  if (wtv && N * K > (int64_t(1) << 56) / R) return fail(AAL_ERR_ARG, "R*N*K must be < 2^56");
  if (!aligned(row, 4) || (wtv && !aligned(acc_all, 4))) return fail(AAL_ERR_ALIGN, "records must be 4-byte aligned");
  float scd, sct;
  aal_status_t st = vp_scales(AAL_VP_EAL, temp_draft, 1.f, &scd, &sct);
  if (st != AAL_OK) return st;
  const hipError_t e = aal::launch_vp_scan(row, wtv ? acc_all : nullptr, wtv ? R : 0, N, K, vp_mode(raw(mode)),
                                           1.0f / temp_draft, grad_scale, loss, eal_per_window, accept,
                                           wtv ? nullptr : target_argmax, stream);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

aal_status_t aal_vp_sequence_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R, int64_t B, int32_t S,
                                  int32_t K, aal_vp_mode_t mode, float temp_draft, const float* grad_scale,
                                  float* loss, float* eal_per_window, float* accept, int32_t* target_argmax,
                                  hipStream_t stream) {
  clear_error();
  if (!valid_vp_mode(raw(mode))) return fail(AAL_ERR_ARG, "unknown mode %d", raw(mode));
  if (!row || !loss || !eal_per_window) return fail(AAL_ERR_ARG, "row, loss and eal_per_window must be non-NULL");
  if (B < 1) return fail(AAL_ERR_ARG, "B must be >= 1 (got %lld)", (long long)B);
  if (K < 1 || K > 64) return fail(AAL_ERR_ARG, "K must be in [1, 64] (got %d)", K);
  if (S < K) return fail(AAL_ERR_ARG, "S must be >= K (got S = %d, K = %d)", S, K);
  if (B > (int64_t(1) << 31) / S) return fail(AAL_ERR_ARG, "B*S must be < 2^31");
  const bool wtv = raw(mode) == AAL_VP_WTV;
  if (wtv && !acc_all) return fail(AAL_ERR_ARG, "acc_all must be non-NULL in WTV mode");
  if (wtv && R < 1) return fail(AAL_ERR_ARG, "R must be >= 1 (got %d)", R);
  if (wtv && B * S > (int64_t(1) << 56) / R) return fail(AAL_ERR_ARG, "R*B*S must be < 2^56");
  if (!aligned(row, 4) || (wtv && !aligned(acc_all, 4))) return fail(AAL_ERR_ALIGN, "records must be 4-byte aligned");
  float scd, sct;
  aal_status_t st = vp_scales(AAL_VP_EAL, temp_draft, 1.f, &scd, &sct);
  if (st != AAL_OK) return st;
  const hipError_t e = aal::launch_vp_seq_scan(row, wtv ? acc_all : nullptr, wtv ? R : 0, B, S, K,
                                               vp_mode(raw(mode)), 1.0f / temp_draft, grad_scale, loss,
                                               eal_per_window, accept, wtv ? nullptr : target_argmax,
                                               stream);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

aal_status_t aal_vp_grad(const void* z_draft, const void* z_target, aal_dtype_t in_dtype, int64_t rows,
                         int32_t V_slice, int32_t v0, aal_vp_mode_t mode, float temp_draft, float temp_target,
                         const aal_vp_row_t* row, void* grad_draft, aal_dtype_t grad_dtype, hipStream_t stream) {
  clear_error();
  if (!valid_vp_mode(raw(mode))) return fail(AAL_ERR_ARG, "unknown mode %d", raw(mode));
  aal_status_t st =
      validate_vp_slice(z_draft, z_target, raw(mode) == AAL_VP_WTV, raw(in_dtype), rows, V_slice, v0);
  if (st != AAL_OK) return st;
  if (!row || !grad_draft) return fail(AAL_ERR_ARG, "row and grad_draft must be non-NULL");
  if (!valid_dtype(raw(grad_dtype))) return fail(AAL_ERR_DTYPE, "unknown grad_dtype %d", raw(grad_dtype));
  if (!aligned(row, 4)) return fail(AAL_ERR_ALIGN, "records must be 4-byte aligned");
  if (!aligned(grad_draft, 16)) return fail(AAL_ERR_ALIGN, "grad_draft must be 16-byte aligned");
  aal::VpSlice s{};
  if ((st = vp_scales(raw(mode), temp_draft, temp_target, &s.scd, &s.sct)) != AAL_OK) return st;
  s.zd = z_draft;
  s.zt = raw(mode) == AAL_VP_WTV ? z_target : nullptr;
  s.in = to_dtype(raw(in_dtype));
  s.rows = rows;
  s.vs = V_slice;
  s.v0 = v0;
  s.mode = vp_mode(raw(mode));
  s.stream = stream;
  const hipError_t e = aal::launch_vp_grad(s, row, grad_draft, to_dtype(raw(grad_dtype)));
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

aal_status_t aal_stream_probe(const void* src0, const void* src1, const void* src2, void* dst, size_t bytes,
                              uint32_t* flag, hipStream_t stream) {
  clear_error();
  if (!src0) return fail(AAL_ERR_ARG, "src0 must be non-NULL");
  if (src2 && !src1) return fail(AAL_ERR_ARG, "src2 given without src1");
  if (bytes == 0 || bytes % 16 != 0) return fail(AAL_ERR_ARG, "bytes must be a positive multiple of 16");
  if (bytes / 16 >= (size_t(1) << 62)) return fail(AAL_ERR_ARG, "bytes too large");
  if (!dst && !flag) return fail(AAL_ERR_ARG, "flag must be non-NULL when dst is NULL");
  const void* src[3] = {src0, src1, src2};
  for (const void* p : src)
    if (p && !aligned(p, 16)) return fail(AAL_ERR_ALIGN, "sources must be 16-byte aligned");
  if (dst && !aligned(dst, 16)) return fail(AAL_ERR_ALIGN, "dst must be 16-byte aligned");
  if (flag && !aligned(flag, 4)) return fail(AAL_ERR_ALIGN, "flag must be 4-byte aligned");
  const int n_src = src2 ? 3 : src1 ? 2 : 1;
  const hipError_t e = aal::launch_stream_probe(src, n_src, dst, bytes, flag, stream);
  if (e != hipSuccess) return fail(AAL_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return AAL_OK;
}

}  // extern "C"
