// Driver for the sanitizer build of libaal's C-ABI layer: every entry point
// with valid arguments (reaching the host-only launcher stand-ins, which write
// the whole workspace they are given) and with the invalid arguments the
// validation must reject.  Built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host side; needs no GPU.  Exits 0 when
// every check passes; a sanitizer finding aborts the process.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "aal.h"

namespace aal {
extern int g_stub_calls;
}

static int g_failures = 0;

#define CHECK(cond)                                                         \
  do {                                                                      \
    if (!(cond)) {                                                          \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond);   \
      ++g_failures;                                                         \
    }                                                                       \
  } while (0)

// A host buffer of exactly `bytes` bytes (a multiple of 256), 256-aligned.
static void* ws_alloc(size_t bytes) {
  CHECK(bytes % 256 == 0);
  return aligned_alloc(256, bytes);
}

static void* const D = reinterpret_cast<void*>(uintptr_t(0x10000));  // a fake device address
static float* const DF = reinterpret_cast<float*>(uintptr_t(0x20000));
static int32_t* const DI = reinterpret_cast<int32_t*>(uintptr_t(0x30000));

static void expect(aal_status_t st, aal_status_t want, int line) {
  if (st != want) {
    fprintf(stderr, "line %d: status %d, wanted %d (%s)\n", line, int(st), int(want), aal_last_error());
    ++g_failures;
  }
  if (want != AAL_OK && aal_last_error()[0] == '\0') {
    fprintf(stderr, "line %d: no error text\n", line);
    ++g_failures;
  }
}
#define EXPECT(call, want) expect((call), (want), __LINE__)

static void test_status_and_workspace() {
  CHECK(aal_version() >= 100);
  for (int s = 0; s <= 5; ++s) CHECK(strncmp(aal_status_string(aal_status_t(s)), "AAL_", 4) == 0);
  CHECK(strcmp(aal_status_string(aal_status_t(99)), "unknown status") == 0);
  CHECK(aal_workspace_bytes(-1, 2) == 0);
  CHECK(aal_workspace_bytes(14336, 2048) % 256 == 0);
  CHECK(aal_loss_workspace_bytes(AAL_LAYOUT_SEQUENCES, 2, 0, 7) == 0);
  CHECK(aal_loss_workspace_bytes(aal_layout_t(5), 2, 8, 7) == 0);
  CHECK(aal_grpo_workspace_bytes(AAL_LAYOUT_SEQUENCES, 4, 2048, 0, 8, 7) == 0);
}

static void test_eal_wtv() {
  const int64_t N = 3;
  const int32_t K = 4, V = 100;
  const size_t wb = aal_workspace_bytes(N * K, N);
  void* ws = ws_alloc(wb);
  int before = aal::g_stub_calls;
  EXPECT(aal_eal_fwd_bwd(D, D, AAL_BF16, N, K, V, 1.0f, DF, nullptr, DF, DI, D, AAL_BF16, nullptr, ws, wb, nullptr),
         AAL_OK);
  EXPECT(aal_wtv_fwd_bwd(D, D, AAL_F32, N, K, V, 0.7f, 1.3f, DF, DF, DF, D, AAL_F32, DF, ws, wb, nullptr), AAL_OK);
  EXPECT(aal_eal_fwd_bwd_ex(D, D, AAL_F32, N, K, V, 1.0f, DF, DF, nullptr, nullptr, nullptr, AAL_F32, nullptr,
                            AAL_FLAG_STREAMING, ws, wb, nullptr),
         AAL_OK);
  EXPECT(aal_wtv_fwd_bwd_ex(D, D, AAL_BF16, N, K, V, 1.0f, 1.0f, DF, nullptr, nullptr, D, AAL_BF16, nullptr,
                            AAL_FLAG_STREAMING, ws, wb, nullptr),
         AAL_OK);
  EXPECT(aal_wtv_fwd_bwd_ex(D, D, AAL_BF16, N, K, V, 1.0f, 1.0f, DF, nullptr, nullptr, D, AAL_BF16, nullptr,
                            AAL_FLAG_COOPERATIVE, ws, wb, nullptr),
         AAL_OK);
  CHECK(aal::g_stub_calls == before + 5);
  before = aal::g_stub_calls;
  EXPECT(aal_wtv_fwd_bwd_ex(D, D, AAL_BF16, N, K, V, 1.0f, 1.0f, DF, nullptr, nullptr, D, AAL_BF16, nullptr, 4u, ws,
                            wb, nullptr),
         AAL_ERR_ARG);
  CHECK(aal::g_stub_calls == before);
  // invalid arguments: nothing reaches a launcher
  before = aal::g_stub_calls;
  EXPECT(aal_eal_fwd_bwd(nullptr, D, AAL_BF16, N, K, V, 1.0f, DF, nullptr, nullptr, nullptr, nullptr, AAL_BF16,
                         nullptr, ws, wb, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_eal_fwd_bwd(D, D, AAL_BF16, N, 65, V, 1.0f, DF, nullptr, nullptr, nullptr, nullptr, AAL_BF16, nullptr,
                         ws, wb, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_eal_fwd_bwd(D, D, AAL_BF16, N, K, V, 0.0f, DF, nullptr, nullptr, nullptr, nullptr, AAL_BF16, nullptr, ws,
                         wb, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_eal_fwd_bwd(D, D, aal_dtype_t(7), N, K, V, 1.0f, DF, nullptr, nullptr, nullptr, nullptr, AAL_BF16,
                         nullptr, ws, wb, nullptr),
         AAL_ERR_DTYPE);
  EXPECT(aal_eal_fwd_bwd(reinterpret_cast<char*>(D) + 2, D, AAL_BF16, N, K, V, 1.0f, DF, nullptr, nullptr, nullptr,
                         nullptr, AAL_BF16, nullptr, ws, wb, nullptr),
         AAL_ERR_ALIGN);
  EXPECT(aal_eal_fwd_bwd(D, D, AAL_BF16, N, K, V, 1.0f, DF, nullptr, nullptr, nullptr, nullptr, AAL_BF16, nullptr, ws,
                         wb - 256, nullptr),
         AAL_ERR_WORKSPACE);
  EXPECT(aal_wtv_fwd_bwd_ex(D, D, AAL_BF16, N, K, V, 1.0f, 1.0f, DF, nullptr, nullptr, nullptr, AAL_BF16, nullptr, 6u,
                            ws, wb, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_wtv_fwd_bwd(D, D, AAL_BF16, int64_t(1) << 40, K, V, 1.0f, 1.0f, DF, nullptr, nullptr, nullptr, AAL_BF16,
                         nullptr, ws, wb, nullptr),
         AAL_ERR_ARG);
  CHECK(aal::g_stub_calls == before);
  free(ws);
}

static void test_sim() {
  const int32_t P = 2, G = 4, K = 3, V = 10;
  const size_t wb = aal_workspace_bytes(int64_t(P) * G * K, int64_t(P) * G);
  void* ws = ws_alloc(wb);
  EXPECT(aal_sim_accept_grpo(D, D, AAL_BF16, P, G, K, V, 1.0f, DF, DF, nullptr, DI, DF, 1e-6f, 0, 0.0f, ws, wb,
                             nullptr),
         AAL_OK);
  EXPECT(aal_sim_accept_grpo_ex(D, D, AAL_F32, P, G, K, V, 0.5f, DF, DF, nullptr, nullptr, DI, DF, 1e-6f, 1, 2.0f, ws,
                                wb, nullptr),
         AAL_OK);
  EXPECT(aal_sim_accept_grpo(D, D, AAL_BF16, P, 1, K, V, 1.0f, DF, DF, nullptr, DI, DF, 1e-6f, 1, 0.0f, ws, wb,
                             nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_sim_accept_grpo(D, D, AAL_BF16, P, G, K, (1 << 21) + 1, 1.0f, DF, DF, nullptr, DI, DF, 1e-6f, 0, 0.0f,
                             ws, wb, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_sim_accept_grpo(D, D, AAL_BF16, P, G, K, V, 1.0f, DF, DF, nullptr, DI, DF, 1e-6f, 0, 0.0f, ws, 8,
                             nullptr),
         AAL_ERR_WORKSPACE);
  free(ws);
}

static void test_loss() {
  const aal_loss_weights_t w = {0.5f, 0.1f, 1.0f, 0.3f};
  // sequences: B=2, S=9, K=3 (ragged last chunk)
  size_t wb = aal_loss_workspace_bytes(AAL_LAYOUT_SEQUENCES, 2, 9, 3);
  void* ws = ws_alloc(wb);
  EXPECT(aal_loss_fwd_bwd(D, D, nullptr, AAL_BF16, AAL_LAYOUT_SEQUENCES, 2, 9, 3, 50, 1.0f, 1.0f, w, DF, DF, DF, DF,
                          DF, DF, DI, D, AAL_BF16, DF, 0u, ws, wb, nullptr),
         AAL_OK);
  EXPECT(aal_loss_fwd_bwd(D, nullptr, DI, AAL_F32, AAL_LAYOUT_SEQUENCES, 2, 9, 3, 50, 1.0f, 1.0f,
                          aal_loss_weights_t{0.f, 1.f, 0.f, 0.f}, DF, nullptr, nullptr, nullptr, nullptr, nullptr,
                          nullptr, nullptr, AAL_F32, nullptr, AAL_FLAG_STREAMING, ws, wb, nullptr),
         AAL_OK);
  EXPECT(aal_loss_fwd_bwd(D, nullptr, nullptr, AAL_F32, AAL_LAYOUT_SEQUENCES, 2, 9, 3, 50, 1.0f, 1.0f, w, DF, nullptr,
                          nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, AAL_F32, nullptr, 0u, ws, wb, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_loss_fwd_bwd(D, D, nullptr, AAL_F32, AAL_LAYOUT_SEQUENCES, 2, 9, 3, 50, 1.0f, 1.0f, w, DF, nullptr,
                          nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, AAL_F32, nullptr, 0u, ws, wb - 256,
                          nullptr),
         AAL_ERR_WORKSPACE);
  free(ws);
  // sequences shorter than a window, and the windows layout
  wb = aal_loss_workspace_bytes(AAL_LAYOUT_SEQUENCES, 3, 2, 5);
  ws = ws_alloc(wb);
  EXPECT(aal_loss_fwd_bwd(D, D, nullptr, AAL_BF16, AAL_LAYOUT_SEQUENCES, 3, 2, 5, 40, 1.0f, 1.0f, w, DF, DF, nullptr,
                          nullptr, DF, DF, DI, D, AAL_F32, nullptr, 0u, ws, wb, nullptr),
         AAL_OK);
  free(ws);
  wb = aal_loss_workspace_bytes(AAL_LAYOUT_WINDOWS, 5, 0, 7);
  ws = ws_alloc(wb);
  EXPECT(aal_loss_fwd_bwd(D, D, nullptr, AAL_BF16, AAL_LAYOUT_WINDOWS, 5, 0, 7, 128, 0.7f, 0.9f, w, DF, DF, DF, DF,
                          DF, DF, DI, D, AAL_BF16, nullptr, 0u, ws, wb, nullptr),
         AAL_OK);
  free(ws);
}

static void test_grpo() {
  const aal_grpo_params_t prm = {1e-6f, 0.0f, 0.2f, 0.0f, __builtin_huge_valf()};
  size_t wb = aal_grpo_workspace_bytes(AAL_LAYOUT_SEQUENCES, 2, 20, 2, 4, 3);
  void* ws = ws_alloc(wb);
  EXPECT(aal_grpo_fwd_bwd(D, D, D, nullptr, AAL_BF16, AAL_LAYOUT_SEQUENCES, 2, 20, 2, 4, 3, 64, DI, 1.0f, prm, DF,
                          DI, DI, DF, DF, D, AAL_BF16, nullptr, ws, wb, nullptr),
         AAL_OK);
  EXPECT(aal_grpo_fwd_bwd(D, D, nullptr, nullptr, AAL_BF16, AAL_LAYOUT_SEQUENCES, 2, 20, 2, 4, 3, 64, DI, 1.0f, prm,
                          DF, nullptr, nullptr, nullptr, nullptr, nullptr, AAL_BF16, nullptr, ws, wb, nullptr),
         AAL_ERR_ARG);
  free(ws);
  wb = aal_grpo_workspace_bytes(AAL_LAYOUT_WINDOWS, 3, 0, 0, 8, 7);
  ws = ws_alloc(wb);
  EXPECT(aal_grpo_fwd_bwd(D, D, nullptr, DI, AAL_F32, AAL_LAYOUT_WINDOWS, 3, 56, 0, 8, 7, 64, nullptr, 0.8f, prm, DF,
                          DI, DI, DF, DF, D, AAL_F32, DF, ws, wb, nullptr),
         AAL_OK);
  free(ws);
}

static void test_vp() {
  aal_vp_part_t* parts = static_cast<aal_vp_part_t*>(D);
  aal_vp_row_t* row = static_cast<aal_vp_row_t*>(D);
  aal_vp_acc_t* acc = static_cast<aal_vp_acc_t*>(D);
  EXPECT(aal_vp_row_partials(D, D, nullptr, AAL_BF16, 6, 64, 128, 256, AAL_VP_WTV, 1.0f, 1.0f, parts, nullptr),
         AAL_OK);
  EXPECT(aal_vp_row_partials(D, nullptr, DI, AAL_BF16, 6, 64, 128, 256, AAL_VP_EAL, 1.0f, 1.0f, parts, nullptr),
         AAL_OK);
  EXPECT(aal_vp_row_partials(D, D, nullptr, AAL_BF16, 6, 64, 200, 256, AAL_VP_WTV, 1.0f, 1.0f, parts, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_vp_merge_rows(parts, 4, 6, AAL_VP_EAL, 1.0f, 1.0f, row, nullptr), AAL_OK);
  EXPECT(aal_vp_accept_partials(D, D, AAL_BF16, 6, 64, 1.0f, 1.0f, row, acc, nullptr), AAL_OK);
  EXPECT(aal_vp_window_scan(row, acc, 4, 2, 3, AAL_VP_WTV, 1.0f, nullptr, DF, DF, nullptr, nullptr, nullptr), AAL_OK);
  EXPECT(aal_vp_sequence_scan(row, acc, 4, 2, 3, 2, AAL_VP_WTV, 1.0f, nullptr, DF, DF, nullptr, nullptr, nullptr),
         AAL_OK);
  EXPECT(aal_vp_sequence_scan(row, acc, 4, 2, 3, 7, AAL_VP_WTV, 1.0f, nullptr, DF, DF, nullptr, nullptr, nullptr),
         AAL_ERR_ARG);
  EXPECT(aal_vp_grad(D, D, AAL_BF16, 6, 64, 0, AAL_VP_WTV, 1.0f, 1.0f, row, D, AAL_BF16, nullptr), AAL_OK);
}

static void test_stream_probe() {
  uint32_t flag = 0;
  EXPECT(aal_stream_probe(D, D, nullptr, D, 4096, nullptr, nullptr), AAL_OK);
  EXPECT(aal_stream_probe(D, nullptr, nullptr, nullptr, 4096, &flag, nullptr), AAL_OK);
  EXPECT(aal_stream_probe(D, nullptr, nullptr, nullptr, 4096, nullptr, nullptr), AAL_ERR_ARG);  // no dst, no flag
  EXPECT(aal_stream_probe(D, nullptr, D, D, 4096, nullptr, nullptr), AAL_ERR_ARG);              // src2 without src1
  EXPECT(aal_stream_probe(D, D, D, D, 4095, nullptr, nullptr), AAL_ERR_ARG);                    // not 16-byte units
  EXPECT(aal_stream_probe(nullptr, nullptr, nullptr, D, 4096, nullptr, nullptr), AAL_ERR_ARG);
}

static void test_noalloc() {
  // too large for the static scratch: rejected before the device is touched
  EXPECT(aal_wtv_fwd_bwd_noalloc(D, D, AAL_BF16, 1000000, 1, 8, 1.0f, 1.0f, DF, nullptr, nullptr, nullptr, AAL_BF16,
                                 nullptr, nullptr),
         AAL_ERR_WORKSPACE);
  // a valid size: without a GPU the device lookup fails cleanly; with one the
  // stand-in launchers accept it
  const aal_status_t st = aal_wtv_fwd_bwd_noalloc(D, D, AAL_BF16, 4, 7, 64, 1.0f, 1.0f, DF, nullptr, nullptr, nullptr,
                                                  AAL_BF16, nullptr, nullptr);
  CHECK(st == AAL_OK || st == AAL_ERR_HIP);
}

int main() {
  test_status_and_workspace();
  test_eal_wtv();
  test_sim();
  test_loss();
  test_grpo();
  test_vp();
  test_stream_probe();
  test_noalloc();
  if (g_failures) {
    fprintf(stderr, "%d checks failed\n", g_failures);
    return 1;
  }
  printf("abi sanitizer driver: all checks passed (%d launches reached the stand-ins)\n", aal::g_stub_calls);
  return 0;
}
