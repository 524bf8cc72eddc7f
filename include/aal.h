/*
 * aal.h -- C ABI of libaal: acceptance-aware draft-training losses on AMD
 * Instinct MI355X (gfx950).
 *
 * The operations follow "Acceptance-Aware Draft Model Training for Speculative
 * Decoding" (arXiv 2609.24150):
 *   - the greedy Expected-Accepted-Length loss (Section "Expected Accepted
 *     Length Loss", Eq. loss_eal) with acceptance q(x*) (Eq. acc_greedy);
 *   - the Window-TV loss (Section "Window TV Loss", Eq. loss_tv) with
 *     acceptance sum_v min(p~, q~) = 1 - TV (Eq. acc_sample, Eq. rejection_rate);
 *   - the simulated accepted-length reward and the group-relative advantage
 *     (Section "GRPO Loss on Acceptance Length", Eq. advantage), with the draft
 *     token drawn and verified by sampling verification (Eq. acc_sample);
 *   - sliding windows over sequences and the weighted objectives of the
 *     experiments (forward-KL anchor, window-mean TV, EAL, WTV) in one call;
 *   - the GRPO loss on the debiased greedy acceptance length with its
 *     policy-ratio surrogate and gradient.
 * Temperature scaling is Eq. (1), i.e. softmax(z / T).  Window aggregation is
 * Eq. eal_generic: E[L] = sum_{k=1..K} prod_{j<k} a_j.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every array argument is a DEVICE pointer into memory the caller
 *   allocated and owns (e.g. a torch tensor).  The library never allocates,
 *   frees, or keeps a pointer past the call.
 * Streams.  `stream` is a hipStream_t (NULL = the default stream).  Every
 *   call only enqueues kernels on it and returns; results are valid once the stream has been synchronised.  No call synchronises the
 *   host.  Nothing else is enqueued (no memset or copy nodes), so with the
 *   default flags a call can be captured into a HIP graph and replayed.
 * Layout.  Logits are contiguous row-major [N, K, V] (simulation: [P, G, K, V]);
 *   row r = n*K + k holds position k of window n; the row stride is V elements.
 *   Element offsets are 64-bit.
 * Alignment.  Logit and gradient pointers must be 16-byte aligned, the
 *   workspace 256-byte aligned; otherwise AAL_ERR_ALIGN.
 * Inputs.  Logits must be finite or -inf (a vocabulary mask); every row needs
 *   at least one finite entry.  NaN inputs give unspecified results.
 * Errors.  Arguments are validated before anything is enqueued; on a
 *   validation error nothing is written.  A failed kernel launch returns
 *   AAL_ERR_HIP.  aal_last_error() gives a per-thread description of the last
 *   error.  Nothing throws across this ABI.
 * Workspace.  Device scratch of at least aal_workspace_bytes(rows, windows)
 *   bytes; its contents on entry are ignored and on exit unspecified.
 *   Concurrent calls must use distinct workspaces.
 * Concurrency.  The register-resident schedule of the loss calls launches a
 *   persistent grid no larger than the device holds at once, whose
 *   workgroups wait for each other's partial results.  Other work on the
 *   device can delay the placement of some of its workgroups, never prevent
 *   it; but two resident launches that run at the same time (several streams
 *   or processes on one device) could each hold part of the device while
 *   waiting for the rest.  Calls on one stream never overlap.  Callers that
 *   issue loss calls on several streams of one device at once pass
 *   AAL_FLAG_COOPERATIVE, which leaves the placement of the whole grid to the
 *   HIP runtime's cooperative launch.  Every wait is bounded: a wait that
 *   times out (seconds) ends the kernel and the loss reads NaN.  With the
 *   environment variable AAL_TEST_PRESET_TIMEOUT=1 the resident kernels start
 *   in that state (a test hook for the time-out path).
 * Determinism.  No floating-point atomics: results are bitwise reproducible
 *   for a given device, shape and flags.
 */
#ifndef AAL_H
#define AAL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* HIP's stream handle, declared exactly as the HIP runtime declares it, so
 * that this header stands alone (C11 / C++: repeating the typedef after
 * <hip/hip_runtime.h> is allowed).  NULL is the default stream. */
typedef struct ihipStream_t* hipStream_t;

/* Element types of logits and gradients. */
typedef enum { AAL_BF16 = 0, AAL_F32 = 1 } aal_dtype_t;

/* Status codes. */
typedef enum {
  AAL_OK = 0,
  AAL_ERR_ARG = 1,       /* a size, temperature or required pointer is invalid     */
  AAL_ERR_DTYPE = 2,     /* unsupported element type or type combination           */
  AAL_ERR_ALIGN = 3,     /* a pointer breaks the alignment rule above               */
  AAL_ERR_WORKSPACE = 4, /* workspace NULL or smaller than aal_workspace_bytes()    */
  AAL_ERR_HIP = 5        /* a HIP runtime call or kernel launch failed              */
} aal_status_t;

/* Flags for the loss entry points (bitwise OR; 0 = automatic choice). */
#define AAL_FLAG_STREAMING 1u /* force the multi-kernel streaming schedule            */
/* Launch the register-resident kernel through the HIP runtime's cooperative
 * launch, which places the whole grid before the kernel starts (see
 * "Concurrency" above; it adds about 20 us per call). */
#define AAL_FLAG_COOPERATIVE 2u

/* Library version as major*10000 + minor*100 + patch. */
int aal_version(void);

/* Workspace bytes needed by any entry point for `rows` logit rows
 * (N*K, or P*G*K for the simulation) and `windows` windows (N, or P*G).
 * Returns 0 for negative arguments. */
size_t aal_workspace_bytes(int64_t rows, int64_t windows);

/* Static text for a status code ("unknown status" for others). */
const char* aal_status_string(aal_status_t status);

/* Text describing the last error raised on the calling thread ("" if none).
 * The pointer stays valid until the thread's next library call. */
const char* aal_last_error(void);

/*
 * Greedy EAL loss, forward and backward (Eq. loss_eal, Eq. acc_greedy).
 *
 *   x*_{n,k}  = argmax_v z_target[n,k,v]        (lowest index on ties)
 *   q_{n,k}   = softmax(z_draft[n,k,:] / temp_draft)
 *   a_{n,k}   = q_{n,k}(x*_{n,k})
 *   E_n       = sum_{k=1..K} prod_{j<k} a_{n,j}
 *   loss      = -(1/N) sum_n E_n
 *   grad_draft[n,k,v] = scale * dloss/dz_draft[n,k,v]
 *                     = scale * g_{n,k} * (a_{n,k}/temp_draft) * (1[v = x*] - q_{n,k}(v)),
 *     with g_{n,k} = dloss/da_{n,k} = -(1/N) dE_n/da_{n,k}.
 *
 * z_draft, z_target : [N,K,V] of in_dtype (both the same type).
 * N >= 1, 1 <= K <= 64, V >= 1, N*K*V < 2^62; temp_draft finite and > 0.
 * loss              : [1] float, required.
 * eal_per_window    : [N] float E_n, or NULL.
 * accept            : [N*K] float a_{n,k}, or NULL.
 * target_argmax     : [N*K] int32 x*, or NULL.
 * grad_draft        : [N,K,V] of grad_dtype, or NULL for a forward-only call.
 *                     grad_dtype may be AAL_F32 for either input type, or
 *                     AAL_BF16 (rounded to nearest even).
 * grad_scale        : device float scalar multiplying the gradient (an
 *                     upstream dL/dloss), or NULL for 1.0.  Not applied to loss.
 * workspace         : at least aal_workspace_bytes(N*K, N) bytes, 256-byte aligned.
 * The default schedule is one register-resident kernel when V is a multiple
 * of 8 (bf16) / 4 (fp32) elements, K is in {1..8, 16} and a window fits the
 * co-resident grid; every other shape takes the multi-kernel streaming
 * schedule.  A poll time-out of the resident schedule (not expected) sets
 * the loss to NaN.
 */
aal_status_t aal_eal_fwd_bwd(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                             int64_t N, int32_t K, int32_t V, float temp_draft,
                             float* loss, float* eal_per_window, float* accept,
                             int32_t* target_argmax,
                             void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/* aal_eal_fwd_bwd with schedule flags: flags = 0 is aal_eal_fwd_bwd;
 * AAL_FLAG_STREAMING forces the multi-kernel schedule (the same results
 * within the stated tolerances; used to cross-check the two schedules);
 * AAL_FLAG_COOPERATIVE launches the resident kernel through the runtime's
 * cooperative launch (the same bits; see "Concurrency").  Unknown bits give
 * AAL_ERR_ARG. */
aal_status_t aal_eal_fwd_bwd_ex(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                int64_t N, int32_t K, int32_t V, float temp_draft,
                                float* loss, float* eal_per_window, float* accept,
                                int32_t* target_argmax,
                                void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                                uint32_t flags, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * Window-TV loss, forward and backward (Eq. loss_tv, Eq. acc_sample).
 *
 *   q = softmax(z_draft / temp_draft),  p = softmax(z_target / temp_target)
 *   a_{n,k} = sum_v min(p(v), q(v)) = 1 - TV(p, q)
 *   E_n, loss as for EAL.
 *   grad_draft[n,k,v] = scale * g_{n,k} * (1/temp_draft) * q(v) * (m(v) - sum_u m(u) q(u)),
 *     m(v) = 1[q(v) < p(v)]  (the subgradient of min taken as 0 at q = p).
 * The target is frozen: no gradient is produced for it.
 *
 * Arguments as for aal_eal_fwd_bwd; both temperatures finite and > 0.
 * accept receives sum_v min(p, q).
 */
aal_status_t aal_wtv_fwd_bwd(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                             int64_t N, int32_t K, int32_t V,
                             float temp_draft, float temp_target,
                             float* loss, float* eal_per_window, float* accept,
                             void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/* aal_wtv_fwd_bwd with schedule flags, as aal_eal_fwd_bwd_ex. */
aal_status_t aal_wtv_fwd_bwd_ex(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                int64_t N, int32_t K, int32_t V,
                                float temp_draft, float temp_target,
                                float* loss, float* eal_per_window, float* accept,
                                void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                                uint32_t flags, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Bytes of the static device scratch that aal_wtv_fwd_bwd_noalloc uses on
 * each GPU (32 MiB): it serves any N, K with aal_workspace_bytes(N*K, N) at
 * most this size, i.e. N*K*32 + N*4 bytes plus 4 MiB, rounded up to 256-byte
 * pieces (at least 815,000 logit rows at any K). */
#define AAL_NOALLOC_SCRATCH_BYTES (32u << 20)

/*
 * aal_wtv_fwd_bwd for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, kernels and results as aal_wtv_fwd_bwd, with the
 * workspace taken from a static device array of AAL_NOALLOC_SCRATCH_BYTES
 * inside the library instead of an argument.  It calls no hipMalloc, hipFree
 * or allocating library routine.  The array's address on a device is looked
 * up on the first call on that device (hipGetSymbolAddress), so that first
 * call must not be made while a graph is being captured.
 *
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents (each call clears what must start at zero itself): calls that
 * overlap on one GPU -- on different streams, or from different host threads
 * without ordering -- race and give undefined results.  Calls on different
 * GPUs do not share memory.
 *
 * Arguments, outputs and validation as for aal_wtv_fwd_bwd, minus the
 * workspace; a size whose workspace would exceed AAL_NOALLOC_SCRATCH_BYTES
 * gives AAL_ERR_WORKSPACE before anything is enqueued.
 */
aal_status_t aal_wtv_fwd_bwd_noalloc(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                     int64_t N, int32_t K, int32_t V,
                                     float temp_draft, float temp_target,
                                     float* loss, float* eal_per_window, float* accept,
                                     void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                                     hipStream_t stream);

/*
 * Simulated acceptance length and group-relative advantage (Section "GRPO
 * Loss on Acceptance Length": the accepted-length count and Eq. advantage;
 * verification by sampling as in Eq. acc_sample).
 *
 * For every prefix p < P, rollout g < G and position k < K:
 *   q = softmax(z_draft[p,g,k,:] / temperature), pt = softmax(z_target[...] / temperature)
 *   token  x = smallest v with sum_{w<=v} q(w) > u1[p,g,k]
 *              (the last v with q(v) > 0 if rounding leaves none)
 *   accept = u2[p,g,k] * q(x) < pt(x)       (u2 < min(1, pt(x)/q(x)))
 * reward[p,g]    = number of accepted positions before the first rejection (0..K)
 * advantage[p,g] = clip((r - mean_g r) / (std_g r + eps), -adv_clip, adv_clip),
 *   std with `std_ddof` (0: population, 1: sample); adv_clip <= 0 disables the clip.
 *
 * z_draft, z_target : [P,G,K,V] of in_dtype.  u1, u2 : [P*G*K] float in [0,1).
 * P, G, K, V >= 1; G > std_ddof; V <= 2^21; temperature finite and > 0; eps >= 0.
 * draft_token : [P*G*K] int32, or NULL.
 * reward    : [P*G] int32, required.   advantage : [P*G] float, required.
 * workspace : at least aal_workspace_bytes(P*G*K, P*G) bytes, 256-byte aligned.
 */
aal_status_t aal_sim_accept_grpo(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                 int32_t P, int32_t G, int32_t K, int32_t V, float temperature,
                                 const float* u1, const float* u2,
                                 int32_t* draft_token, int32_t* reward, float* advantage,
                                 float eps, int32_t std_ddof, float adv_clip,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* aal_sim_accept_grpo that also returns the per-position verification
 * outcome: accept [P*G*K] int32 (1 = the drafted token passes, 0 = it is
 * rejected; positions after the first rejection are evaluated too), or NULL. */
aal_status_t aal_sim_accept_grpo_ex(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                    int32_t P, int32_t G, int32_t K, int32_t V, float temperature,
                                    const float* u1, const float* u2,
                                    int32_t* draft_token, int32_t* accept,
                                    int32_t* reward, float* advantage,
                                    float eps, int32_t std_ddof, float adv_clip,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Row layouts of the combined-objective entry point. */
typedef enum {
  AAL_LAYOUT_WINDOWS = 0,  /* [B,K,V]: B disjoint windows of K positions                */
  AAL_LAYOUT_SEQUENCES = 1 /* [B,S,V]: B sequences of S positions; a window of K positions
                              starts at every t = 0..S-K (windows slide by one)          */
} aal_layout_t;

/* Weights of the terms of the combined objective (any may be 0). */
typedef struct {
  float wtv; /* L_WTV: -(1/W) sum_windows E[L], a = 1 - TV                                */
  float eal; /* L_EAL: -(1/W) sum_windows E[L], a = q(x*)                                 */
  float kl;  /* L_KL : (1/R) sum_positions KL(p || q), the forward-KL anchor              */
  float tv;  /* L_TV : (1/W) sum_windows (1/K) sum_{j<K} TV(p, q), the window-mean TV     */
} aal_loss_weights_t;

/* Workspace bytes of aal_loss_fwd_bwd for the given layout and sizes (0 for
 * invalid arguments). */
size_t aal_loss_workspace_bytes(aal_layout_t layout, int64_t B, int32_t S, int32_t K);

/*
 * Combined training objective, forward and backward: the paper's sliding
 * windows over sequences (Section "Window TV Loss", Figure wtv: one draft and
 * one target pass give a_t for every position, each window reads
 * a_t..a_{t+K-1}) and the objectives of its experiments (Section "Settings":
 * the forward-KL anchor alone or plus 0.1 L_EAL, plus the window-mean TV, and
 * L_WTV alone).
 *
 *   q = softmax(z_draft / temp_draft), p = softmax(z_target / temp_target), per row
 *   a_tv = sum_v min(p, q);   a_eal = q(x*), x* = labels[r] if labels, else
 *                             argmax_v z_target (lowest index on ties)
 *   KL_r = sum_v p (log p - log q)
 *   loss = wtv L_WTV + eal L_EAL + kl L_KL + tv L_TV   (see aal_loss_weights_t)
 *   E over a window of rows r_0..r_{K-1}: sum_{k=1..K} prod_{j<k} a_{r_j}
 *   grad_draft = scale * dloss/dz_draft, with
 *     d a_tv/dz = q (m - sum_u m(u) q(u)) / temp_draft, m = 1[q < p],
 *     d a_eal/dz = a_eal (1[v = x*] - q) / temp_draft,
 *     d KL/dz = (q - p) / temp_draft;
 *   a row's dloss/da sums over every window that contains it.
 *
 * Rows: R = B*K (windows layout; S is ignored) or B*S (sequences layout),
 * row-major [R, V]; windows: W = B or B*max(0, S-K+1).  With W = 0 the window
 * terms are 0.
 * z_draft : [R,V] of in_dtype, required.
 * z_target: [R,V] of in_dtype; may be NULL only when wtv = kl = tv = 0 and
 *           labels are given (the EAL term then needs no target).
 * labels  : [R] int32 token ids in [0, V), or NULL; out-of-range ids are
 *           clamped into [0, V).
 * B >= 1, 1 <= K <= 64, V >= 1, S >= 1 (sequences), R*V < 2^62; temperatures
 * finite and > 0; weights finite.
 * loss    : [1] float, required.   terms: [4] float (L_WTV, L_EAL, L_KL, L_TV) or NULL;
 *           a term whose weight is 0 is not evaluated and reads 0.
 * e_tv, e_eal : [W] float window expectations, or NULL.
 * accept_tv, accept_eal : [R] float a_tv / a_eal, or NULL.   xstar: [R] int32, or NULL.
 *           a_tv and e_tv are evaluated when wtv, kl or tv is non-zero; a_eal,
 *           e_eal and x* when eal is non-zero; otherwise they read 0 (x*: -1).
 * grad_draft, grad_dtype, grad_scale : as for aal_eal_fwd_bwd.
 * flags   : AAL_FLAG_* bits.  By default one register-resident kernel reads each
 *           logit once and writes the gradient once when V is a multiple of 8
 *           (bf16) / 4 (fp32), K is in {1..8, 16} and z_target is given; other
 *           shapes, and AAL_FLAG_STREAMING, take the multi-kernel schedule.
 *           AAL_FLAG_COOPERATIVE: see "Concurrency".  A poll time-out of the
 *           resident schedule (not expected) sets the loss to NaN.
 * workspace : at least aal_loss_workspace_bytes(layout, B, S, K) bytes.
 */
aal_status_t aal_loss_fwd_bwd(const void* z_draft, const void* z_target, const int32_t* labels,
                              aal_dtype_t in_dtype, aal_layout_t layout, int64_t B, int32_t S,
                              int32_t K, int32_t V, float temp_draft, float temp_target,
                              aal_loss_weights_t weights, float* loss, float* terms,
                              float* e_tv, float* e_eal, float* accept_tv, float* accept_eal,
                              int32_t* xstar, void* grad_draft, aal_dtype_t grad_dtype,
                              const float* grad_scale, uint32_t flags, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Constants of the GRPO loss that the paper leaves unstated (its Eq. advantage
 * uses eps = 1e-6). */
typedef struct {
  float eps;      /* advantage denominator: (R - mean) / (std + eps), eps >= 0        */
  float adv_clip; /* C_A: advantages clipped to [-C_A, C_A]; <= 0 disables the clip   */
  float eps_clip; /* PPO clip of the ratio: [1 - eps_clip, 1 + eps_clip], >= 0        */
  float rho_min;  /* ratio clip before the surrogate: [rho_min, rho_max],             */
  float rho_max;  /*   0 <= rho_min <= rho_max (rho_max may be +inf)                   */
} aal_grpo_params_t;

/* Workspace bytes of aal_grpo_fwd_bwd (0 for invalid arguments). */
size_t aal_grpo_workspace_bytes(aal_layout_t layout, int64_t B, int32_t S, int32_t G, int32_t m, int32_t K);

/*
 * GRPO loss on the debiased greedy acceptance length, forward and backward
 * w.r.t. the current draft's logits (Section "GRPO Loss on Acceptance
 * Length": greedy trajectories S^theta, S^ref; simulated greedy
 * verification; Eq. debiased_reward; the per-token geometric-mean policy
 * ratio clipped to [-10, 10]; Eq. advantage; the PPO-clipped group loss and
 * its mean over groups).
 *
 * Per window of K positions (rows r_0..r_{K-1}) of a group of m windows:
 *   S^pi_k   = argmax_v z_pi[r_k, v]  (pi = theta, ref; lowest index on ties)
 *   tau^pi   = number of leading k with S^pi_k = x*_k, x* = labels or argmax z_target
 *   R        = tau^theta - tau^ref                       (no gradient)
 *   log rho  = clip((1/K) sum_k [log pi_theta(S^theta_k) - log pi_ref(S^theta_k)], -10, 10),
 *              pi = softmax(z / temperature)
 *   rho      = clip(exp(log rho), rho_min, rho_max)
 *   A        = clip((R - mean_g R) / (std_g R + eps), -adv_clip, adv_clip)  (population
 *              std over the group's m windows; no gradient)
 *   L_g      = -(1/m) sum_windows min(rho A, clip(rho, 1 - eps_clip, 1 + eps_clip) A)
 *   loss     = mean over groups of L_g
 *   grad_theta[r, v] = scale * sum over windows w containing r of
 *              (dloss/dlog rho_w) (1/K) (1/temperature) (1[v = S^theta_r] - pi_theta,r(v)),
 *   where a clip passes derivative 1 strictly inside its interval and 0 elsewhere,
 *   and min(u, v) takes u's derivative when u <= v.
 *
 * Layouts: AAL_LAYOUT_WINDOWS: logits [B*m*K, V]: B groups of m windows of K
 *   rows each (S, G, anchors ignored).  AAL_LAYOUT_SEQUENCES: logits [B*S, V]:
 *   B sequences of S positions and anchors [B*G] int32; group (b, g) holds
 *   the m windows starting at anchors[b*G+g] + i, i < m (anchors are clamped
 *   into [0, S - m - K + 1]).  Rows in no window get a zero gradient.
 * z_theta, z_ref : [rows, V] of in_dtype, required.  z_target : [rows, V] or
 *   NULL when labels [rows] int32 are given (clamped into [0, V)).
 * B >= 1, 1 <= K <= 64, 1 <= m <= 64, V >= 1; sequences: G >= 1 and S >= m + K - 1;
 * temperature finite and > 0; params as documented at aal_grpo_params_t.
 * loss : [1] float, required.  tau_theta, tau_ref : [groups*m] int32, or NULL.
 * advantage, log_rho : [groups*m] float (the clipped log rho), or NULL.
 * grad_theta, grad_dtype, grad_scale : as for aal_eal_fwd_bwd.
 */
aal_status_t aal_grpo_fwd_bwd(const void* z_theta, const void* z_ref, const void* z_target,
                              const int32_t* labels, aal_dtype_t in_dtype, aal_layout_t layout,
                              int64_t B, int32_t S, int32_t G, int32_t m, int32_t K, int32_t V,
                              const int32_t* anchors, float temperature, aal_grpo_params_t params,
                              float* loss, int32_t* tau_theta, int32_t* tau_ref, float* advantage,
                              float* log_rho, void* grad_theta, aal_dtype_t grad_dtype,
                              const float* grad_scale, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/*
 * Vocabulary-parallel pieces of aal_eal_fwd_bwd and aal_wtv_fwd_bwd: the work
 * of one rank of a tensor-parallel LM head that splits the vocabulary into
 * contiguous slices.  The losses and gradients are those of the two calls
 * above (Eq. acc_greedy, Eq. acc_sample, Eq. eal_generic, Eq. loss_eal,
 * Eq. loss_tv); a row's softmax, greedy token and sum_v min(p, q) span all
 * slices, so they are assembled from per-slice partial records that the
 * caller gathers over the ranks (an all-gather of a few bytes per row) and
 * every rank merges in the same rank order.  With R ranks, rank r holding
 * vocabulary entries [v0_r, v0_r + Vs_r) of every row as its own contiguous
 * [rows, Vs_r] arrays (rows = N*K, row stride Vs_r):
 *
 *   1. aal_vp_row_partials(slice)            -> part_r[rows]
 *      gather part_r over r                  -> part_all[R][rows]   (caller)
 *   2. aal_vp_merge_rows(part_all)           -> row[rows]           (same on every rank)
 *   3. WTV only: aal_vp_accept_partials(slice, row) -> acc_r[rows]
 *      gather acc_r over r                   -> acc_all[R][rows]    (caller)
 *   4. aal_vp_window_scan(row, acc_all)      -> loss, E_n, a, x*, row[].coef
 *   5. aal_vp_grad(slice, row)               -> grad_draft slice [rows, Vs_r]
 *
 * Records are plain structs so that a collective can move them as bytes.
 * Every value is a function of the inputs and R's slicing alone: each rank
 * obtains bit-identical row records, and the results do not depend on which
 * rank runs steps 2 and 4.  Conventions (device pointers, streams, 16-byte
 * alignment of logit and gradient pointers, errors) are those stated at the
 * top of this file; these calls take no workspace.  Temperatures must be the
 * same in every call of one pass.
 */
typedef enum { AAL_VP_EAL = 0, AAL_VP_WTV = 1 } aal_vp_mode_t;

/* Partial statistics of one row over one vocabulary slice.  32 bytes.
 *   zmax_d, zmax_t : largest raw draft / target logit in the slice (-inf if none)
 *   s_d, s_t       : sum over the slice of 2^(z*sc - fl(zmax*sc)), sc = log2(e)/T
 *                    (s_t is 0 in EAL mode)
 *   zd_at          : EAL: the draft logit at t_idx (0 if t_idx is INT32_MAX)
 *   t_idx          : EAL: global index of the slice's largest target logit,
 *                    lowest index on ties, INT32_MAX if the slice has no finite
 *                    target logit (with labels: the row's label if the slice
 *                    holds it, else INT32_MAX); WTV: -1 */
typedef struct {
  float zmax_d, s_d, zmax_t, s_t, zd_at;
  int32_t t_idx, reserved0, reserved1;
} aal_vp_part_t;

/* Partial sums of one row over one slice (WTV): sum_v min(p, q) and
 * Q< = sum over entries with q < p of q, with the merged normalisers. */
typedef struct {
  float smin, qlt;
} aal_vp_acc_t;

/* Merged record of one row.  32 bytes.
 *   msc_d, msc_t : fl(zmax * sc) of the whole row, the reference of l2s_*
 *   l2s_d, l2s_t : log2 of sum_v 2^(z*sc - msc), so log2 q(v) = z*sc - msc_d - l2s_d
 *                  (msc_t, l2s_t are 0 in EAL mode)
 *   a            : acceptance (EAL: q(x*), set by step 2; WTV: sum min(p, q), step 4)
 *   qlt          : WTV: Q< (step 4); EAL: 0
 *   coef         : gradient coefficient of the row (step 4)
 *   xstar        : EAL: greedy target token (0 for a row with no finite target
 *                  logit); WTV: -1 */
typedef struct {
  float msc_d, l2s_d, msc_t, l2s_t, a, qlt, coef;
  int32_t xstar;
} aal_vp_row_t;

/*
 * Step 1.  z_draft, z_target : [rows, V_slice] of in_dtype, the slice that
 * starts at global vocabulary index v0 of a vocabulary of V_total entries.
 * rows >= 1, V_slice >= 1, v0 >= 0, v0 + V_slice <= V_total < 2^31,
 * rows*V_slice < 2^62.  EAL ignores temp_target.
 * labels : EAL only, [rows] int32 global token ids that replace the target's
 *          greedy token, or NULL.  As in aal_loss_fwd_bwd, an id outside
 *          [0, V_total) is clamped into it.  With labels the target logits
 *          are not read and z_target may be NULL; the slice that holds a
 *          row's (clamped) label supplies its candidate.
 * parts : [rows] records, required.
 */
aal_status_t aal_vp_row_partials(const void* z_draft, const void* z_target, const int32_t* labels,
                                 aal_dtype_t in_dtype, int64_t rows, int32_t V_slice, int32_t v0,
                                 int32_t V_total, aal_vp_mode_t mode, float temp_draft,
                                 float temp_target, aal_vp_part_t* parts, hipStream_t stream);

/*
 * Step 2.  parts_all : [R, rows] records, rank-major (rank r's records at
 * parts_all + r*rows), R >= 1.  Merged in rank order 0..R-1: the maxima, the
 * sums rescaled to them, the greedy token by (largest logit, lowest index).
 * Every row needs a finite draft logit (and in WTV a finite target logit) in
 * some slice.  row : [rows] records, required; EAL sets a and xstar.
 */
aal_status_t aal_vp_merge_rows(const aal_vp_part_t* parts_all, int32_t R, int64_t rows,
                               aal_vp_mode_t mode, float temp_draft, float temp_target,
                               aal_vp_row_t* row, hipStream_t stream);

/*
 * Step 3 (WTV).  The slice as in step 1, row from step 2.  acc : [rows], required.
 */
aal_status_t aal_vp_accept_partials(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                    int64_t rows, int32_t V_slice, float temp_draft, float temp_target,
                                    const aal_vp_row_t* row, aal_vp_acc_t* acc, hipStream_t stream);

/*
 * Step 4.  row : [N*K] records from step 2, updated in place (WTV: a and qlt
 * summed from acc_all in rank order; both modes: coef).  acc_all : [R, N*K],
 * rank-major, required for WTV and ignored (may be NULL) for EAL.
 * N >= 1, 1 <= K <= 64, N*K < 2^31.  loss [1] and eal_per_window [N] are
 * required; accept [N*K] and target_argmax [N*K] (EAL) may be NULL.  grad_scale
 * as for aal_eal_fwd_bwd.
 */
aal_status_t aal_vp_window_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R,
                                int64_t N, int32_t K, aal_vp_mode_t mode, float temp_draft,
                                const float* grad_scale, float* loss, float* eal_per_window,
                                float* accept, int32_t* target_argmax, hipStream_t stream);

/*
 * Step 4 for sequences (the layout of aal_loss_fwd_bwd with
 * AAL_LAYOUT_SEQUENCES): the N*K rows are B sequences of S positions, and a
 * window of K positions starts at every position t <= S - K of a sequence
 * (windows sliding by one, Section "Window TV Loss"); W = B (S - K + 1).
 *   loss = -(1/W) sum_windows E_w, and each row's coefficient sums dE_w/da
 *   over the (at most K) windows that contain it.
 * row : [B*S] records from step 2, updated in place as in aal_vp_window_scan.
 * acc_all : [R, B*S] (WTV), as there.  B >= 1, 1 <= K <= 64, K <= S,
 * B*S < 2^31.  loss [1] and eal_per_window [W] (window t of sequence b at
 * b (S - K + 1) + t) are required; accept [B*S] and target_argmax [B*S] (EAL)
 * may be NULL.
 */
aal_status_t aal_vp_sequence_scan(aal_vp_row_t* row, const aal_vp_acc_t* acc_all, int32_t R,
                                  int64_t B, int32_t S, int32_t K, aal_vp_mode_t mode,
                                  float temp_draft, const float* grad_scale, float* loss,
                                  float* eal_per_window, float* accept, int32_t* target_argmax,
                                  hipStream_t stream);

/*
 * Step 5.  The slice as in step 1 (EAL reads only z_draft; z_target may then be
 * NULL), row from step 4.  grad_draft : [rows, V_slice] of grad_dtype, the
 * slice of the gradient of the loss, times *grad_scale as folded into coef.
 */
aal_status_t aal_vp_grad(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                         int64_t rows, int32_t V_slice, int32_t v0, aal_vp_mode_t mode,
                         float temp_draft, float temp_target, const aal_vp_row_t* row,
                         void* grad_draft, aal_dtype_t grad_dtype, hipStream_t stream);

/*
 * Measurement aid, not part of the method: streams 1 to 3 device buffers of
 * `bytes` bytes each (src0, then src1 and src2 when non-NULL) with 16-byte
 * nontemporal loads -- the access the loss kernels use -- and, when dst is not
 * NULL, writes their element-wise 32-bit wrapping sum to dst (`bytes` bytes),
 * so that a timed call gives this device's practical HBM rate for a mix of
 * reads and zero or one write.  Without dst, *flag ([1] uint32) is set to 1
 * only where a summed 64-bit word is all ones, a data-dependent store that
 * keeps every load live; fill the sources so that it does not happen.
 * bytes : a positive multiple of 16.  Pointers 16-byte aligned (flag 4-byte);
 * dst may alias none of the sources.  Four 256-thread workgroups per CU.
 */
aal_status_t aal_stream_probe(const void* src0, const void* src1, const void* src2, void* dst, size_t bytes,
                              uint32_t* flag, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* AAL_H */
