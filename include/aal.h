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
 *     token drawn and verified by sampling verification (Eq. acc_sample).
 * Temperature scaling is Eq. (1), i.e. softmax(z / T).  Window aggregation is
 * Eq. eal_generic: E[L] = sum_{k=1..K} prod_{j<k} a_j.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every array argument is a DEVICE pointer into memory the caller
 *   allocated and owns (e.g. a torch tensor).  The library never allocates,
 *   frees, or keeps a pointer past the call.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = the default
 *   stream).  Every call only enqueues kernels on it and returns; results are
 *   valid once the stream has been synchronised.  No call synchronises the
 *   host.
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

/* Library version as major*10000 + minor*100 + patch. */
int aal_version(void);

/* Workspace bytes needed by any entry point for `rows` logit rows
 * (N*K, or P*G*K for the simulation) and `windows` windows (N, or P*G).
 * Returns 0 for negative arguments. */
size_t aal_workspace_bytes(int64_t rows, int64_t windows);

/* Static text for a status code ("unknown status" for others). */
const char* aal_status_string(int status);

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
 * flags             : AAL_FLAG_* bits.
 */
aal_status_t aal_eal_fwd_bwd(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                             int64_t N, int32_t K, int32_t V, float temp_draft,
                             float* loss, float* eal_per_window, float* accept,
                             int32_t* target_argmax,
                             void* grad_draft, aal_dtype_t grad_dtype, const float* grad_scale,
                             uint32_t flags, void* workspace, size_t workspace_bytes,
                             void* stream);

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
                             uint32_t flags, void* workspace, size_t workspace_bytes,
                             void* stream);

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
 * draft_token, accept : [P*G*K] int32, or NULL.
 * reward    : [P*G] int32, required.   advantage : [P*G] float, required.
 */
aal_status_t aal_sim_accept_grpo(const void* z_draft, const void* z_target, aal_dtype_t in_dtype,
                                 int32_t P, int32_t G, int32_t K, int32_t V, float temperature,
                                 const float* u1, const float* u2,
                                 int32_t* draft_token, int32_t* accept,
                                 int32_t* reward, float* advantage,
                                 float eps, int32_t std_ddof, float adv_clip,
                                 void* workspace, size_t workspace_bytes, void* stream);

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
 * workspace : at least aal_loss_workspace_bytes(layout, B, S, K) bytes.
 */
aal_status_t aal_loss_fwd_bwd(const void* z_draft, const void* z_target, const int32_t* labels,
                              aal_dtype_t in_dtype, aal_layout_t layout, int64_t B, int32_t S,
                              int32_t K, int32_t V, float temp_draft, float temp_target,
                              aal_loss_weights_t weights, float* loss, float* terms,
                              float* e_tv, float* e_eal, float* accept_tv, float* accept_eal,
                              int32_t* xstar, void* grad_draft, aal_dtype_t grad_dtype,
                              const float* grad_scale, void* workspace, size_t workspace_bytes,
                              void* stream);

#ifdef __cplusplus
}
#endif

#endif /* AAL_H */
