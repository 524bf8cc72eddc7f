"""fp64 CPU oracle for the acceptance-aware draft-training losses.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` use it.  It shares no code with the HIP library.

Every function is a plain, slow, literal transcription of a definition in
"Acceptance-Aware Draft Model Training for Speculative Decoding"
(arXiv 2609.24150), computed in float64 on the exact input values (bf16 and
fp32 inputs are exactly representable in float64).  Array layout follows the
library's: logits are ``[N, K, V]`` (N windows, K = the speculative window size
gamma, V = vocabulary), row ``n*K + k`` is position ``k`` of window ``n``.

Readings of places where the paper is silent:

* temperature: Eq. (1) scales log-probabilities; ``tempered_log_softmax``
  applies it literally to ``log softmax(z)``;
* greedy token ``x*``: argmax of the raw target logits, lowest index on ties;
* ``d min(p, q) / d q`` is taken as ``1[q < p]`` (0 at ties);
* the loss is normalised by the number of windows (the window-start set W);
* the simulated-acceptance draft token is the inverse-CDF sample of q with a
  uniform ``u1`` (smallest v whose cumulative mass exceeds u1), accepted iff
  ``u2 * q(x) < p(x)``; the group standard deviation uses ``ddof`` (default 0);
* sliding windows count only when all K positions lie in the sequence; the
  forward-KL anchor is normalised per position, the window-mean TV per window;
* GRPO: the log ratio uses one temperature for both drafts; the constants the
  paper leaves open (eps_clip, rho_min, rho_max, the advantage clip) are
  arguments; a clip passes the derivative strictly inside its interval only,
  and min(u, v) takes u's derivative when u <= v.

Pinning: every function here is checked by ``tests/test_oracle_pins.py``
against hand-computed cases, closed forms, identities the paper states,
finite differences and brute-force enumeration.  No function is "parity
unpinned".
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "tempered_log_softmax",
    "greedy_token",
    "acceptance_greedy",
    "acceptance_sampling",
    "total_variation",
    "prob_accepted_at_least",
    "length_distribution",
    "expected_length_full",
    "expected_length",
    "expected_length_grad",
    "eal_loss",
    "wtv_loss",
    "inverse_cdf_token",
    "simulate_acceptance",
    "group_advantage",
    "sim_accept_grpo",
    "sim_near_threshold",
    "LAYOUT_WINDOWS",
    "LAYOUT_SEQUENCES",
    "window_rows",
    "forward_kl",
    "window_length_coefficients",
    "combined_loss",
    "greedy_accepted_length",
    "grpo_windows",
    "grpo_loss",
]


# ---------------------------------------------------------------------------
# Temperature scaling (Section "Preliminaries and Notation", Eq. 1)
# ---------------------------------------------------------------------------
def _log_softmax(x: np.ndarray) -> np.ndarray:
    """Log of a normalised exponential over the last axis, max-shifted."""
    m = np.max(x, axis=-1, keepdims=True)
    return x - (m + np.log(np.sum(np.exp(x - m), axis=-1, keepdims=True)))


def tempered_log_softmax(z, T: float) -> np.ndarray:
    """log p~ for logits z at temperature T > 0 (Eq. 1).

    The paper defines p~(v) proportional to exp(log p(v) / T) with p the
    untempered next-token distribution.  We first form log p = log softmax(z)
    and then renormalise exp(log p / T), exactly in that order.
    """
    if not T > 0:
        raise ValueError("temperature must be > 0")
    logp = _log_softmax(np.asarray(z, dtype=np.float64))
    return _log_softmax(logp / np.float64(T))


# ---------------------------------------------------------------------------
# Per-position acceptance (Eqs. acc_greedy and acc_sample)
# ---------------------------------------------------------------------------
def greedy_token(z_target) -> np.ndarray:
    """x* = argmax_v p(v) = argmax_v z_t(v); lowest index on ties (Eq. acc_greedy)."""
    return np.argmax(np.asarray(z_target, dtype=np.float64), axis=-1)


def acceptance_greedy(z_draft, z_target, T_draft: float = 1.0):
    """a = q(x*), the draft mass on the target's greedy token (Eq. acc_greedy).

    Returns (a, x*, q).
    """
    q = np.exp(tempered_log_softmax(z_draft, T_draft))
    xs = greedy_token(z_target)
    a = np.take_along_axis(q, xs[..., None], axis=-1)[..., 0]
    return a, xs, q


def acceptance_sampling(z_draft, z_target, T_draft: float, T_target: float):
    """a = sum_v min(p~(v), q~(v)) = 1 - TV (Eq. acc_sample, Eq. rejection_rate).

    Returns (a, q, p).
    """
    q = np.exp(tempered_log_softmax(z_draft, T_draft))
    p = np.exp(tempered_log_softmax(z_target, T_target))
    a = np.sum(np.minimum(p, q), axis=-1)
    return a, q, p


def total_variation(p, q) -> np.ndarray:
    """TV(p, q) = 1/2 sum_v |p(v) - q(v)| (used by Eq. rejection_rate)."""
    return 0.5 * np.sum(np.abs(np.asarray(p, np.float64) - np.asarray(q, np.float64)), axis=-1)


# ---------------------------------------------------------------------------
# Speculative window (Eqs. eal_generic, eal_full, eal_compact)
# ---------------------------------------------------------------------------
def prob_accepted_at_least(a) -> np.ndarray:
    """P(L >= k) = prod_{j<k} a_j for k = 1..K (Eq. eal_generic); shape [..., K]."""
    return np.cumprod(np.asarray(a, np.float64), axis=-1)


def length_distribution(a) -> np.ndarray:
    """P(L = l) for l = 0..K from the three cases of Section "Expected Accepted
    Length Loss": 1 - a_0, (prod_{j<l} a_j)(1 - a_l), and prod_{j<K} a_j.
    Shape [..., K+1]."""
    a = np.asarray(a, np.float64)
    K = a.shape[-1]
    out = np.empty(a.shape[:-1] + (K + 1,), np.float64)
    out[..., 0] = 1.0 - a[..., 0]
    for l in range(1, K):
        out[..., l] = np.prod(a[..., :l], axis=-1) * (1.0 - a[..., l])
    out[..., K] = np.prod(a, axis=-1)
    return out


def expected_length_full(a) -> np.ndarray:
    """E[L] = sum_l l * P(L = l) (Eq. eal_full)."""
    d = length_distribution(a)
    ell = np.arange(d.shape[-1], dtype=np.float64)
    return np.sum(ell * d, axis=-1)


def expected_length(a) -> np.ndarray:
    """E[L] = sum_{k=1..K} prod_{j<k} a_j (Eq. eal_compact / eal_generic)."""
    return np.sum(prob_accepted_at_least(a), axis=-1)


def expected_length_grad(a) -> np.ndarray:
    """dE[L]/da_j, from the definition of Eq. eal_compact term by term.

    E = sum_{k=1..K} prod_{i<k} a_i, so a_j appears in every term with k > j
    and d(term_k)/da_j = prod_{i<k, i != j} a_i.  Computed without division,
    so it is exact when some a_i is zero.
    """
    a = np.asarray(a, np.float64)
    K = a.shape[-1]
    g = np.zeros_like(a)
    for j in range(K):
        b = a.copy()
        b[..., j] = 1.0
        cp = np.cumprod(b, axis=-1)  # cp[k-1] = prod_{i<k, i != j} a_i
        g[..., j] = np.sum(cp[..., j:], axis=-1)
    return g


# ---------------------------------------------------------------------------
# Losses (Eq. loss_eal, Eq. loss_tv) and their gradients w.r.t. draft logits
# ---------------------------------------------------------------------------
def _window_loss(a):
    """loss = -(1/|W|) sum_windows E[L]; g = dloss/da.  a has shape [N, K]."""
    N = a.shape[0]
    E = expected_length(a)
    loss = -np.sum(E) / N
    g = -expected_length_grad(a) / N
    return loss, E, g


def eal_loss(z_draft, z_target, T_draft: float = 1.0, grad_scale: float = 1.0):
    """Greedy Expected-Accepted-Length loss and d loss / d z_draft (Eq. loss_eal).

    a_{n,j} = q_{n,j}(x*_{n,j}) with q = softmax of the draft logits at T_draft.
    The gradient chains dloss/da_j through the softmax Jacobian at temperature T:
    d q(x*) / d z(v) = (1/T) q(x*) (1[v = x*] - q(v)).  The target is frozen.
    ``grad_scale`` multiplies the returned gradient only (an upstream dL/dloss).

    Returns a dict with loss, E [N], a [N,K], xstar [N,K], grad [N,K,V].
    """
    zd = np.asarray(z_draft, np.float64)
    a, xs, q = acceptance_greedy(zd, z_target, T_draft)
    loss, E, g = _window_loss(a)
    onehot = np.zeros_like(q)
    np.put_along_axis(onehot, xs[..., None], 1.0, axis=-1)
    grad = (grad_scale * g * a / T_draft)[..., None] * (onehot - q)
    return {"loss": loss, "E": E, "a": a, "xstar": xs, "grad": grad}


def wtv_loss(z_draft, z_target, T_draft: float, T_target: float, grad_scale: float = 1.0):
    """Window-TV loss and d loss / d z_draft (Eq. loss_tv).

    a_{n,j} = sum_v min(p(v), q(v)) = 1 - TV.  With the reading
    d min(p, q)/dq = 1[q < p], d a / d q(u) = m(u) = 1[q(u) < p(u)], and the
    softmax Jacobian gives d a / d z(v) = (1/T_d) q(v) (m(v) - sum_u m(u) q(u)).
    Gradients flow only into the draft (the target is frozen).

    Returns a dict with loss, E [N], a [N,K], qlt [N,K] (= sum of q where
    q < p), tv [N,K], grad [N,K,V].
    """
    a, q, p = acceptance_sampling(z_draft, z_target, T_draft, T_target)
    loss, E, g = _window_loss(a)
    m = (q < p).astype(np.float64)
    qlt = np.sum(m * q, axis=-1)
    grad = (grad_scale * g / T_draft)[..., None] * q * (m - qlt[..., None])
    return {"loss": loss, "E": E, "a": a, "qlt": qlt, "tv": total_variation(p, q), "grad": grad}


# ---------------------------------------------------------------------------
# Simulated acceptance length and group-relative advantage (Section "GRPO Loss
# on Acceptance Length"; sampling verification of Eq. acc_sample)
# ---------------------------------------------------------------------------
def inverse_cdf_token(q, u1) -> np.ndarray:
    """Draft token drawn from q with the uniform u1: the smallest v with
    sum_{w <= v} q(w) > u1.  If rounding leaves no such v, the last v with
    q(v) > 0 is taken."""
    q = np.asarray(q, np.float64)
    C = np.cumsum(q, axis=-1)
    x = np.sum(C <= np.asarray(u1, np.float64)[..., None], axis=-1)
    V = q.shape[-1]
    over = x >= V
    if np.any(over):
        last_pos = V - 1 - np.argmax((q > 0)[..., ::-1], axis=-1)
        x = np.where(over, last_pos, x)
    return x


def simulate_acceptance(z_draft, z_target, T: float, u1, u2):
    """One simulated sampling-verification pass over windows of K positions.

    Per position: draw x ~ q~ by inverse CDF with u1, accept iff u2 < min(1, p~(x)/q~(x))
    (evaluated as u2 * q~(x) < p~(x)); the reward is the accepted length
    sum_k prod_{j<=k} accept_j, i.e. the count up to the first rejection
    (Section "Reward construction via simulated greedy verification", in its
    sampling-verification form).

    z_* have shape [..., K, V]; u1, u2 have shape [..., K].
    Returns (token, accept, reward, q, p).
    """
    q = np.exp(tempered_log_softmax(z_draft, T))
    p = np.exp(tempered_log_softmax(z_target, T))
    x = inverse_cdf_token(q, u1)
    qx = np.take_along_axis(q, x[..., None], axis=-1)[..., 0]
    px = np.take_along_axis(p, x[..., None], axis=-1)[..., 0]
    acc = np.asarray(u2, np.float64) * qx < px
    reward = np.sum(np.cumprod(acc.astype(np.int64), axis=-1), axis=-1)
    return x, acc, reward, q, p


def group_advantage(reward, eps: float = 1e-6, ddof: int = 0, clip: float | None = None):
    """A = clip((R - mean_g R) / (std_g R + eps), -C_A, C_A) (Eq. advantage).

    ``reward`` has shape [P, G]: P groups of G samples.  std is the group
    standard deviation with ``ddof`` (0: population).  ``clip`` None or <= 0
    leaves A unclipped.
    """
    r = np.asarray(reward, np.float64)
    G = r.shape[-1]
    mean = np.sum(r, axis=-1, keepdims=True) / G
    std = np.sqrt(np.sum((r - mean) ** 2, axis=-1, keepdims=True) / (G - ddof))
    A = (r - mean) / (std + eps)
    if clip is not None and clip > 0:
        A = np.clip(A, -clip, clip)
    return A


def sim_accept_grpo(z_draft, z_target, T: float, u1, u2, eps: float = 1e-6,
                    ddof: int = 0, clip: float | None = None):
    """Simulated acceptance reward and group advantages.

    z_* have shape [P, G, K, V], u1 and u2 [P, G, K].
    Returns a dict with token [P,G,K], accept [P,G,K], reward [P,G], advantage [P,G].
    """
    x, acc, r, _, _ = simulate_acceptance(z_draft, z_target, T, u1, u2)
    return {"token": x, "accept": acc, "reward": r,
            "advantage": group_advantage(r, eps, ddof, clip)}


# ---------------------------------------------------------------------------
# Sliding windows over sequences and the combined objectives of the
# experiments (Section "Window TV Loss", Figure wtv; Section "Settings")
# ---------------------------------------------------------------------------
LAYOUT_WINDOWS = 0    # [N, K, V]: N disjoint windows of K positions
LAYOUT_SEQUENCES = 1  # [B, S, V]: B sequences; a window starts at every t <= S - K


def window_rows(layout: int, B: int, S: int, K: int) -> np.ndarray:
    """Row indices [W, K] of every window.

    Windows layout: window n covers rows n*K .. n*K+K-1 (S is ignored).
    Sequences layout: the draft and the target are run once over each
    sequence and a window of K positions starts at every position t of it
    (the windows slide by one); only windows that fit entirely in the
    sequence are counted, so sequence b contributes windows t = 0..S-K,
    covering rows b*S + t .. b*S + t + K - 1.
    """
    if layout == LAYOUT_WINDOWS:
        return np.arange(B * K, dtype=np.int64).reshape(B, K)
    if layout == LAYOUT_SEQUENCES:
        if S < K:
            return np.zeros((0, K), np.int64)
        starts = (np.arange(B)[:, None] * S + np.arange(S - K + 1)[None, :]).reshape(-1)
        return starts[:, None] + np.arange(K)[None, :]
    raise ValueError("unknown layout")


def forward_kl(z_draft, z_target, T_draft: float, T_target: float):
    """Per-position forward KL of the anchor loss: KL(p~ || q~) =
    sum_v p~(v) (log p~(v) - log q~(v)), target p~ against draft q~, both at
    their temperatures (Section "Settings").  Returns (kl, q, p)."""
    lq = tempered_log_softmax(z_draft, T_draft)
    lp = tempered_log_softmax(z_target, T_target)
    p = np.exp(lp)
    return np.sum(p * (lp - lq), axis=-1), np.exp(lq), p


def window_length_coefficients(a, windows: np.ndarray):
    """For per-row acceptances ``a`` [R] and window rows [W, K]: the expected
    lengths E_w = sum_k prod_{j<k} a_{w,j} (Eq. eal_generic) and, per row,
    sum over the windows that contain it of dE_w/da_row."""
    a = np.asarray(a, np.float64)
    A = a[windows]
    E = expected_length(A) if len(windows) else np.zeros(0)
    dE = expected_length_grad(A) if len(windows) else np.zeros((0, windows.shape[1]))
    per_row = np.zeros_like(a)
    np.add.at(per_row, windows.reshape(-1), dE.reshape(-1))
    return E, per_row


def combined_loss(z_draft, z_target, T_draft: float, T_target: float, weights, layout: int,
                  B: int, S: int, K: int, labels=None, grad_scale: float = 1.0):
    """A weighted sum of the paper's training objectives over one batch:

        loss = w_wtv L_WTV + w_eal L_EAL + w_kl L_KL + w_tv L_TV

    * L_WTV = -(1/W) sum_windows E[L] with a = 1 - TV (Eq. loss_tv);
    * L_EAL = -(1/W) sum_windows E[L] with a = q~(x*) (Eq. loss_eal), x* the
      given label of the position, else the target's greedy token;
    * L_KL  = (1/R) sum_positions KL(p~ || q~), the forward-KL anchor;
    * L_TV  = (1/W) sum_windows (1/K) sum_j TV(p~, q~), the per-window mean
      TV auxiliary of the baselines (Section "Settings").
    W is the number of windows (``window_rows``), R the number of positions.
    Logits are [R, V] rows (any leading shape is flattened).  The gradient
    w.r.t. the draft logits chains each term through the softmax Jacobian at
    T_draft (the target is frozen): d a_tv / d z = (1/T) q (m - Q<),
    d a_eal / d z = (1/T) a (1[v=x*] - q), d KL / d z = (1/T) (q - p).

    Returns a dict: loss, terms [4] (L_WTV, L_EAL, L_KL, L_TV), E_tv [W],
    E_eal [W], a_tv [R], qlt [R], a_eal [R], xstar [R], kl [R], grad [R, V],
    and the per-row Jacobian coefficients coef_tv, coef_eal, coef_kl [R]
    (grad = coef_tv q (m - Q<) + coef_eal (1[v=x*] - q) + coef_kl (q - p)).
    """
    zd = np.asarray(z_draft, np.float64)
    zt = np.asarray(z_target, np.float64)
    V = zd.shape[-1]
    zd = zd.reshape(-1, V)
    zt = zt.reshape(-1, V)
    R = zd.shape[0]
    w_wtv, w_eal, w_kl, w_tv = (float(x) for x in weights)
    win = window_rows(layout, B, S, K)
    W = len(win)

    a_tv, q, p = acceptance_sampling(zd, zt, T_draft, T_target)
    m = (q < p).astype(np.float64)
    qlt = np.sum(m * q, axis=-1)
    xs = greedy_token(zt) if labels is None else np.asarray(labels, np.int64).reshape(-1)
    a_eal = np.take_along_axis(q, xs[:, None], axis=-1)[:, 0]
    kl, _, _ = forward_kl(zd, zt, T_draft, T_target)

    E_tv, dEtv = window_length_coefficients(a_tv, win)
    E_eal, dEeal = window_length_coefficients(a_eal, win)
    count = np.zeros(R)
    np.add.at(count, win.reshape(-1), 1.0)  # windows that contain each row

    terms = np.array([
        -np.sum(E_tv) / W if W else 0.0,
        -np.sum(E_eal) / W if W else 0.0,
        np.sum(kl) / R,
        np.sum(count * (1.0 - a_tv)) / (W * K) if W else 0.0,
    ])
    loss = w_wtv * terms[0] + w_eal * terms[1] + w_kl * terms[2] + w_tv * terms[3]

    # dloss/da per row, then through the softmax Jacobians
    g_tv = (-w_wtv * dEtv - w_tv * count / K) / W if W else np.zeros(R)
    g_eal = -w_eal * dEeal / W if W else np.zeros(R)
    g_kl = np.full(R, w_kl / R)
    onehot = np.zeros_like(q)
    np.put_along_axis(onehot, xs[:, None], 1.0, axis=-1)
    grad = (g_tv[:, None] * q * (m - qlt[:, None])
            + (g_eal * a_eal)[:, None] * (onehot - q)
            + g_kl[:, None] * (q - p)) * (grad_scale / T_draft)
    f = grad_scale / T_draft
    return {"loss": loss, "terms": terms, "E_tv": E_tv, "E_eal": E_eal, "a_tv": a_tv,
            "qlt": qlt, "a_eal": a_eal, "xstar": xs, "kl": kl, "grad": grad,
            "coef_tv": g_tv * f, "coef_eal": g_eal * a_eal * f, "coef_kl": g_kl * f}


# ---------------------------------------------------------------------------
# GRPO on the simulated greedy acceptance length (Section "GRPO Loss on
# Acceptance Length": greedy trajectories, Eq. debiased_reward, the policy
# ratio, Eq. advantage and the clipped surrogate)
# ---------------------------------------------------------------------------
def greedy_accepted_length(S_tokens, x_star) -> np.ndarray:
    """tau = sum_{k=1..K} prod_{j<=k} 1[S_j = x*_j]: the number of leading
    positions where the greedy draft token equals the target's token."""
    match = (np.asarray(S_tokens) == np.asarray(x_star)).astype(np.int64)
    return np.sum(np.cumprod(match, axis=-1), axis=-1)


def grpo_windows(layout: int, n_groups_or_B: int, S: int, m: int, K: int, anchors=None) -> np.ndarray:
    """Row indices [n_groups, m, K] of the windows of every group.

    Windows layout: rows are [n_groups * m * K]; group g holds windows
    g*m .. g*m+m-1, each K consecutive rows.  Sequences layout: B sequences of
    S positions and ``anchors`` [B, G] (start of each group's first window);
    group (b, g) holds the m windows starting at anchor, anchor+1, ...,
    anchor+m-1, each covering K consecutive positions (all sliced from the one
    forward pass over the sequence)."""
    if layout == LAYOUT_WINDOWS:
        return np.arange(n_groups_or_B * m * K, dtype=np.int64).reshape(n_groups_or_B, m, K)
    B = n_groups_or_B
    a = np.asarray(anchors, np.int64).reshape(B, -1)
    G = a.shape[1]
    starts = (np.arange(B)[:, None] * S + a)[:, :, None] + np.arange(m)[None, None, :]  # [B, G, m]
    rows = starts[..., None] + np.arange(K)  # [B, G, m, K]
    return rows.reshape(B * G, m, K)


def grpo_loss(z_theta, z_ref, z_target, T: float, layout: int, B: int, S: int, m: int, K: int,
              anchors=None, labels=None, eps: float = 1e-6, adv_clip: float = 0.0,
              eps_clip: float = 0.2, rho_min: float = 0.0, rho_max: float = np.inf,
              grad_scale: float = 1.0):
    """GRPO loss on the debiased greedy acceptance length and its gradient
    w.r.t. the current draft's logits ``z_theta`` (rows [R, V]).

    Per window (K positions) of group g:
      S^pi_k = argmax z_pi,k (lowest index on ties), for pi = theta and ref;
      tau^pi = greedy_accepted_length(S^pi, x*), x* = labels or argmax z_target;
      R = tau^theta - tau^ref (no gradient);
      log rho = (1/K) sum_k [log pi_theta(S^theta_k) - log pi_ref(S^theta_k)],
        pi = softmax(z / T), clipped to [-10, 10];
      rho = clip(exp(log rho), rho_min, rho_max);
      A = clip((R - mean_g R) / (std_g R + eps), -adv_clip, adv_clip)
        (population std over the group's m windows; adv_clip <= 0: no clip;
        no gradient);
      L_g = -(1/m) sum_{windows of g} min(rho A, clip(rho, 1-eps_clip, 1+eps_clip) A);
    loss = mean over all groups of L_g.

    The gradient flows through log pi_theta only.  Conventions at kinks: the
    derivative of a clip is taken as 1 strictly inside its interval and 0
    elsewhere, and min(u, v) takes the derivative of u when u <= v.
    d log pi_theta(S_k) / d z_theta,k(v) = (1/T) (1[v = S_k] - pi_theta,k(v)).

    Returns a dict: loss, group_loss [n_groups], S_theta, S_ref, x_star [R],
    tau_theta, tau_ref, reward, log_rho, rho, adv, coef [n_groups, m] (dloss /
    dlog rho of each window), grad [R, V].
    """
    zth = np.asarray(z_theta, np.float64)
    V = zth.shape[-1]
    zth = zth.reshape(-1, V)
    zrf = np.asarray(z_ref, np.float64).reshape(-1, V)
    n_groups = B if layout == LAYOUT_WINDOWS else B * np.asarray(anchors).reshape(B, -1).shape[1]
    win = grpo_windows(layout, B, S, m, K, anchors)  # [n_groups, m, K]

    lth = tempered_log_softmax(zth, T)
    lrf = tempered_log_softmax(zrf, T)
    S_th = np.argmax(zth, axis=-1)
    S_rf = np.argmax(zrf, axis=-1)
    if labels is not None:
        xs = np.asarray(labels, np.int64).reshape(-1)
    else:
        xs = greedy_token(np.asarray(z_target, np.float64).reshape(-1, V))
    rows = np.arange(zth.shape[0])
    lp_th = lth[rows, S_th]          # log pi_theta(S^theta)
    lp_rf = lrf[rows, S_th]          # log pi_ref(S^theta)

    tau_th = greedy_accepted_length(S_th[win], xs[win])   # [n_groups, m]
    tau_rf = greedy_accepted_length(S_rf[win], xs[win])
    reward = (tau_th - tau_rf).astype(np.float64)
    lr_raw = np.mean(lp_th[win] - lp_rf[win], axis=-1)    # [n_groups, m]
    log_rho = np.clip(lr_raw, -10.0, 10.0)
    rho_e = np.exp(log_rho)
    rho = np.clip(rho_e, rho_min, rho_max)
    adv = group_advantage(reward, eps, 0, adv_clip if adv_clip > 0 else None)
    clipped = np.clip(rho, 1.0 - eps_clip, 1.0 + eps_clip)
    u = rho * adv
    v = clipped * adv
    surrogate = np.minimum(u, v)
    group_loss = -np.mean(surrogate, axis=-1)
    loss = np.mean(group_loss)

    # dloss / d log rho, window by window
    d_clip = ((rho > 1.0 - eps_clip) & (rho < 1.0 + eps_clip)).astype(np.float64)
    d_sur_d_rho = np.where(u <= v, adv, adv * d_clip)
    d_rho_d_lr = np.where((rho_e > rho_min) & (rho_e < rho_max) & (lr_raw > -10.0) & (lr_raw < 10.0), rho_e, 0.0)
    coef = -(1.0 / (n_groups * m)) * d_sur_d_rho * d_rho_d_lr   # dloss/dlog rho
    # log rho = (1/K) sum_k log pi_theta(S_k) - const: spread over the window's rows
    row_coef = np.zeros(zth.shape[0])
    np.add.at(row_coef, win.reshape(-1), np.repeat(coef.reshape(-1), K) / K)
    pth = np.exp(lth)
    onehot = np.zeros_like(pth)
    onehot[rows, S_th] = 1.0
    grad = (grad_scale * row_coef / T)[:, None] * (onehot - pth)
    return {"loss": loss, "group_loss": group_loss, "S_theta": S_th, "S_ref": S_rf, "x_star": xs,
            "tau_theta": tau_th, "tau_ref": tau_rf, "reward": reward, "log_rho": log_rho, "rho": rho,
            "adv": adv, "coef": coef, "grad": grad}


# ---------------------------------------------------------------------------
# Flags for decisions that sit on a floating-point boundary
# ---------------------------------------------------------------------------
def sim_near_threshold(z_draft, z_target, T: float, u1, u2, tol: float = 1e-6):
    """Per position: True where u1 lies within ``tol`` of a CDF boundary of the
    chosen token, or u2 within ``tol`` of min(1, p/q) at that token.  Such
    decisions may legitimately differ between fp64 and a lower precision."""
    q = np.exp(tempered_log_softmax(z_draft, T))
    p = np.exp(tempered_log_softmax(z_target, T))
    u1 = np.asarray(u1, np.float64)
    x = inverse_cdf_token(q, u1)
    C = np.cumsum(q, axis=-1)
    hi = np.take_along_axis(C, x[..., None], axis=-1)[..., 0]
    lo = hi - np.take_along_axis(q, x[..., None], axis=-1)[..., 0]
    near1 = (np.abs(u1 - lo) <= tol) | (np.abs(u1 - hi) <= tol)
    qx = np.take_along_axis(q, x[..., None], axis=-1)[..., 0]
    px = np.take_along_axis(p, x[..., None], axis=-1)[..., 0]
    with np.errstate(divide="ignore", invalid="ignore"):
        thr = np.minimum(1.0, np.where(qx > 0, px / qx, 1.0))
    near2 = np.abs(np.asarray(u2, np.float64) - thr) <= tol
    return near1 | near2

