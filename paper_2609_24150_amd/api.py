"""Python face of libaal: the C entry points under the same names, taking torch
tensors.  Each function checks shapes and dtypes, allocates its outputs and
workspace with torch, passes raw device pointers and the current HIP stream,
and returns.  It computes nothing itself.
"""
from __future__ import annotations

import torch

from . import _lib
from ._lib import (  # noqa: F401
    AAL_BF16, AAL_F32, AAL_FLAG_COOPERATIVE, AAL_FLAG_STREAMING, AAL_LAYOUT_SEQUENCES, AAL_LAYOUT_WINDOWS,
    AAL_VP_EAL, AAL_VP_WTV,
)

_DT = {torch.bfloat16: AAL_BF16, torch.float32: AAL_F32}


def _dtype_code(t: torch.dtype) -> int:
    if t not in _DT:
        raise TypeError(f"unsupported dtype {t}; use torch.bfloat16 or torch.float32")
    return _DT[t]


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device, stream):
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def aal_workspace_bytes(rows: int, windows: int) -> int:
    return int(_lib.lib().aal_workspace_bytes(rows, windows))


def workspace(rows: int, windows: int, device) -> torch.Tensor:
    """A workspace tensor sized for `rows` logit rows and `windows` windows."""
    return torch.empty(aal_workspace_bytes(rows, windows), dtype=torch.uint8, device=device)


def _check_logits(z_draft: torch.Tensor, z_target: torch.Tensor, ndim: int):
    if z_draft.shape != z_target.shape or z_draft.dim() != ndim:
        raise ValueError(f"z_draft and z_target must both have {ndim} dims and equal shapes; got "
                         f"{tuple(z_draft.shape)} and {tuple(z_target.shape)}")
    if z_draft.dtype != z_target.dtype:
        raise TypeError("z_draft and z_target must share a dtype")
    if not (z_draft.is_cuda and z_target.is_cuda):
        raise ValueError("logits must be device tensors")
    if not (z_draft.is_contiguous() and z_target.is_contiguous()):
        raise ValueError("logits must be contiguous")


def _loss_outputs(N, K, V, dev, grad, grad_dtype, ref_dtype):
    out = {
        "loss": torch.empty(1, dtype=torch.float32, device=dev),
        "E": torch.empty(N, dtype=torch.float32, device=dev),
        "accept": torch.empty(N, K, dtype=torch.float32, device=dev),
    }
    out["grad"] = (torch.empty(N, K, V, dtype=grad_dtype or ref_dtype, device=dev) if grad else None)
    return out


def aal_eal_fwd_bwd(z_draft: torch.Tensor, z_target: torch.Tensor, temp_draft: float = 1.0, *,
                    grad: bool = True, grad_dtype: torch.dtype | None = None,
                    grad_scale: torch.Tensor | None = None, flags: int = 0,
                    ws: torch.Tensor | None = None, stream=None) -> dict:
    """Greedy EAL loss forward + backward on [N, K, V] logits.

    Returns a dict: loss [1], E [N], accept [N, K], xstar [N, K] int32 and
    grad [N, K, V] (None when grad=False)."""
    _check_logits(z_draft, z_target, 3)
    N, K, V = z_draft.shape
    dev = z_draft.device
    out = _loss_outputs(N, K, V, dev, grad, grad_dtype, z_draft.dtype)
    out["xstar"] = torch.empty(N, K, dtype=torch.int32, device=dev)
    g = out["grad"]
    if ws is None:
        ws = workspace(N * K, N, dev)
    if grad_scale is not None and (grad_scale.dtype != torch.float32 or grad_scale.device != dev):
        raise TypeError("grad_scale must be a float32 device tensor")
    args = [_ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), N, K, V, float(temp_draft),
            _ptr(out["loss"]), _ptr(out["E"]), _ptr(out["accept"]), _ptr(out["xstar"]),
            _ptr(g), _dtype_code(g.dtype) if g is not None else AAL_F32, _ptr(grad_scale)]
    tail = [_ptr(ws), ws.numel(), _stream(dev, stream)]
    if flags:
        st = _lib.lib().aal_eal_fwd_bwd_ex(*args, int(flags), *tail)
    else:
        st = _lib.lib().aal_eal_fwd_bwd(*args, *tail)
    _lib.check(st, "aal_eal_fwd_bwd")
    return out


def aal_wtv_fwd_bwd(z_draft: torch.Tensor, z_target: torch.Tensor, temp_draft: float = 1.0,
                    temp_target: float = 1.0, *, grad: bool = True, grad_dtype: torch.dtype | None = None,
                    grad_scale: torch.Tensor | None = None, flags: int = 0,
                    ws: torch.Tensor | None = None, stream=None) -> dict:
    """Window-TV loss forward + backward on [N, K, V] logits.

    Returns a dict: loss [1], E [N], accept [N, K] (= sum min(p, q)) and
    grad [N, K, V] (None when grad=False)."""
    _check_logits(z_draft, z_target, 3)
    N, K, V = z_draft.shape
    dev = z_draft.device
    out = _loss_outputs(N, K, V, dev, grad, grad_dtype, z_draft.dtype)
    g = out["grad"]
    if ws is None:
        ws = workspace(N * K, N, dev)
    if grad_scale is not None and (grad_scale.dtype != torch.float32 or grad_scale.device != dev):
        raise TypeError("grad_scale must be a float32 device tensor")
    args = [_ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), N, K, V,
            float(temp_draft), float(temp_target),
            _ptr(out["loss"]), _ptr(out["E"]), _ptr(out["accept"]),
            _ptr(g), _dtype_code(g.dtype) if g is not None else AAL_F32, _ptr(grad_scale)]
    tail = [_ptr(ws), ws.numel(), _stream(dev, stream)]
    if flags:
        st = _lib.lib().aal_wtv_fwd_bwd_ex(*args, int(flags), *tail)
    else:
        st = _lib.lib().aal_wtv_fwd_bwd(*args, *tail)
    _lib.check(st, "aal_wtv_fwd_bwd")
    return out


def aal_sim_accept_grpo(z_draft: torch.Tensor, z_target: torch.Tensor, u1: torch.Tensor, u2: torch.Tensor,
                        temperature: float = 1.0, *, eps: float = 1e-6, std_ddof: int = 0,
                        adv_clip: float = 0.0, accept: bool = True, ws: torch.Tensor | None = None,
                        stream=None) -> dict:
    """Simulated acceptance length and group advantages on [P, G, K, V] logits
    with uniforms u1, u2 of shape [P, G, K].

    Returns a dict: token [P, G, K] int32, accept [P, G, K] int32 (None with
    accept=False, which calls the entry point without that output),
    reward [P, G] int32, advantage [P, G] float32."""
    _check_logits(z_draft, z_target, 4)
    P, G, K, V = z_draft.shape
    dev = z_draft.device
    for u in (u1, u2):
        if u.shape != (P, G, K) or u.dtype != torch.float32 or u.device != dev or not u.is_contiguous():
            raise ValueError("u1 and u2 must be contiguous float32 device tensors of shape [P, G, K]")
    out = {
        "token": torch.empty(P, G, K, dtype=torch.int32, device=dev),
        "accept": torch.empty(P, G, K, dtype=torch.int32, device=dev) if accept else None,
        "reward": torch.empty(P, G, dtype=torch.int32, device=dev),
        "advantage": torch.empty(P, G, dtype=torch.float32, device=dev),
    }
    if ws is None:
        ws = workspace(P * G * K, P * G, dev)
    head = [_ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), P, G, K, V, float(temperature),
            _ptr(u1), _ptr(u2), _ptr(out["token"])]
    tail = [_ptr(out["reward"]), _ptr(out["advantage"]), float(eps), int(std_ddof), float(adv_clip),
            _ptr(ws), ws.numel(), _stream(dev, stream)]
    if accept:
        st = _lib.lib().aal_sim_accept_grpo_ex(*head, _ptr(out["accept"]), *tail)
    else:
        st = _lib.lib().aal_sim_accept_grpo(*head, *tail)
    _lib.check(st, "aal_sim_accept_grpo")
    return out


def aal_loss_workspace_bytes(layout: int, B: int, S: int, K: int) -> int:
    return int(_lib.lib().aal_loss_workspace_bytes(int(layout), int(B), int(S), int(K)))


def aal_loss_fwd_bwd(z_draft: torch.Tensor, z_target: torch.Tensor | None, K: int, *,
                     weights=(0.0, 0.0, 0.0, 0.0), temp_draft: float = 1.0, temp_target: float = 1.0,
                     layout: int = AAL_LAYOUT_WINDOWS, labels: torch.Tensor | None = None,
                     grad: bool = True, grad_dtype: torch.dtype | None = None,
                     grad_scale: torch.Tensor | None = None, flags: int = 0, outputs: bool = True,
                     ws: torch.Tensor | None = None, stream=None) -> dict:
    """Combined objective forward + backward (weights = (wtv, eal, kl, tv)).

    Windows layout: logits [N, K, V] (N disjoint windows).  Sequences layout:
    logits [B, S, V]; a window of K positions starts at every t <= S - K.
    labels: int32 [rows] (or the logits' leading shape) replacing the greedy
    target token of the EAL term, or None.  z_target may be None only when
    the EAL term alone is asked for with labels.

    Returns a dict: loss [1], terms [4] (L_WTV, L_EAL, L_KL, L_TV), E_tv [W],
    E_eal [W], accept_tv [R], accept_eal [R], xstar [R] int32, grad (the
    logits' shape, or None).  With outputs=False the per-window and per-row
    arrays are not requested (None in the dict)."""
    if z_draft.dim() != 3 or not z_draft.is_cuda or not z_draft.is_contiguous():
        raise ValueError("z_draft must be a contiguous [B, S or K, V] device tensor")
    if z_target is not None:
        if z_target.shape != z_draft.shape or z_target.dtype != z_draft.dtype or not z_target.is_contiguous():
            raise ValueError("z_target must match z_draft in shape, dtype and layout")
    B, S, V = z_draft.shape
    if layout == AAL_LAYOUT_WINDOWS and S != K:
        raise ValueError("windows layout needs logits of shape [N, K, V]")
    R = B * S
    W = B if layout == AAL_LAYOUT_WINDOWS else B * max(0, S - K + 1)
    dev = z_draft.device
    if labels is not None and (labels.dtype != torch.int32 or labels.numel() != R or not labels.is_contiguous()
                               or labels.device != dev):
        raise ValueError("labels must be a contiguous int32 device tensor with one entry per row")
    if grad_scale is not None and (grad_scale.dtype != torch.float32 or grad_scale.device != dev):
        raise TypeError("grad_scale must be a float32 device tensor")
    out = {
        "loss": torch.empty(1, dtype=torch.float32, device=dev),
        "terms": torch.empty(4, dtype=torch.float32, device=dev),
        "E_tv": torch.empty(W, dtype=torch.float32, device=dev) if outputs else None,
        "E_eal": torch.empty(W, dtype=torch.float32, device=dev) if outputs else None,
        "accept_tv": torch.empty(R, dtype=torch.float32, device=dev) if outputs else None,
        "accept_eal": torch.empty(R, dtype=torch.float32, device=dev) if outputs else None,
        "xstar": torch.empty(R, dtype=torch.int32, device=dev) if outputs else None,
        "grad": torch.empty(B, S, V, dtype=grad_dtype or z_draft.dtype, device=dev) if grad else None,
    }
    if ws is None:
        ws = torch.empty(aal_loss_workspace_bytes(layout, B, S, K), dtype=torch.uint8, device=dev)
    g = out["grad"]
    w = _lib.LossWeights(*(float(x) for x in weights))
    st = _lib.lib().aal_loss_fwd_bwd(
        _ptr(z_draft), _ptr(z_target), _ptr(labels), _dtype_code(z_draft.dtype), int(layout), B, S, K, V,
        float(temp_draft), float(temp_target), w, _ptr(out["loss"]), _ptr(out["terms"]),
        _ptr(out["E_tv"]) if W and outputs else None, _ptr(out["E_eal"]) if W and outputs else None,
        _ptr(out["accept_tv"]), _ptr(out["accept_eal"]), _ptr(out["xstar"]),
        _ptr(g), _dtype_code(g.dtype) if g is not None else AAL_F32, _ptr(grad_scale), int(flags),
        _ptr(ws), ws.numel(), _stream(dev, stream))
    _lib.check(st, "aal_loss_fwd_bwd")
    return out


def aal_grpo_workspace_bytes(layout: int, B: int, S: int, G: int, m: int, K: int) -> int:
    return int(_lib.lib().aal_grpo_workspace_bytes(int(layout), int(B), int(S), int(G), int(m), int(K)))


def aal_grpo_fwd_bwd(z_theta: torch.Tensor, z_ref: torch.Tensor, z_target: torch.Tensor | None, m: int, K: int, *,
                     layout: int = AAL_LAYOUT_WINDOWS, anchors: torch.Tensor | None = None,
                     labels: torch.Tensor | None = None, temperature: float = 1.0, eps: float = 1e-6,
                     adv_clip: float = 0.0, eps_clip: float = 0.2, rho_min: float = 0.0,
                     rho_max: float = float("inf"), grad: bool = True, grad_dtype: torch.dtype | None = None,
                     grad_scale: torch.Tensor | None = None, ws: torch.Tensor | None = None, stream=None) -> dict:
    """GRPO loss on the debiased greedy acceptance length, forward + backward
    w.r.t. z_theta.

    Windows layout: logits [B, m*K, V] (B groups of m windows of K rows).
    Sequences layout: logits [B, S, V] and anchors int32 [B, G].
    Returns a dict: loss [1], tau_theta, tau_ref [groups, m] int32,
    advantage, log_rho [groups, m], grad (the logits' shape, or None)."""
    for t in (z_theta, z_ref) + ((z_target,) if z_target is not None else ()):
        if t.dim() != 3 or not t.is_cuda or not t.is_contiguous() or t.shape != z_theta.shape or t.dtype != z_theta.dtype:
            raise ValueError("logits must be contiguous device tensors of one shape [B, rows, V] and dtype")
    B, S, V = z_theta.shape
    dev = z_theta.device
    if layout == AAL_LAYOUT_WINDOWS:
        if S != m * K:
            raise ValueError("windows layout needs logits of shape [groups, m*K, V]")
        G, groups = 1, B
    else:
        if anchors is None or anchors.dim() != 2 or anchors.shape[0] != B or anchors.dtype != torch.int32:
            raise ValueError("sequences layout needs int32 anchors of shape [B, G]")
        G = anchors.shape[1]
        groups = B * G
        anchors = anchors.contiguous()
    if labels is not None and (labels.dtype != torch.int32 or labels.numel() != B * S or labels.device != dev):
        raise ValueError("labels must be an int32 device tensor with one entry per row")
    if grad_scale is not None and (grad_scale.dtype != torch.float32 or grad_scale.device != dev):
        raise TypeError("grad_scale must be a float32 device tensor")
    out = {
        "loss": torch.empty(1, dtype=torch.float32, device=dev),
        "tau_theta": torch.empty(groups, m, dtype=torch.int32, device=dev),
        "tau_ref": torch.empty(groups, m, dtype=torch.int32, device=dev),
        "advantage": torch.empty(groups, m, dtype=torch.float32, device=dev),
        "log_rho": torch.empty(groups, m, dtype=torch.float32, device=dev),
        "grad": torch.empty(B, S, V, dtype=grad_dtype or z_theta.dtype, device=dev) if grad else None,
    }
    if ws is None:
        ws = torch.empty(aal_grpo_workspace_bytes(layout, B, S, G, m, K), dtype=torch.uint8, device=dev)
    g = out["grad"]
    prm = _lib.GrpoParams(float(eps), float(adv_clip), float(eps_clip), float(rho_min), float(rho_max))
    st = _lib.lib().aal_grpo_fwd_bwd(
        _ptr(z_theta), _ptr(z_ref), _ptr(z_target), _ptr(labels), _dtype_code(z_theta.dtype), int(layout),
        B, S, G, m, K, V, _ptr(anchors), float(temperature), prm, _ptr(out["loss"]), _ptr(out["tau_theta"]),
        _ptr(out["tau_ref"]), _ptr(out["advantage"]), _ptr(out["log_rho"]),
        _ptr(g), _dtype_code(g.dtype) if g is not None else AAL_F32, _ptr(grad_scale),
        _ptr(ws), ws.numel(), _stream(dev, stream))
    _lib.check(st, "aal_grpo_fwd_bwd")
    return out


# ----------------------------------------------------------------------------
# Vocabulary-parallel pieces (one rank's share of a vocabulary-split LM head).
# Records are uint8 device tensors of shape [rows, record bytes]; view them as
# float32 / int32 to read fields.  The caller gathers the records over ranks.

def _vp_slice(z_draft, z_target, need_target=True):
    if z_draft.dim() != 2:
        raise ValueError("vocabulary slices are [rows, V_slice]")
    if need_target or z_target is not None:
        _check_logits(z_draft, z_target, 2)
    elif not (z_draft.is_cuda and z_draft.is_contiguous()):
        raise ValueError("z_draft must be a contiguous device tensor")
    return z_draft.shape[0], z_draft.shape[1], z_draft.device


def _records(t: torch.Tensor, nbytes: int, name: str, lead: int):
    if t.dtype != torch.uint8 or t.dim() != lead + 1 or t.shape[-1] != nbytes or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous uint8 tensor of records of {nbytes} bytes")


def aal_vp_row_partials(z_draft: torch.Tensor, z_target: torch.Tensor | None, v0: int, mode: int,
                        temp_draft: float = 1.0, temp_target: float = 1.0, *, V_total: int,
                        labels: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Step 1: partial row statistics of the slice [v0, v0 + V_slice) of a
    vocabulary of V_total entries.  EAL may take int32 labels [rows] (global
    token ids, clamped into [0, V_total)) in place of the target's greedy
    token; the target slice may then be None.  Returns [rows, 32] records."""
    rows, vs, dev = _vp_slice(z_draft, z_target, need_target=labels is None)
    if labels is not None and (labels.dtype != torch.int32 or labels.numel() != rows or labels.device != dev
                               or not labels.is_contiguous()):
        raise ValueError("labels must be a contiguous int32 device tensor with one entry per row")
    parts = torch.empty(rows, _lib.VP_PART_BYTES, dtype=torch.uint8, device=dev)
    st = _lib.lib().aal_vp_row_partials(_ptr(z_draft), _ptr(z_target), _ptr(labels), _dtype_code(z_draft.dtype),
                                        rows, vs, int(v0), int(V_total), int(mode), float(temp_draft),
                                        float(temp_target),
                                        _ptr(parts), _stream(dev, stream))
    _lib.check(st, "aal_vp_row_partials")
    return parts


def aal_vp_merge_rows(parts_all: torch.Tensor, mode: int, temp_draft: float = 1.0, temp_target: float = 1.0, *,
                      stream=None) -> torch.Tensor:
    """Step 2: merge gathered partials [R, rows, 32] in rank order.  Returns [rows, 32] row records."""
    _records(parts_all, _lib.VP_PART_BYTES, "parts_all", 2)
    R, rows = parts_all.shape[0], parts_all.shape[1]
    dev = parts_all.device
    row = torch.empty(rows, _lib.VP_ROW_BYTES, dtype=torch.uint8, device=dev)
    st = _lib.lib().aal_vp_merge_rows(_ptr(parts_all), R, rows, int(mode), float(temp_draft), float(temp_target),
                                      _ptr(row), _stream(dev, stream))
    _lib.check(st, "aal_vp_merge_rows")
    return row


def aal_vp_accept_partials(z_draft: torch.Tensor, z_target: torch.Tensor, row: torch.Tensor,
                           temp_draft: float = 1.0, temp_target: float = 1.0, *, stream=None) -> torch.Tensor:
    """Step 3 (WTV): the slice's sum min(p, q) and Q< partials.  Returns [rows, 8] records."""
    rows, vs, dev = _vp_slice(z_draft, z_target)
    _records(row, _lib.VP_ROW_BYTES, "row", 1)
    if row.shape[0] != rows:
        raise ValueError("row must hold one record per logit row")
    acc = torch.empty(rows, _lib.VP_ACC_BYTES, dtype=torch.uint8, device=dev)
    st = _lib.lib().aal_vp_accept_partials(_ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), rows, vs,
                                           float(temp_draft), float(temp_target), _ptr(row), _ptr(acc),
                                           _stream(dev, stream))
    _lib.check(st, "aal_vp_accept_partials")
    return acc


def aal_vp_window_scan(row: torch.Tensor, acc_all: torch.Tensor | None, N: int, K: int, mode: int,
                       temp_draft: float = 1.0, *, grad_scale: torch.Tensor | None = None, stream=None) -> dict:
    """Step 4: window scan over the merged rows (updated in place with a, qlt
    and coef).  acc_all [R, N*K, 8] in WTV mode.  Returns loss [1], E [N],
    accept [N, K] and, in EAL mode, xstar [N, K]."""
    _records(row, _lib.VP_ROW_BYTES, "row", 1)
    if row.shape[0] != N * K:
        raise ValueError("row must hold N*K records")
    dev = row.device
    R = 0
    if mode == _lib.AAL_VP_WTV:
        if acc_all is None:
            raise ValueError("acc_all is required in WTV mode")
        _records(acc_all, _lib.VP_ACC_BYTES, "acc_all", 2)
        if acc_all.shape[1] != N * K:
            raise ValueError("acc_all must be [R, N*K, 8]")
        R = acc_all.shape[0]
    if grad_scale is not None and (grad_scale.dtype != torch.float32 or grad_scale.device != dev):
        raise TypeError("grad_scale must be a float32 device tensor")
    out = {
        "loss": torch.empty(1, dtype=torch.float32, device=dev),
        "E": torch.empty(N, dtype=torch.float32, device=dev),
        "accept": torch.empty(N, K, dtype=torch.float32, device=dev),
    }
    if mode == _lib.AAL_VP_EAL:
        out["xstar"] = torch.empty(N, K, dtype=torch.int32, device=dev)
    st = _lib.lib().aal_vp_window_scan(_ptr(row), _ptr(acc_all) if R else None, R, N, K, int(mode),
                                       float(temp_draft), _ptr(grad_scale), _ptr(out["loss"]), _ptr(out["E"]),
                                       _ptr(out["accept"]), _ptr(out.get("xstar")), _stream(dev, stream))
    _lib.check(st, "aal_vp_window_scan")
    return out


def aal_vp_sequence_scan(row: torch.Tensor, acc_all: torch.Tensor | None, B: int, S: int, K: int, mode: int,
                         temp_draft: float = 1.0, *, grad_scale: torch.Tensor | None = None, stream=None) -> dict:
    """Step 4 for B sequences of S positions with windows of K sliding by one
    (rows updated in place).  Returns loss [1], E [B*(S-K+1)], accept [B, S]
    and, in EAL mode, xstar [B, S]."""
    _records(row, _lib.VP_ROW_BYTES, "row", 1)
    if row.shape[0] != B * S:
        raise ValueError("row must hold B*S records")
    dev = row.device
    R = 0
    if mode == _lib.AAL_VP_WTV:
        if acc_all is None:
            raise ValueError("acc_all is required in WTV mode")
        _records(acc_all, _lib.VP_ACC_BYTES, "acc_all", 2)
        if acc_all.shape[1] != B * S:
            raise ValueError("acc_all must be [R, B*S, 8]")
        R = acc_all.shape[0]
    if grad_scale is not None and (grad_scale.dtype != torch.float32 or grad_scale.device != dev):
        raise TypeError("grad_scale must be a float32 device tensor")
    out = {
        "loss": torch.empty(1, dtype=torch.float32, device=dev),
        "E": torch.empty(B * max(0, S - K + 1), dtype=torch.float32, device=dev),
        "accept": torch.empty(B, S, dtype=torch.float32, device=dev),
    }
    if mode == _lib.AAL_VP_EAL:
        out["xstar"] = torch.empty(B, S, dtype=torch.int32, device=dev)
    st = _lib.lib().aal_vp_sequence_scan(_ptr(row), _ptr(acc_all) if R else None, R, B, S, K, int(mode),
                                         float(temp_draft), _ptr(grad_scale), _ptr(out["loss"]), _ptr(out["E"]),
                                         _ptr(out["accept"]), _ptr(out.get("xstar")), _stream(dev, stream))
    _lib.check(st, "aal_vp_sequence_scan")
    return out


def aal_vp_grad(z_draft: torch.Tensor, z_target: torch.Tensor | None, row: torch.Tensor, v0: int, mode: int,
                temp_draft: float = 1.0, temp_target: float = 1.0, *, grad_dtype: torch.dtype | None = None,
                stream=None) -> torch.Tensor:
    """Step 5: the slice [v0, v0 + V_slice) of dloss/dz_draft.  Returns [rows, V_slice]."""
    rows, vs, dev = _vp_slice(z_draft, z_target, need_target=(mode == _lib.AAL_VP_WTV))
    _records(row, _lib.VP_ROW_BYTES, "row", 1)
    if row.shape[0] != rows:
        raise ValueError("row must hold one record per logit row")
    g = torch.empty(rows, vs, dtype=grad_dtype or z_draft.dtype, device=dev)
    st = _lib.lib().aal_vp_grad(_ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), rows, vs, int(v0),
                                int(mode), float(temp_draft), float(temp_target), _ptr(row), _ptr(g),
                                _dtype_code(g.dtype), _stream(dev, stream))
    _lib.check(st, "aal_vp_grad")
    return g


def aal_stream_probe(srcs, dst: torch.Tensor | None = None, flag: torch.Tensor | None = None, stream=None):
    """Measurement aid: stream 1-3 equally sized device tensors (16-byte
    nontemporal loads) and, with dst, write their 32-bit wrapping sum there;
    without dst, flag ([1] int32/uint32) is set only where a sum is all ones.
    Enqueues and returns; time it with events on `stream`."""
    srcs = list(srcs)
    if not 1 <= len(srcs) <= 3:
        raise ValueError("one to three sources")
    nbytes = srcs[0].numel() * srcs[0].element_size()
    for t in srcs + ([dst] if dst is not None else []):
        if not t.is_cuda or not t.is_contiguous() or t.numel() * t.element_size() != nbytes:
            raise ValueError("sources and dst must be contiguous device tensors of one size")
    if dst is None and flag is None:
        raise ValueError("flag is required without dst")
    ptrs = [_ptr(t) for t in srcs] + [None] * (3 - len(srcs))
    st = _lib.lib().aal_stream_probe(ptrs[0], ptrs[1], ptrs[2], _ptr(dst), nbytes, _ptr(flag),
                                     _stream(srcs[0].device, stream))
    _lib.check(st, "aal_stream_probe")
