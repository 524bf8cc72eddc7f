"""Python face of libaal: the C entry points under the same names, taking torch
tensors.  Each function checks shapes and dtypes, allocates its outputs and
workspace with torch, passes raw device pointers and the current HIP stream,
and returns.  It computes nothing itself.
"""
from __future__ import annotations

import torch

from . import _lib
from ._lib import AAL_BF16, AAL_F32, AAL_FLAG_STREAMING  # noqa: F401

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
    st = _lib.lib().aal_eal_fwd_bwd(
        _ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), N, K, V, float(temp_draft),
        _ptr(out["loss"]), _ptr(out["E"]), _ptr(out["accept"]), _ptr(out["xstar"]),
        _ptr(g), _dtype_code(g.dtype) if g is not None else AAL_F32, _ptr(grad_scale),
        int(flags), _ptr(ws), ws.numel(), _stream(dev, stream))
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
    st = _lib.lib().aal_wtv_fwd_bwd(
        _ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), N, K, V,
        float(temp_draft), float(temp_target),
        _ptr(out["loss"]), _ptr(out["E"]), _ptr(out["accept"]),
        _ptr(g), _dtype_code(g.dtype) if g is not None else AAL_F32, _ptr(grad_scale),
        int(flags), _ptr(ws), ws.numel(), _stream(dev, stream))
    _lib.check(st, "aal_wtv_fwd_bwd")
    return out


def aal_sim_accept_grpo(z_draft: torch.Tensor, z_target: torch.Tensor, u1: torch.Tensor, u2: torch.Tensor,
                        temperature: float = 1.0, *, eps: float = 1e-6, std_ddof: int = 0,
                        adv_clip: float = 0.0, ws: torch.Tensor | None = None, stream=None) -> dict:
    """Simulated acceptance length and group advantages on [P, G, K, V] logits
    with uniforms u1, u2 of shape [P, G, K].

    Returns a dict: token [P, G, K] int32, accept [P, G, K] int32,
    reward [P, G] int32, advantage [P, G] float32."""
    _check_logits(z_draft, z_target, 4)
    P, G, K, V = z_draft.shape
    dev = z_draft.device
    for u in (u1, u2):
        if u.shape != (P, G, K) or u.dtype != torch.float32 or u.device != dev or not u.is_contiguous():
            raise ValueError("u1 and u2 must be contiguous float32 device tensors of shape [P, G, K]")
    out = {
        "token": torch.empty(P, G, K, dtype=torch.int32, device=dev),
        "accept": torch.empty(P, G, K, dtype=torch.int32, device=dev),
        "reward": torch.empty(P, G, dtype=torch.int32, device=dev),
        "advantage": torch.empty(P, G, dtype=torch.float32, device=dev),
    }
    if ws is None:
        ws = workspace(P * G * K, P * G, dev)
    st = _lib.lib().aal_sim_accept_grpo(
        _ptr(z_draft), _ptr(z_target), _dtype_code(z_draft.dtype), P, G, K, V, float(temperature),
        _ptr(u1), _ptr(u2), _ptr(out["token"]), _ptr(out["accept"]), _ptr(out["reward"]),
        _ptr(out["advantage"]), float(eps), int(std_ddof), float(adv_clip),
        _ptr(ws), ws.numel(), _stream(dev, stream))
    _lib.check(st, "aal_sim_accept_grpo")
    return out
