"""Comparison helpers between the HIP library and the fp64 oracle.

Tolerances (stated once, used by every parity test):
  fp32 logits : loss and per-window E relative 1e-5; gradient max-abs 1e-6.
  bf16 logits : loss and E relative 1e-3 (fp32 accumulation of exact bf16
                inputs; observed errors are ~1e-6).
  gradients, elementwise, with c the row's coefficient (dloss/da times the
  softmax-Jacobian scale, from the oracle: G = c (1[v=x*] - q) for EAL,
  G = c q (m - Q<) for WTV):
      fp32 output : |G - G_o| <= 2^-18 |c| + 2^-126
      bf16 output : |G - bf16(G_o)| <= ulp_bf16(bf16(G_o)) + 2^-18 |c| + 2^-126
  The kernels compute every q in fp32, so each q carries an absolute error of
  a few 2^-24, and the sums Q< carry a few 2^-24 per term added; 2^-18 |c|
  bounds the resulting gradient error with margin.  The 2^-126 floor admits
  results below the fp32 normal range, which flush to zero.
  integers    : greedy tokens, sampled tokens and rewards bit-exact, except
                decisions the oracle flags as within 1e-6 of a threshold.
  WTV entries whose 1[q < p] may flip between fp32 and fp64 (|q - p| <=
  1e-5 max(p, q), ten times the fp32 error of the kernels' comparison in the
  log domain) are "near".  A flip of the near set F changes Q< by at most
  S = sum_{u in F} q_u, so every entry of such a row gets the extra allowance
  |c| q_v (S + 1[v in F]) on top of the tolerance above (the near entries'
  own mask may flip too); nothing is excluded, and the widened rows and the
  near entries are counted.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle as O


def host64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |x| (normal range; 2^-133 floor)."""
    ax = np.abs(x)
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    return np.where(ax > 0, np.exp2(np.maximum(e, -126) - 7), 2.0 ** -133)


def round_bf16(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def rel_err(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-30)))


KAPPA = 2.0 ** -18
FLOOR = 2.0 ** -126


def grad_stats(G: np.ndarray, Go: np.ndarray, coef: np.ndarray, in_dtype: torch.dtype, g_dtype: torch.dtype,
               exclude_rows: np.ndarray | None = None, exclude_elems: np.ndarray | None = None,
               extra_tol: np.ndarray | None = None) -> dict:
    """Elementwise gradient comparison over [rows, V] against the tolerance
    above (plus `extra_tol`, elementwise, where given); returns error
    statistics with the number of entries outside it ("bad") instead of
    asserting."""
    V = G.shape[-1]
    G = G.reshape(-1, V)
    Go = Go.reshape(-1, V)
    c = np.abs(coef).reshape(-1)
    keep = np.ones(G.shape[0], bool) if exclude_rows is None else ~exclude_rows.reshape(-1)
    emask = (np.zeros_like(G, bool) if exclude_elems is None else exclude_elems.reshape(-1, V))[keep]
    G, Go, c = G[keep], Go[keep], c[keep]
    err = np.where(emask, 0.0, np.abs(G - Go))
    stats = {"max_abs": float(err.max()) if err.size else 0.0, "gmax": float(np.abs(Go).max()) if Go.size else 0.0,
             "rows_checked": int(keep.sum()), "rows_excluded": int((~keep).sum()),
             "elems_checked": int(emask.size - emask.sum()), "elems_excluded": int(emask.sum())}
    tol = KAPPA * c[:, None] + FLOOR
    if extra_tol is not None:
        xt = extra_tol.reshape(-1, V)[keep]
        tol = tol + xt
        stats["rows_widened"] = int(np.sum(np.any(xt > 0, axis=1)))
        stats["max_widening_over_c"] = float(np.max(xt / np.maximum(c[:, None], 1e-300))) if xt.size else 0.0
    if g_dtype == torch.bfloat16:
        R = round_bf16(Go)
        bad = (np.abs(G - R) > bf16_ulp(R) * 1.0001 + tol) & ~emask
    else:
        bad = (err > tol) & ~emask
        if in_dtype == torch.float32 and stats["max_abs"] > 1e-6:
            bad = bad | (err > np.maximum(1e-6, tol))
    stats["bad"] = int(bad.sum())
    return stats


def check_grad(G: np.ndarray, Go: np.ndarray, coef: np.ndarray, in_dtype: torch.dtype, g_dtype: torch.dtype,
               exclude_rows: np.ndarray | None = None, exclude_elems: np.ndarray | None = None,
               extra_tol: np.ndarray | None = None) -> dict:
    """Elementwise gradient check over [rows, V]; returns error statistics."""
    stats = grad_stats(G, Go, coef, in_dtype, g_dtype, exclude_rows, exclude_elems, extra_tol)
    assert stats["bad"] == 0, f"gradient outside tolerance at {stats['bad']} entries: {stats}"
    return stats


def loss_tol(in_dtype: torch.dtype) -> float:
    return 1e-5 if in_dtype == torch.float32 else 1e-3


def wtv_flips(zd: np.ndarray, zt: np.ndarray, Td: float, Tt: float, coef: np.ndarray):
    """Extra elementwise allowance [rows, V] for a WTV gradient whose mask
    1[q < p] may flip between precisions at the near entries, and the near
    entries themselves [rows, V] (see the module docstring)."""
    q = np.exp(O.tempered_log_softmax(zd, Td))
    p = np.exp(O.tempered_log_softmax(zt, Tt))
    near = np.abs(q - p) <= 1e-5 * np.maximum(p, q)
    s_near = np.sum(np.where(near, q, 0.0), axis=-1, keepdims=True)
    extra = np.abs(np.asarray(coef, np.float64))[..., None] * q * (s_near + near)
    return extra, near


def eal_coef(o: dict, N: int, T: float, scale: float = 1.0) -> np.ndarray:
    return -O.expected_length_grad(o["a"]) / N * o["a"] / T * scale


def wtv_coef(o: dict, N: int, T: float, scale: float = 1.0) -> np.ndarray:
    return -O.expected_length_grad(o["a"]) / N / T * scale
