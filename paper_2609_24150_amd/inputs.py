"""Seeded synthetic logits and uniforms for the five benchmark workloads.

This module only draws random numbers and mixes them affinely: it holds none
of the arithmetic of the losses, so tests feed its output both to the HIP
library and to the fp64 oracle.  Tensors are generated in row chunks with a
generator seeded per (seed, recipe, stream, chunk), so a given call is
reproducible on a given device.

Recipes (logit rows are iid unless stated):
  c1  z_t ~ N(0, 2^2);                       z_d = 0.8 z_t + N(0, 1.2^2)
  c2  z_t ~ N(0, 3^2) + 8 on 32 peak tokens; z_d = 0.7 z_t + N(0, 1.5^2)
  c3  z_t ~ N(0, 2.5^2) + 10 on 8 peaks;     z_d = 0.6 z_t + N(0, 2^2); on 10% of
      rows (a seeded choice) the draft's +6 bumps at the target peaks move to 8
      other distinct non-peak tokens (low acceptance)
  c4  z_t ~ N(0, 2^2);                       z_d = 0.9 z_t + N(0, 0.5^2)
  c5  as c2, over [P, G, K, V], plus u1, u2 ~ U[0, 1) of shape [P, G, K]
Peak tokens are distinct per row, uniform without replacement.  bf16 logits
are drawn in fp32 and rounded to nearest even.
"""
from __future__ import annotations

import math

import torch

RECIPES = {
    "c1": dict(sigma_t=2.0, peaks=0, bump=0.0, alpha=0.8, sigma_d=1.2, shift_frac=0.0),
    "c2": dict(sigma_t=3.0, peaks=32, bump=8.0, alpha=0.7, sigma_d=1.5, shift_frac=0.0),
    "c3": dict(sigma_t=2.5, peaks=8, bump=10.0, alpha=0.6, sigma_d=2.0, shift_frac=0.1),
    "c4": dict(sigma_t=2.0, peaks=0, bump=0.0, alpha=0.9, sigma_d=0.5, shift_frac=0.0),
    "c5": dict(sigma_t=3.0, peaks=32, bump=8.0, alpha=0.7, sigma_d=1.5, shift_frac=0.0),
}
_RECIPE_ID = {k: i + 1 for i, k in enumerate(RECIPES)}

# The five workloads at full size.
CONFIGS = {
    "c1": dict(recipe="c1", op="eal", N=64, K=4, V=1024, dtype=torch.float32, temp_draft=1.0),
    "c2": dict(recipe="c2", op="wtv", N=2048, K=7, V=128256, dtype=torch.bfloat16,
               temp_draft=1.0, temp_target=1.0),
    "c3": dict(recipe="c3", op="eal+wtv", N=4096, K=5, V=151936, dtype=torch.bfloat16,
               temp_draft=1.0, wtv_temp=0.7),
    "c4": dict(recipe="c4", op="wtv", N=16384, K=16, V=32000, dtype=torch.float32,
               temp_draft=0.5, temp_target=0.5),
    "c5": dict(recipe="c5", op="sim", P=256, G=8, K=7, V=128256, dtype=torch.bfloat16, temp=1.0),
}


def _seed(seed: int, recipe: str, stream: int, chunk: int) -> int:
    s = seed
    for v in (_RECIPE_ID[recipe], stream, chunk):
        s = (s * 1_000_003 + v) % (1 << 62)
    return s


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_logits(recipe: str, shape, dtype=torch.bfloat16, seed: int = 0, device="cuda",
                chunk_elems: int = 1 << 27):
    """(z_draft, z_target) of `shape` ([..., V]) drawn from `recipe`."""
    r = RECIPES[recipe]
    shape = tuple(int(s) for s in shape)
    V = shape[-1]
    rows = math.prod(shape[:-1])
    zt = torch.empty(rows, V, dtype=dtype, device=device)
    zd = torch.empty(rows, V, dtype=dtype, device=device)
    npk = min(r["peaks"], V)
    nshift = 0
    shifted = None
    if r["shift_frac"] > 0 and npk > 0:
        nshift = int(round(r["shift_frac"] * rows))
        shifted = torch.zeros(rows, dtype=torch.bool, device=device)
        perm = torch.randperm(rows, generator=_gen(device, _seed(seed, recipe, 9, 0)), device=device)
        shifted[perm[:nshift]] = True
    chunk = max(1, chunk_elems // V)
    for ci, r0 in enumerate(range(0, rows, chunk)):
        r1 = min(rows, r0 + chunk)
        n = r1 - r0
        g = _gen(device, _seed(seed, recipe, 0, ci))
        t = torch.randn(n, V, generator=g, device=device) * r["sigma_t"]
        if npk > 0:
            keys = torch.rand(n, V, generator=g, device=device)
            peak_idx = keys.topk(npk, dim=1).indices
            t.scatter_add_(1, peak_idx, torch.full((n, npk), r["bump"], device=device))
        d = r["alpha"] * t + torch.randn(n, V, generator=g, device=device) * r["sigma_d"]
        if shifted is not None:
            sel = shifted[r0:r1]
            m = int(sel.sum())
            if m > 0 and V >= 2 * npk:
                rows_sel = sel.nonzero().squeeze(1)
                bump = r["alpha"] * r["bump"]
                sub = d[rows_sel]
                sub.scatter_add_(1, peak_idx[rows_sel], torch.full((m, npk), -bump, device=device))
                k2 = torch.rand(m, V, generator=g, device=device)
                k2.scatter_(1, peak_idx[rows_sel], -1.0)  # never pick a target peak
                new_idx = k2.topk(npk, dim=1).indices
                sub.scatter_add_(1, new_idx, torch.full((m, npk), bump, device=device))
                d[rows_sel] = sub
        zt[r0:r1] = t.to(dtype)
        zd[r0:r1] = d.to(dtype)
        del t, d
    return zd.view(shape), zt.view(shape)


def make_uniforms(shape, seed: int = 0, device="cuda"):
    """(u1, u2), fp32 in [0, 1), of `shape`."""
    g = _gen(device, _seed(seed, "c5", 7, 0))
    u1 = torch.rand(tuple(shape), generator=g, device=device, dtype=torch.float32)
    u2 = torch.rand(tuple(shape), generator=g, device=device, dtype=torch.float32)
    return u1, u2


def make_config(name: str, seed: int = 0, device="cuda", **overrides):
    """Inputs of workload `name` (optionally resized via N/K/V/P/G overrides).

    Returns a dict with z_draft, z_target (and u1, u2 for the simulation)."""
    cfg = dict(CONFIGS[name])
    cfg.update(overrides)
    if cfg["op"] == "sim":
        shape = (cfg["P"], cfg["G"], cfg["K"], cfg["V"])
    else:
        shape = (cfg["N"], cfg["K"], cfg["V"])
    zd, zt = make_logits(cfg["recipe"], shape, cfg["dtype"], seed, device)
    out = {"cfg": cfg, "z_draft": zd, "z_target": zt}
    if cfg["op"] == "sim":
        out["u1"], out["u2"] = make_uniforms(shape[:3], seed, device)
    return out
