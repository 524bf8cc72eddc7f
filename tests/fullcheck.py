"""Full-size comparison of the HIP library with the fp64 oracle, every window.

The GPU computes a whole workload; its inputs and its gradient are copied
into host shared memory, and a pool of host processes runs the oracle over
chunks of windows (or rows, prefixes, groups) and compares the gradient
elementwise in place, returning the oracle's per-window and per-row values and
the comparison statistics.  The parent then compares every window's E, every
row's acceptance and greedy token, and the loss (minus the mean of the oracle's
E over all windows), and reports the exclusion and near-threshold counts.

The pool is started with the "spawn" method, so no worker inherits the GPU
state of the parent; workers use only NumPy and the oracle (and torch on the
CPU for bf16 rounding).  At most 16 workers run: one GPU's share of the host.
"""
from __future__ import annotations

import json
import multiprocessing as mp
import os
from multiprocessing import shared_memory

import numpy as np
import torch

HOST_CPU_SHARE = 16

_KINDS = {torch.bfloat16: ("bf16", np.int16, torch.int16), torch.float32: ("f32", np.float32, torch.float32),
          torch.int32: ("i32", np.int32, torch.int32)}


def n_workers() -> int:
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    return max(1, min(HOST_CPU_SHARE, cores))


def make_pool():
    return mp.get_context("spawn").Pool(n_workers())


class Shared:
    """Named host shared-memory copies of device tensors (unlinked on exit)."""

    def __init__(self):
        self.blocks = []

    def put(self, t: torch.Tensor):
        kind, npdt, tdt = _KINDS[t.dtype]
        t = t.contiguous()
        nbytes = t.numel() * t.element_size()
        shm = shared_memory.SharedMemory(create=True, size=max(nbytes, 8))
        self.blocks.append(shm)
        arr = np.ndarray(tuple(t.shape), dtype=npdt, buffer=shm.buf)
        torch.from_numpy(arr).copy_(t.view(tdt))
        del arr
        return (shm.name, tuple(t.shape), kind)

    def drop(self, spec):
        """Unlink one block (its spec came from put)."""
        for shm in list(self.blocks):
            if shm.name == spec[0]:
                shm.close()
                shm.unlink()
                self.blocks.remove(shm)

    def close(self):
        for shm in self.blocks:
            shm.close()
            shm.unlink()
        self.blocks = []

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


# ------------------------------------------------------------------ workers
_ATTACHED: dict = {}


def _raw(spec):
    name, shape, kind = spec
    if name not in _ATTACHED:
        # spawned workers share the parent's resource tracker, so attaching
        # re-registers the parent's own entry, which the parent's unlink clears
        _ATTACHED[name] = shared_memory.SharedMemory(name=name)
    npdt = {"bf16": np.int16, "f32": np.float32, "i32": np.int32}[kind]
    return np.ndarray(shape, dtype=npdt, buffer=_ATTACHED[name].buf)


def _forget_except(specs):
    keep = {s[0] for s in specs.values() if s is not None}
    for name in list(_ATTACHED):
        if name not in keep:
            _ATTACHED.pop(name).close()


def f64(spec, lo, hi):
    """Leading-axis slice [lo, hi) of a shared tensor as float64 (bf16 exactly)."""
    a = _raw(spec)[lo:hi]
    if spec[2] == "bf16":
        return (a.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _tdt(name):
    return torch.bfloat16 if name == "bf16" else torch.float32


def _work(args):
    op, specs, lo, hi, prm = args
    _forget_except(specs)
    import oracle as O
    from parity import grad_stats, wtv_flips
    out = {"lo": lo, "hi": hi}
    if op in ("wtv", "eal"):
        zd, zt = f64(specs["zd"], lo, hi), f64(specs["zt"], lo, hi)
        n = hi - lo
        N, Td = prm["N"], prm["Td"]
        gs = n / N
        if op == "wtv":
            o = O.wtv_loss(zd, zt, Td, prm["Tt"], grad_scale=gs)
            out.update(a=o["a"], E=o["E"])
        else:
            o = O.eal_loss(zd, zt, Td, grad_scale=gs)
            out.update(a=o["a"], E=o["E"], xstar=o["xstar"])
            out["tie_rows"] = int(np.sum(np.sum(zt == zt.max(-1, keepdims=True), -1) > 1))
        if specs.get("grad") is not None:
            G = f64(specs["grad"], lo, hi)
            coef = -O.expected_length_grad(o["a"]) / N / Td
            if op == "eal":
                coef = coef * o["a"]
            extra = None
            if op == "wtv":
                extra, near = wtv_flips(zd, zt, Td, prm["Tt"], coef)
            out["grad"] = grad_stats(G, o["grad"], coef, _tdt(specs["zd"][2]), _tdt(specs["grad"][2]),
                                     extra_tol=extra)
            if extra is not None:
                out["grad"]["near_elems"] = int(near.sum())
    elif op == "combined":
        # windows layout: windows [lo, hi) of K rows; window and row counts
        # scale alike, so the chunk's gradient times n/N is the full one
        K = prm["K"]
        zd, zt = f64(specs["zd"], lo, hi), f64(specs["zt"], lo, hi)
        n = hi - lo
        o = O.combined_loss(zd, zt, prm["Td"], prm["Tt"], prm["w"], O.LAYOUT_WINDOWS, n, K, K,
                            grad_scale=n / prm["N"])
        out.update(a_tv=o["a_tv"], a_eal=o["a_eal"], kl=o["kl"], xstar=o["xstar"], E_tv=o["E_tv"],
                   E_eal=o["E_eal"])
        if specs.get("grad") is not None:
            G = f64(specs["grad"], lo, hi)
            coef = np.abs(o["coef_tv"]) + np.abs(o["coef_eal"]) + np.abs(o["coef_kl"])
            extra = None
            if prm["w"][0] or prm["w"][3]:
                extra, near = wtv_flips(zd.reshape(-1, zd.shape[-1]), zt.reshape(-1, zt.shape[-1]), prm["Td"],
                                        prm["Tt"], o["coef_tv"])
            out["grad"] = grad_stats(G.reshape(-1, G.shape[-1]), o["grad"], coef, _tdt(specs["zd"][2]),
                                     _tdt(specs["grad"][2]), extra_tol=extra)
            if extra is not None:
                out["grad"]["near_elems"] = int(near.sum())
    elif op == "seqgrad":
        # rows [lo, hi) of one sequence (flattened row indices): the oracle on
        # the sub-sequence that holds every window containing them, rescaled
        # from the sub-sequence's window and row counts to the full ones
        S, K = prm["S"], prm["K"]
        b = lo // S
        s0 = max(b * S, lo - (K - 1))
        s1 = min((b + 1) * S, hi + (K - 1))
        zd, zt = f64(specs["zd"], s0, s1), f64(specs["zt"], s0, s1)
        L = s1 - s0
        Wsub = max(0, L - K + 1)
        g = 0.0
        coef = 0.0
        for t, w in enumerate(prm["w"]):
            if w == 0:
                continue
            e = [0.0] * 4
            e[t] = 1.0
            o = O.combined_loss(zd, zt, prm["Td"], prm["Tt"], e, O.LAYOUT_SEQUENCES, 1, L, K)
            f = (L / prm["R"]) if t == 2 else (Wsub / prm["W"])
            g = g + w * f * o["grad"][lo - s0:hi - s0]
            c = (o["coef_tv"], o["coef_eal"], o["coef_kl"], o["coef_tv"])[t][lo - s0:hi - s0]
            coef = coef + np.abs(w * f * c)
        G = f64(specs["grad"], lo, hi)
        extra = None
        if prm["w"][0] or prm["w"][3]:
            extra, near = wtv_flips(zd[lo - s0:hi - s0], zt[lo - s0:hi - s0], prm["Td"], prm["Tt"], coef)
        out["grad"] = grad_stats(G, g, coef, _tdt(specs["zd"][2]), _tdt(specs["grad"][2]),
                                 extra_tol=extra)
        if extra is not None:
            out["grad"]["near_elems"] = int(near.sum())
    elif op == "sim":
        zd, zt = f64(specs["zd"], lo, hi), f64(specs["zt"], lo, hi)
        u1, u2 = f64(specs["u1"], lo, hi), f64(specs["u2"], lo, hi)
        o = O.sim_accept_grpo(zd, zt, prm["T"], u1, u2)
        out.update(token=o["token"], accept=o["accept"], reward=o["reward"], advantage=o["advantage"],
                   flag=O.sim_near_threshold(zd, zt, prm["T"], u1, u2))
    elif op == "grpo":
        m, K = prm["m"], prm["K"]
        n = hi - lo
        zth, zrf, ztg = (f64(specs[k], lo, hi) for k in ("zth", "zrf", "ztg"))
        o = O.grpo_loss(zth, zrf, ztg, prm["T"], O.LAYOUT_WINDOWS, n, m * K, m, K, eps_clip=prm["eps_clip"],
                        grad_scale=n / prm["n_groups"])
        out.update(tau_theta=o["tau_theta"], tau_ref=o["tau_ref"], log_rho=o["log_rho"], adv=o["adv"],
                   group_loss=o["group_loss"])
        # windows whose ratio sits within 1e-4 of a clip bound may legitimately
        # switch derivative: their rows are left out of the elementwise check
        near = (np.abs(o["rho"] - (1 - prm["eps_clip"])) <= 1e-4) | (np.abs(o["rho"] - (1 + prm["eps_clip"])) <= 1e-4)
        rows = np.repeat(near.reshape(-1), K)
        out["clip_near_windows"] = int(near.sum())
        G = f64(specs["grad"], lo, hi)
        coef = np.repeat(np.abs(o["coef"]).reshape(-1) / K, K) * (n / prm["n_groups"]) / prm["T"]
        out["grad"] = grad_stats(G.reshape(-1, G.shape[-1]), o["grad"], coef, _tdt(specs["zth"][2]),
                                 _tdt(specs["grad"][2]), exclude_rows=rows)
    else:
        raise ValueError(op)
    return out


def run(pool, op, specs, n, step, prm):
    """The op over [0, n) in chunks of `step`, in order."""
    tasks = [(op, specs, lo, min(n, lo + step), prm) for lo in range(0, n, step)]
    return pool.map(_work, tasks, chunksize=1)


def cat(res, key):
    return np.concatenate([r[key] for r in res], axis=0)


def merge_grad(res) -> dict:
    tot = {"max_abs": 0.0, "gmax": 0.0, "rows_checked": 0, "rows_excluded": 0, "elems_checked": 0,
           "elems_excluded": 0, "bad": 0, "rows_widened": 0, "near_elems": 0, "max_widening_over_c": 0.0}
    for r in res:
        g = r.get("grad")
        if not g:
            continue
        for k in ("rows_checked", "rows_excluded", "elems_checked", "elems_excluded", "bad", "rows_widened",
                  "near_elems"):
            tot[k] += g.get(k, 0)
        tot["max_widening_over_c"] = max(tot["max_widening_over_c"], g.get("max_widening_over_c", 0.0))
        tot["max_abs"] = max(tot["max_abs"], g["max_abs"])
        tot["gmax"] = max(tot["gmax"], g["gmax"])
    return tot


def report(name: str, stats: dict) -> None:
    """Print the statistics and append them to $AAL_PARITY_REPORT (JSON lines)."""
    line = json.dumps({"case": name, **stats}, default=float)
    print(line)
    path = os.environ.get("AAL_PARITY_REPORT")
    if path:
        with open(path, "a") as f:
            f.write(line + "\n")
