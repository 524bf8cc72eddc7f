"""Benchmark: fused WTV loss forward + backward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2]

A step is one aal_wtv_fwd_bwd call (per-row softmaxes of both logit sets,
sum min(p, q), window prefix products, loss, and dloss/dz_draft) over the
whole workload, inputs resident in HBM.  The default workload is the WTV
configuration at V=128256 bf16: N=2048 windows x K=7 positions, T=1.0 for
both distributions, bf16 gradient.

Prints ONE JSON line.  `value` is logit rows/s; `roofline` prices the step
against HBM bandwidth with the algorithmic byte count (both logit tensors read
once, the gradient written once: (2 s_in + s_grad) V bytes per row) over the
average step time measured with HIP events on the stream the kernels run on.
Secondary measurements (EAL on the same inputs; the combined-objective entry
point on the same rows read as sliding-window sequences and with the paper's
KL-anchored objectives; the simulated-acceptance reward on the GRPO workload)
are reported under "also".  `cpu_baseline` times
the fp64 oracle on a bounded sample of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import json
import multiprocessing as mp
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
SIMDS = 1024          # 256 CUs x 4 SIMDs
CLOCK_HZ = 2.4e9      # MI355X peak engine clock
HOST_CPU_SHARE = 16
PMC_PROFILE = os.path.join(ROOT, "profiles", "resident_wtv_c2_pmc.txt")
KERNEL_SOURCES = ["paper_2609_24150_amd/csrc/aal_resident.hip", "paper_2609_24150_amd/csrc/aal_resident_common.h",
                  "paper_2609_24150_amd/csrc/aal_device.h", "paper_2609_24150_amd/csrc/aal_internal.h"]
WORKLOAD_TEXT = {
    "c2": "WTV fwd+bwd: N=2048 windows x K=7 x V=128256, bf16 logits, bf16 grad, T=1.0/1.0",
    "c4": "WTV fwd+bwd: N=16384 windows x K=16 x V=32000, fp32 logits, fp32 grad, T=0.5/0.5",
}


# ------------------------------------------------------------- CPU baseline
def _cpu_worker(args):
    wid, recipe, K, V, nwin, budget_s = args
    import numpy as np
    import torch

    import oracle as O
    from paper_2609_24150_amd.inputs import CONFIGS, make_logits
    cfg = CONFIGS[recipe]
    torch.set_num_threads(1)
    zd, zt = make_logits(cfg["recipe"], (nwin, K, V), cfg["dtype"], seed=1000 + wid, device="cpu")
    zd = zd.to(torch.float64).numpy()
    zt = zt.to(torch.float64).numpy()
    Td, Tt = cfg["temp_draft"], cfg["temp_target"]
    n = 0
    t0 = time.perf_counter()
    while True:
        o = O.wtv_loss(zd, zt, Td, Tt)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            # the last evaluation, kept for the parity sample of the GPU results
            res = {"loss": float(o["loss"]), "E": np.asarray(o["E"]), "a": np.asarray(o["a"]),
                   "grad": np.asarray(o["grad"], dtype=np.float32)}
            return n * nwin * K, el, res


def cpu_baseline(workload: str, budget_s: float = 12.0) -> dict:
    from paper_2609_24150_amd.inputs import CONFIGS
    cfg = CONFIGS[workload]
    K, V = cfg["K"], cfg["V"]
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    # one GPU's share of the host is 16 CPUs, whatever the affinity mask shows
    workers = max(1, min(HOST_CPU_SHARE, cores))
    nwin = 2
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(workers) as pool:
        res = pool.map(_cpu_worker, [(w, workload, K, V, nwin, budget_s) for w in range(workers)])
    wall = time.perf_counter() - t0
    rows = sum(r[0] for r in res)
    # each worker's rate over its own timed loop, summed: the aggregate rate
    rate = sum(r[0] / r[1] for r in res)
    _ORACLE_SAMPLES[:] = [(1000 + w, nwin, r[2]) for w, r in enumerate(res)]
    return {"value": rate, "unit": "logit rows/s", "cores": workers, "kind": "oracle",
            "sample": f"{workers} processes x {nwin} windows of the workload (K={K}, V={V}), each repeated "
                      f"for ~{budget_s:.0f}s; {rows} rows in {wall:.1f}s wall",
            "rows_per_s_per_core": rate / workers, "affinity_cores": cores,
            "worker_cap": f"{HOST_CPU_SHARE} (the host CPU share of one GPU)", "cpu_model": _cpu_model()}


# (seed, windows, oracle result) of each CPU worker's input: the oracle's own
# results, compared after the timed legs with the library's on the same inputs
_ORACLE_SAMPLES = []


def parity_sample(workload: str) -> dict:
    """The library's WTV call on each CPU worker's seeded windows against the
    oracle's results for them (computed in the CPU leg): the largest relative
    error of the loss and of E, the largest absolute error of the acceptances,
    and the largest gradient error relative to the largest gradient entry.
    Reported, not asserted (the parity tests assert the stated tolerances)."""
    import numpy as np
    import torch

    import paper_2609_24150_amd as A
    from paper_2609_24150_amd.inputs import CONFIGS, make_logits
    cfg = CONFIGS[workload]
    K, V = cfg["K"], cfg["V"]
    worst = {"loss_rel": 0.0, "E_rel": 0.0, "accept_abs": 0.0, "grad_abs_over_max": 0.0}
    n = 0
    for seed, nwin, o in _ORACLE_SAMPLES:
        zd, zt = make_logits(cfg["recipe"], (nwin, K, V), cfg["dtype"], seed=seed, device="cpu")
        r = A.aal_wtv_fwd_bwd(zd.cuda(), zt.cuda(), cfg["temp_draft"], cfg["temp_target"], grad_dtype=cfg["dtype"])
        torch.cuda.synchronize()
        rel = lambda a, b: float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-30)))  # noqa: E731
        worst["loss_rel"] = max(worst["loss_rel"], rel(np.float64(r["loss"].item()), np.float64(o["loss"])))
        worst["E_rel"] = max(worst["E_rel"], rel(r["E"].cpu().double().numpy(), o["E"]))
        worst["accept_abs"] = max(worst["accept_abs"],
                                  float(np.max(np.abs(r["accept"].cpu().double().numpy() - o["a"]))))
        g = r["grad"].cpu().float().numpy()
        worst["grad_abs_over_max"] = max(worst["grad_abs_over_max"],
                                         float(np.max(np.abs(g - o["grad"])) / np.max(np.abs(o["grad"]))))
        n += nwin
        del r, zd, zt
    return {"windows": n, **worst, "inputs": "each CPU worker's seeded windows of the workload"}


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def profile_fields(workload: str) -> dict:
    """Per-launch figures of the fused kernel from the committed rocprofv3
    summary (HBM traffic from FETCH_SIZE / WRITE_SIZE, VALU instruction and
    issue-cycle counts), or {} when that summary does not cover this workload
    or the kernel sources changed since it was taken."""
    import hashlib
    if workload != "c2" or not os.path.exists(PMC_PROFILE):
        return {}
    fields = {}
    for line in open(PMC_PROFILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.split()[0]
    h = hashlib.sha256()
    for src in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if fields.get("kernel_source_sha256") != h.hexdigest():
        return {}
    return fields


def alu_roofline(fields: dict, ms: float, alg_bytes: float):
    """The VALU roofline of the fused kernel: its VALU instructions per launch
    (SQ_INSTS_VALU) over the measured time, against the issue rate of 1024
    SIMDs at 2.4 GHz for this kernel's own instruction mix.  A wave64 VALU
    instruction occupies a 16-lane SIMD for 4 cycles; the counters give the
    mix's average, 4 SQ_ACTIVE_INST_VALU / SQ_INSTS_VALU cycles (v_exp_f32
    takes about 8).  frac is then the fraction of the SIMDs' cycles spent
    issuing VALU work, and floor_ms the time at 100%."""
    if "valu_instructions_per_launch" not in fields:
        return None
    valu = float(fields["valu_instructions_per_launch"])
    cycles = 4.0 * float(fields["valu_active_quad_cycles_per_launch"])
    cpi = cycles / valu
    peak = SIMDS * CLOCK_HZ / cpi
    achieved = valu / (ms * 1e-3)
    floor_s = cycles / SIMDS / CLOCK_HZ
    return {"bound": "alu", "achieved": achieved / 1e9, "peak": peak / 1e9, "unit": "G VALU wave-instructions/s",
            "frac": achieved / peak, "cycles_per_instruction": cpi, "valu_instructions_per_launch": valu,
            "floor_ms": floor_s * 1e3, "hbm_frac_at_alu_floor": alg_bytes / floor_s / 1e9 / HBM_PEAK_GBPS,
            "counters": "profiles/resident_wtv_c2_pmc.txt"}


# ----------------------------------------------------------------- GPU legs
def _progress(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _time_calls(fn, steps, warmup, stream):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        fn()
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps  # ms per call
    _progress(f"timed {steps} calls: {ms:.4f} ms each")
    return ms


def _fail(msg):
    print(f"bench.py: invalid measurement: {msg}", file=sys.stderr)
    sys.exit(3)


def check_outputs(fn, outs, name, e_max=None):
    """The timed calls left their results in `outs`; one more untimed call
    must reproduce them bit for bit (the kernels are deterministic), the loss
    must be finite (a poll time-out of a resident kernel makes it NaN) and
    every per-window expectation must lie in [0, K]."""
    import torch
    torch.cuda.synchronize()
    first = {k: v.clone() for k, v in outs.items() if v is not None}
    fn()
    torch.cuda.synchronize()
    loss = outs["loss"].item() if "loss" in outs else None
    if loss is not None and (loss != loss or abs(loss) == float("inf")):
        _fail(f"{name}: loss is {loss}")
    for k, v in first.items():
        if not torch.equal(v.view(torch.uint8) if v.dtype != torch.uint8 else v,
                           outs[k].view(torch.uint8) if outs[k].dtype != torch.uint8 else outs[k]):
            _fail(f"{name}: output {k} differs between two identical calls")
    if e_max is not None and "E" in outs:
        E = outs["E"]
        if not bool(torch.isfinite(E).all()) or E.min().item() < 0 or E.max().item() > e_max * (1 + 1e-6):
            _fail(f"{name}: E outside [0, {e_max}]")
    return {"loss": loss, "repeat_bitwise_equal": True}


def ceilings(dev, nbytes=1 << 32):
    """Practical HBM ceilings on this GPU from plain device kernels (torch's
    copy, a two-input elementwise add, a full-tensor sum, and the library's
    streaming probe for each traffic mix of the loss kernels), each timed with
    HIP events over 10 launches after 3 warm-up launches."""
    import torch
    n = nbytes // 2
    a = torch.ones(n, dtype=torch.bfloat16, device=dev)
    b = torch.ones(n, dtype=torch.bfloat16, device=dev)
    c = torch.empty(n, dtype=torch.bfloat16, device=dev)
    st = torch.cuda.current_stream(dev)
    legs = {"read (sum of one bf16 tensor)": (lambda: torch.sum(a, dtype=torch.float32), nbytes),
            "copy (1 read, 1 write)": (lambda: c.copy_(a), 2 * nbytes),
            "2 reads, 1 write (a + b)": (lambda: torch.add(a, b, out=c), 3 * nbytes)}
    # the library's streaming probe: the loss kernels' own access (16-byte nontemporal loads and
    # stores) for each traffic mix the kernels have
    import paper_2609_24150_amd as A
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    d = torch.ones(n, dtype=torch.bfloat16, device=dev)
    legs.update({
        "probe: 1 read": (lambda: A.aal_stream_probe([a], flag=flag), nbytes),
        "probe: 3 reads (the GRPO row pass's mix)": (lambda: A.aal_stream_probe([a, b, d], flag=flag), 3 * nbytes),
        "probe: 1 read, 1 write (the GRPO gradient pass's mix)": (lambda: A.aal_stream_probe([a], c), 2 * nbytes),
        "probe: 2 reads, 1 write (the fused losses' mix)": (lambda: A.aal_stream_probe([a, b], c), 3 * nbytes),
    })
    res = {}
    for name, (fn, by) in legs.items():
        ms = _time_calls(fn, 10, 3, st)
        res[name] = {"GBps": by / (ms * 1e-3) / 1e9, "frac_of_peak": by / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                     "bytes": by}
    torch.cuda.synchronize()
    if flag.item() != 0:
        _fail("the streaming probe saw a word it should not have")
    del a, b, c, d
    _free_gpu(torch)
    return res


def loss_call(op, inp, grad_dtype, flags=0, temp_draft=None):
    """A zero-allocation closure over the C entry point with preallocated outputs."""
    import torch

    import paper_2609_24150_amd as A
    from paper_2609_24150_amd import _lib
    zd, zt = inp["z_draft"], inp["z_target"]
    cfg = inp["cfg"]
    N, K, V = zd.shape
    dev = zd.device
    loss = torch.empty(1, device=dev)
    E = torch.empty(N, device=dev)
    acc = torch.empty(N, K, device=dev)
    grad = torch.empty(N, K, V, dtype=grad_dtype, device=dev)
    ws = A.workspace(N * K, N, dev)
    L = _lib.lib()
    stream = torch.cuda.current_stream(dev)
    dcode = _lib.AAL_BF16 if zd.dtype == torch.bfloat16 else _lib.AAL_F32
    gcode = _lib.AAL_BF16 if grad_dtype == torch.bfloat16 else _lib.AAL_F32
    if op == "wtv":
        if "wtv_temp" in cfg:  # a workload that runs both losses states one WTV temperature for both
            Td = Tt = cfg["wtv_temp"]
        else:
            Td, Tt = cfg.get("temp_draft", 1.0), cfg.get("temp_target", 1.0)

        def fn():
            head = (zd.data_ptr(), zt.data_ptr(), dcode, N, K, V, Td, Tt, loss.data_ptr(), E.data_ptr(),
                    acc.data_ptr(), grad.data_ptr(), gcode, None)
            if flags:
                st = L.aal_wtv_fwd_bwd_ex(*head, flags, ws.data_ptr(), ws.numel(), stream.cuda_stream)
            else:
                st = L.aal_wtv_fwd_bwd(*head, ws.data_ptr(), ws.numel(), stream.cuda_stream)
            _lib.check(st, "aal_wtv_fwd_bwd")
    else:
        xs = torch.empty(N, K, dtype=torch.int32, device=dev)
        Td = cfg.get("temp_draft", 1.0) if temp_draft is None else temp_draft

        def fn():
            head = (zd.data_ptr(), zt.data_ptr(), dcode, N, K, V, Td, loss.data_ptr(), E.data_ptr(),
                    acc.data_ptr(), xs.data_ptr(), grad.data_ptr(), gcode, None)
            if flags:
                st = L.aal_eal_fwd_bwd_ex(*head, flags, ws.data_ptr(), ws.numel(), stream.cuda_stream)
            else:
                st = L.aal_eal_fwd_bwd(*head, ws.data_ptr(), ws.numel(), stream.cuda_stream)
            _lib.check(st, "aal_eal_fwd_bwd")
        return fn, stream, {"loss": loss, "E": E, "accept": acc, "xstar": xs, "grad": grad}
    return fn, stream, {"loss": loss, "E": E, "accept": acc, "grad": grad}


def sim_call(inp):
    import torch

    import paper_2609_24150_amd as A
    from paper_2609_24150_amd import _lib
    zd, zt, u1, u2 = inp["z_draft"], inp["z_target"], inp["u1"], inp["u2"]
    P, G, K, V = zd.shape
    dev = zd.device
    tok = torch.empty(P, G, K, dtype=torch.int32, device=dev)
    rew = torch.empty(P, G, dtype=torch.int32, device=dev)
    adv = torch.empty(P, G, device=dev)
    ws = A.workspace(P * G * K, P * G, dev)
    L = _lib.lib()
    stream = torch.cuda.current_stream(dev)
    dcode = _lib.AAL_BF16 if zd.dtype == torch.bfloat16 else _lib.AAL_F32

    def fn():
        st = L.aal_sim_accept_grpo(zd.data_ptr(), zt.data_ptr(), dcode, P, G, K, V, 1.0, u1.data_ptr(),
                                   u2.data_ptr(), tok.data_ptr(), rew.data_ptr(), adv.data_ptr(),
                                   1e-6, 0, 0.0, ws.data_ptr(), ws.numel(), stream.cuda_stream)
        _lib.check(st, "aal_sim_accept_grpo")
    return fn, stream, {"token": tok, "reward": rew, "advantage": adv}


def general_call(zd, zt, layout, B, S, K, weights, grad_dtype):
    """A zero-allocation closure over aal_loss_fwd_bwd (combined objectives)."""
    import torch

    from paper_2609_24150_amd import _lib
    V = zd.shape[-1]
    dev = zd.device
    R = B * S
    W = B if layout == _lib.AAL_LAYOUT_WINDOWS else B * max(0, S - K + 1)
    L = _lib.lib()
    loss = torch.empty(1, device=dev)
    terms = torch.empty(4, device=dev)
    grad = torch.empty(R, V, dtype=grad_dtype, device=dev)
    ws = torch.empty(L.aal_loss_workspace_bytes(layout, B, S, K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    dcode = _lib.AAL_BF16 if zd.dtype == torch.bfloat16 else _lib.AAL_F32
    gcode = _lib.AAL_BF16 if grad_dtype == torch.bfloat16 else _lib.AAL_F32
    w = _lib.LossWeights(*weights)

    def fn():
        st = L.aal_loss_fwd_bwd(zd.data_ptr(), zt.data_ptr(), None, dcode, layout, B, S, K, V, 1.0, 1.0, w,
                                loss.data_ptr(), terms.data_ptr(), None, None, None, None, None, grad.data_ptr(),
                                gcode, None, 0, ws.data_ptr(), ws.numel(), stream.cuda_stream)
        _lib.check(st, "aal_loss_fwd_bwd")
    return fn, stream, R, W, {"loss": loss, "terms": terms, "grad": grad}


def vp_call(zd_s, zt_s, v0, V, R, N, K, mode, grad_dtype):
    """A zero-allocation closure over one rank's five vocabulary-parallel calls
    on its [rows, V_slice] slice.  The rank's own records copied into every
    rank's place stand in for the two all-gathers' outputs."""
    import torch

    from paper_2609_24150_amd import _lib
    rows, vs = zd_s.shape
    dev = zd_s.device
    L = _lib.lib()
    stream = torch.cuda.current_stream(dev)
    parts = torch.empty(R, rows, _lib.VP_PART_BYTES, dtype=torch.uint8, device=dev)
    row = torch.empty(rows, _lib.VP_ROW_BYTES, dtype=torch.uint8, device=dev)
    acc = torch.empty(R, rows, _lib.VP_ACC_BYTES, dtype=torch.uint8, device=dev)
    loss = torch.empty(1, device=dev)
    E = torch.empty(N, device=dev)
    grad = torch.empty(rows, vs, dtype=grad_dtype, device=dev)
    dcode = _lib.AAL_BF16 if zd_s.dtype == torch.bfloat16 else _lib.AAL_F32
    gcode = _lib.AAL_BF16 if grad_dtype == torch.bfloat16 else _lib.AAL_F32
    wtv = mode == _lib.AAL_VP_WTV
    s = stream.cuda_stream

    def fn():
        _lib.check(L.aal_vp_row_partials(zd_s.data_ptr(), zt_s.data_ptr(), None, dcode, rows, vs, v0, V, mode,
                                         1.0, 1.0, parts[0].data_ptr(), s), "aal_vp_row_partials")
        parts[1:].copy_(parts[0].expand(R - 1, -1, -1))
        _lib.check(L.aal_vp_merge_rows(parts.data_ptr(), R, rows, mode, 1.0, 1.0, row.data_ptr(), s),
                   "aal_vp_merge_rows")
        if wtv:
            _lib.check(L.aal_vp_accept_partials(zd_s.data_ptr(), zt_s.data_ptr(), dcode, rows, vs, 1.0, 1.0,
                                                row.data_ptr(), acc[0].data_ptr(), s), "aal_vp_accept_partials")
            acc[1:].copy_(acc[0].expand(R - 1, -1, -1))
        _lib.check(L.aal_vp_window_scan(row.data_ptr(), acc.data_ptr() if wtv else None, R, N, K, mode, 1.0, None,
                                        loss.data_ptr(), E.data_ptr(), None, None, s), "aal_vp_window_scan")
        _lib.check(L.aal_vp_grad(zd_s.data_ptr(), zt_s.data_ptr() if wtv else None, dcode, rows, vs, v0, mode,
                                 1.0, 1.0, row.data_ptr(), grad.data_ptr(), gcode, s), "aal_vp_grad")
    return fn, stream, {"loss": loss, "E": E, "grad": grad}


def grpo_call(zth, zref, zt, m, K, grad_dtype):
    """A zero-allocation closure over aal_grpo_fwd_bwd (windows layout, groups of m windows)."""
    import torch

    from paper_2609_24150_amd import _lib
    B, S, V = zth.shape
    dev = zth.device
    L = _lib.lib()
    loss = torch.empty(1, device=dev)
    tt = torch.empty(B, m, dtype=torch.int32, device=dev)
    tr = torch.empty_like(tt)
    adv = torch.empty(B, m, device=dev)
    lrho = torch.empty_like(adv)
    grad = torch.empty(B, S, V, dtype=grad_dtype, device=dev)
    ws = torch.empty(L.aal_grpo_workspace_bytes(_lib.AAL_LAYOUT_WINDOWS, B, S, 1, m, K), dtype=torch.uint8,
                     device=dev)
    stream = torch.cuda.current_stream(dev)
    dcode = _lib.AAL_BF16 if zth.dtype == torch.bfloat16 else _lib.AAL_F32
    gcode = _lib.AAL_BF16 if grad_dtype == torch.bfloat16 else _lib.AAL_F32
    prm = _lib.GrpoParams(1e-6, 0.0, 0.2, 0.0, float("inf"))

    def fn():
        st = L.aal_grpo_fwd_bwd(zth.data_ptr(), zref.data_ptr(), zt.data_ptr(), None, dcode,
                                _lib.AAL_LAYOUT_WINDOWS, B, S, 1, m, K, V, None, 1.0, prm, loss.data_ptr(),
                                tt.data_ptr(), tr.data_ptr(), adv.data_ptr(), lrho.data_ptr(), grad.data_ptr(),
                                gcode, None, ws.data_ptr(), ws.numel(), stream.cuda_stream)
        _lib.check(st, "aal_grpo_fwd_bwd")
    return fn, stream, {"loss": loss, "tau_theta": tt, "advantage": adv, "grad": grad}


def _free_gpu(torch):
    import gc
    gc.collect()
    torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-also", action="store_true", help="skip the secondary EAL and simulation legs")
    ap.add_argument("--flags", type=int, default=0, help="AAL_FLAG_* bits for the timed call")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run one device copy of 4 GiB (a reference kernel of known "
                         "traffic for hardware-counter runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    # The CPU leg runs first, in forked workers, before this process touches the GPU.
    cpu = None if args.no_cpu_baseline else cpu_baseline(args.workload)

    import torch

    from paper_2609_24150_amd.inputs import CONFIGS, make_config
    cfg = CONFIGS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    inp = make_config(args.workload, seed=0, device=dev)
    N, K, V = cfg["N"], cfg["K"], cfg["V"]
    rows = N * K
    s_in = 2 if cfg["dtype"] == torch.bfloat16 else 4
    gdt = cfg["dtype"]
    s_g = s_in
    fn, stream, outs = loss_call("wtv", inp, gdt, args.flags)
    ms = _time_calls(fn, args.steps, args.warmup, stream)
    valid = check_outputs(fn, outs, "wtv", e_max=K)
    del outs
    alg_bytes = rows * (2 * s_in + s_g) * V
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    prof = profile_fields(args.workload)
    traffic = float(prof["traffic_bytes_per_launch"]) if "traffic_bytes_per_launch" in prof else None
    out = {
        "metric": "EAL/WTV fwd+bwd logit rows/s + % of HBM peak, V=128256 bf16, 1 GPU",
        "value": rows / (ms * 1e-3),
        "unit": "logit rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg["dtype"] == torch.bfloat16 else "f32",
        "data": "synthetic (seeded logits with the workload's distribution)",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "N": N, "K": K, "V": V,
                   "windows_per_s": N / (ms * 1e-3)},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "algorithmic_bytes": alg_bytes,
                     "kernel": "k_resident (timed: the whole aal_wtv_fwd_bwd call, i.e. k_resident plus "
                               "two microsecond-scale kernels: slot clear, loss reduction)",
                     "alu": alu_roofline(prof, ms, alg_bytes)},
        "cpu_baseline": cpu,
        "validation": valid,
        "practical_ceilings": ceilings(dev),
    }
    if args.copy_calibration:
        # the shape of the ceiling legs' copy (2^31 bf16 elements): a byte copy of exactly 2^32
        # elements has been seen to read and write several times its size in the counters
        src = torch.empty(1 << 31, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = {"read": 1 << 32, "write": 1 << 32}
        del src, dst
        torch.cuda.empty_cache()
    if not args.no_also:
        also = {}
        fn_e, st_e, o_e = loss_call("eal", inp, gdt, args.flags)
        ms_e = _time_calls(fn_e, args.steps, args.warmup, st_e)
        check_outputs(fn_e, o_e, "eal", e_max=K)
        del o_e
        also["eal_same_inputs"] = {"ms": ms_e, "rows_per_s": rows / (ms_e * 1e-3),
                                   "windows_per_s": N / (ms_e * 1e-3),
                                   "alg_GBps": rows * (2 * s_in + s_g) * V / (ms_e * 1e-3) / 1e9}
        if args.workload == "c2":
            from paper_2609_24150_amd import _lib
            zd, zt = inp["z_draft"], inp["z_target"]
            # the same rows read as 7 sequences of 2048 positions, windows sliding by one
            legs = [("wtv_sliding_7x2048", _lib.AAL_LAYOUT_SEQUENCES, 7, 2048, (1.0, 0.0, 0.0, 0.0)),
                    ("kl_plus_0.1eal_c2", _lib.AAL_LAYOUT_WINDOWS, N, K, (0.0, 0.1, 1.0, 0.0)),
                    ("kl_plus_0.1eal_sliding_7x2048", _lib.AAL_LAYOUT_SEQUENCES, 7, 2048, (0.0, 0.1, 1.0, 0.0)),
                    ("kl_plus_tv_c2", _lib.AAL_LAYOUT_WINDOWS, N, K, (0.0, 0.0, 1.0, 1.0))]
            for name, layout, B_, S_, wts in legs:
                fn_g, st_g, R_, W_, o_g = general_call(zd, zt, layout, B_, S_, K, wts, gdt)
                ms_g = _time_calls(fn_g, args.steps, args.warmup, st_g)
                check_outputs(fn_g, o_g, name)
                del fn_g, o_g
                also[name] = {"ms": ms_g, "rows_per_s": R_ / (ms_g * 1e-3), "windows_per_s": W_ / (ms_g * 1e-3),
                              "alg_GBps": R_ * (2 * s_in + s_g) * V / (ms_g * 1e-3) / 1e9,
                              "entry": "aal_loss_fwd_bwd", "weights(wtv,eal,kl,tv)": wts}
            # GRPO over the same rows: 256 groups of m=8 windows; the reference
            # policy's logits are the draft's plus seeded noise
            m_ = 8
            g_ = torch.Generator(device=dev).manual_seed(11)
            zref = (zd.float() + 0.5 * torch.randn(zd.shape, generator=g_, device=dev)).to(zd.dtype)
            shp = (N // m_, m_ * K, V)
            fn_r, st_r, o_r = grpo_call(zd.view(shp), zref.view(shp), zt.view(shp), m_, K, gdt)
            ms_r = _time_calls(fn_r, args.steps, args.warmup, st_r)
            check_outputs(fn_r, o_r, "grpo")
            del fn_r, o_r
            also["grpo_c2_m8"] = {"ms": ms_r, "rows_per_s": rows / (ms_r * 1e-3), "windows_per_s": N / (ms_r * 1e-3),
                                  "alg_GBps": rows * (3 * s_in + s_g) * V / (ms_r * 1e-3) / 1e9,
                                  "entry": "aal_grpo_fwd_bwd", "groups": N // m_, "m": m_}
            # one rank's share of the same rows with the vocabulary split over 8
            # ranks (a vocabulary-parallel LM head): slice 3 of 8
            R_vp = 8
            vs = V // R_vp
            zd_s = zd.view(rows, V)[:, 3 * vs:4 * vs].contiguous()
            zt_s = zt.view(rows, V)[:, 3 * vs:4 * vs].contiguous()
            for name, mode in (("vp_wtv_c2_rank_share_8", _lib.AAL_VP_WTV), ("vp_eal_c2_rank_share_8", _lib.AAL_VP_EAL)):
                fn_v, st_v, o_v = vp_call(zd_s, zt_s, 3 * vs, V, R_vp, N, K, mode, gdt)
                ms_v = _time_calls(fn_v, args.steps, args.warmup, st_v)
                check_outputs(fn_v, o_v, name, e_max=K)
                del fn_v, o_v
                also[name] = {"ms": ms_v, "rows_per_s": rows / (ms_v * 1e-3),
                              "alg_GBps": rows * (2 * s_in + s_g) * vs / (ms_v * 1e-3) / 1e9,
                              "entry": "aal_vp_*", "shape": f"{rows}x{vs} (V={V} over {R_vp} ranks)"}
            del zd_s, zt_s
            del zd, zt, zref
        del inp
        torch.cuda.empty_cache()
        sim = make_config("c5", seed=0, device=dev)
        c5 = CONFIGS["c5"]
        rows5 = c5["P"] * c5["G"] * c5["K"]
        fn_s, st_s, o_s = sim_call(sim)
        ms_s = _time_calls(fn_s, args.steps, args.warmup, st_s)
        check_outputs(fn_s, o_s, "sim")
        rw = o_s["reward"]
        if rw.min().item() < 0 or rw.max().item() > c5["K"]:
            _fail("sim: reward outside [0, K]")
        del o_s
        also["sim_grpo_c5"] = {"ms": ms_s, "rows_per_s": rows5 / (ms_s * 1e-3),
                               "windows_per_s": c5["P"] * c5["G"] / (ms_s * 1e-3),
                               "alg_GBps": rows5 * 2 * 2 * c5["V"] / (ms_s * 1e-3) / 1e9}
        del fn_s, st_s
        if args.workload == "c2":
            # every other loss workload, each timed the same way (parity cases in the tests)
            # (c3 EAL also at T_d = 0.7: the workload states no draft temperature
            # for its greedy leg, so both readings are measured)
            prev = None
            for name, op, td_c in (("c1_eal_fp32", "eal", None), ("c3_eal_bf16", "eal", None),
                                   ("c3_eal_bf16_Td0.7", "eal", 0.7), ("c3_wtv_bf16_T0.7", "wtv", None),
                                   ("c4_wtv_fp32_T0.5", "wtv", None)):
                wl = name[:2]
                c = CONFIGS[wl]
                if wl != prev:
                    del sim
                    _free_gpu(torch)
                    sim = make_config(wl, seed=0, device=dev)
                    prev = wl
                fn_c, st_c, o_c = loss_call(op, sim, c["dtype"], args.flags, temp_draft=td_c)
                ms_c = _time_calls(fn_c, args.steps, args.warmup, st_c)
                check_outputs(fn_c, o_c, name, e_max=c["K"])
                del o_c
                r_c = c["N"] * c["K"]
                s_c = 2 if c["dtype"] == torch.bfloat16 else 4
                gbps = r_c * 3 * s_c * c["V"] / (ms_c * 1e-3) / 1e9
                also[name] = {"ms": ms_c, "rows_per_s": r_c / (ms_c * 1e-3), "windows_per_s": c["N"] / (ms_c * 1e-3),
                              "alg_GBps": gbps, "frac": gbps / HBM_PEAK_GBPS,
                              "shape": f"{c['N']}x{c['K']}x{c['V']}"}
                del fn_c
        for name, leg in also.items():
            if "alg_GBps" in leg and "frac" not in leg:
                leg["frac"] = leg["alg_GBps"] / HBM_PEAK_GBPS
        out["also"] = also
    if cpu is not None and _ORACLE_SAMPLES:
        _progress("parity sample against the CPU leg's oracle results")
        cpu["parity_sample"] = parity_sample(args.workload)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
