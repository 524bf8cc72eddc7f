"""GPU parity of the vocabulary-parallel entry points against the fp64 oracle.

One GPU plays every rank: the vocabulary is cut into contiguous slices, each
slice is copied into arrays of its own (as a rank of a vocabulary-split LM
head holds it), the per-slice records are stacked in rank order (what an
all-gather would deliver), and the slices of the gradient are concatenated
again.  The assembled loss, windows, acceptances, greedy tokens and gradient
must meet the tolerances of the fused calls (tests/parity.py) against the
oracle's full-vocabulary definitions."""
import numpy as np
import pytest
import torch

import oracle as O
from parity import check_grad, eal_coef, host64, loss_tol, rel_err, wtv_coef, wtv_flips

pytestmark = pytest.mark.gpu

BF16, F32 = torch.bfloat16, torch.float32


@pytest.fixture(scope="module")
def A():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_24150_amd as lib
    return lib


@pytest.fixture(scope="module")
def dev(A):
    return torch.device("cuda:0")


def _inputs(recipe, shape, dtype, seed, dev):
    from paper_2609_24150_amd.inputs import make_logits
    zd, zt = make_logits(recipe, shape, dtype, seed=seed, device="cpu")
    return zd.to(dev), zt.to(dev)


def _bounds(V, widths):
    assert sum(widths) == V
    v0 = np.concatenate([[0], np.cumsum(widths)[:-1]])
    return [(int(a), int(w)) for a, w in zip(v0, widths)]


def run_vp(A, zd, zt, mode, widths, Td=1.0, Tt=1.0, gdtype=None, scale=None, labels=None):
    """The five steps over slices of the given widths; returns the fused calls' outputs."""
    N, K, V = zd.shape
    rows = N * K
    sl = [(v0, w, zd.reshape(rows, V)[:, v0:v0 + w].contiguous(), zt.reshape(rows, V)[:, v0:v0 + w].contiguous())
          for v0, w in _bounds(V, widths)]
    parts = torch.stack([A.aal_vp_row_partials(d, None if labels is not None else t, v0, mode, Td, Tt, V_total=V,
                                               labels=labels)
                         for v0, w, d, t in sl])
    row = A.aal_vp_merge_rows(parts, mode, Td, Tt)
    acc = None
    if mode == A.AAL_VP_WTV:
        acc = torch.stack([A.aal_vp_accept_partials(d, t, row, Td, Tt) for v0, w, d, t in sl])
    gs = None if scale is None else torch.tensor([scale], device=zd.device)
    r = A.aal_vp_window_scan(row, acc, N, K, mode, Td, grad_scale=gs)
    g = [A.aal_vp_grad(d, t if mode == A.AAL_VP_WTV else None, row, v0, mode, Td, Tt, grad_dtype=gdtype)
         for v0, w, d, t in sl]
    r["grad"] = torch.cat(g, dim=1).reshape(N, K, V)
    r["row"] = row
    torch.cuda.synchronize()
    return r


def check_eal(A, zd, zt, widths, T=1.0, gdtype=None, scale=None):
    r = run_vp(A, zd, zt, A.AAL_VP_EAL, widths, T, 1.0, gdtype, scale)
    s = 1.0 if scale is None else scale
    o = O.eal_loss(host64(zd), host64(zt), T, grad_scale=s)
    assert np.array_equal(r["xstar"].cpu().numpy(), o["xstar"]), "greedy tokens differ"
    tol = loss_tol(zd.dtype)
    assert rel_err(r["loss"].item(), o["loss"]) <= tol
    assert rel_err(host64(r["E"]), o["E"]) <= tol
    np.testing.assert_allclose(host64(r["accept"]), o["a"], rtol=tol, atol=1e-7)
    coef = eal_coef(o, zd.shape[0], T, s)
    check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, gdtype or zd.dtype)
    return r


def check_wtv(A, zd, zt, widths, Td=1.0, Tt=1.0, gdtype=None, scale=None):
    r = run_vp(A, zd, zt, A.AAL_VP_WTV, widths, Td, Tt, gdtype, scale)
    s = 1.0 if scale is None else scale
    zd64, zt64 = host64(zd), host64(zt)
    o = O.wtv_loss(zd64, zt64, Td, Tt, grad_scale=s)
    tol = loss_tol(zd.dtype)
    assert rel_err(r["loss"].item(), o["loss"]) <= tol
    assert rel_err(host64(r["E"]), o["E"]) <= tol
    np.testing.assert_allclose(host64(r["accept"]), o["a"], rtol=tol, atol=1e-6 if zd.dtype == F32 else 1e-4)
    coef = wtv_coef(o, zd.shape[0], Td, s)
    extra, near = wtv_flips(zd64, zt64, Td, Tt, coef)
    check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, gdtype or zd.dtype, extra_tol=extra)
    return r


# (dtype, gdtype, N, K, slice widths): one slice (the whole vocabulary), equal
# vector-multiple slices, ragged slices that leave the 16-byte vector path,
# slices narrower than a vector, slices spanning several 256-thread tiles with
# ragged tails, and one rank's share of 128,256- and 151,936-entry vocabularies over 8 ranks.
CASES = [
    (BF16, BF16, 3, 4, [1000]),
    (BF16, BF16, 3, 7, [1024] * 4),
    (BF16, F32, 2, 5, [300, 301, 399]),
    (F32, F32, 3, 3, [1, 2, 5, 992]),
    (F32, BF16, 2, 4, [2500, 1599]),
    (BF16, BF16, 2, 7, [16032] * 8),
    (BF16, BF16, 1, 5, [18992] * 8),
    (F32, F32, 2, 16, [4000] * 8),
]


@pytest.mark.parametrize("dtype,gdtype,N,K,widths", CASES)
def test_vp_eal(A, dev, dtype, gdtype, N, K, widths):
    zd, zt = _inputs("c1" if dtype == F32 else "c2", (N, K, sum(widths)), dtype, seed=len(widths) + K, dev=dev)
    check_eal(A, zd, zt, widths, 1.0, gdtype)


@pytest.mark.parametrize("dtype,gdtype,N,K,widths", CASES)
def test_vp_wtv(A, dev, dtype, gdtype, N, K, widths):
    zd, zt = _inputs("c4" if dtype == F32 else "c2", (N, K, sum(widths)), dtype, seed=3 * len(widths) + K, dev=dev)
    check_wtv(A, zd, zt, widths, 1.0, 1.0, gdtype)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_vp_temperatures_and_scale(A, dev, dtype):
    zd, zt = _inputs("c3", (3, 5, 3001), dtype, seed=9, dev=dev)
    check_eal(A, zd, zt, [1000, 1000, 1001], 0.5, F32, scale=-2.5)
    check_wtv(A, zd, zt, [1000, 1000, 1001], 0.7, 1.3, F32, scale=0.125)


def test_vp_greedy_tie_across_slices(A, dev):
    # equal largest target logits in two slices: the lower global index wins
    zd, zt = _inputs("c1", (2, 3, 600), F32, seed=4, dev=dev)
    top = float(zt.max()) + 1.0
    zt[0, 0, 450] = top
    zt[0, 0, 150] = top
    zt[1, 2, 200] = top
    zt[1, 2, 199] = top
    r = check_eal(A, zd, zt, [200, 200, 200])
    assert r["xstar"][0, 0].item() == 150 and r["xstar"][1, 2].item() == 199


def test_vp_masked_slice(A, dev):
    # a rank whose slice is masked out entirely (-inf) contributes nothing
    zd, zt = _inputs("c4", (3, 4, 1200), F32, seed=11, dev=dev)
    zd[:, :, 400:800] = float("-inf")
    zt[:, :, 400:800] = float("-inf")
    check_eal(A, zd, zt, [400, 400, 400])
    check_wtv(A, zd, zt, [400, 400, 400], 0.8, 0.8)


def test_vp_matches_fused_call_and_is_deterministic(A, dev):
    zd, zt = _inputs("c2", (4, 7, 8192), BF16, seed=21, dev=dev)
    a = run_vp(A, zd, zt, A.AAL_VP_WTV, [2048] * 4)
    b = run_vp(A, zd, zt, A.AAL_VP_WTV, [2048] * 4)
    for k in ("loss", "E", "accept", "grad", "row"):
        assert torch.equal(a[k], b[k]), k
    f = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0)
    torch.cuda.synchronize()
    assert rel_err(a["loss"].item(), f["loss"].item()) <= 1e-5
    np.testing.assert_allclose(host64(a["accept"]), host64(f["accept"]), rtol=1e-5, atol=1e-6)


def test_vp_argument_errors(A, dev):
    zd, zt = _inputs("c2", (2, 3, 64), BF16, seed=1, dev=dev)
    d, t = zd.reshape(6, 64).contiguous(), zt.reshape(6, 64).contiguous()
    with pytest.raises(A.AalError):
        A.aal_vp_row_partials(d, t, -1, A.AAL_VP_EAL, V_total=64)
    with pytest.raises(A.AalError):
        A.aal_vp_row_partials(d, t, 0, 7, V_total=64)
    with pytest.raises(A.AalError):
        A.aal_vp_row_partials(d, t, 0, A.AAL_VP_WTV, 1.0, 0.0, V_total=64)
    with pytest.raises(A.AalError):
        A.aal_vp_row_partials(d, t, 8, A.AAL_VP_EAL, V_total=64)  # the slice ends past V_total


@pytest.mark.parametrize("mode", ["wtv", "eal"])
def test_vp_full_c2_over_8_ranks(A, dev, mode):
    """The c2 workload (2048 windows x 7 x 128256, bf16) with the vocabulary over
    8 ranks of 16032 entries, every slice at full size; the oracle recomputes a
    sample of windows, and over all windows the loss equals -mean(E)."""
    import gc

    from paper_2609_24150_amd.inputs import make_config
    inp = make_config("c2", seed=0, device=dev)
    zd, zt = inp["z_draft"], inp["z_target"]
    N, K, V = zd.shape
    m = A.AAL_VP_WTV if mode == "wtv" else A.AAL_VP_EAL
    r = run_vp(A, zd, zt, m, [V // 8] * 8)
    E = host64(r["E"])
    assert np.all(np.isfinite(E)) and E.min() >= 0 and E.max() <= K * (1 + 1e-6)
    assert rel_err(r["loss"].item(), -E.mean()) <= 1e-6
    rng = np.random.default_rng(5)
    idx = np.unique(np.concatenate([[0, N - 1], rng.choice(N, size=8, replace=False)]))
    sel = torch.as_tensor(idx, device=dev)
    zd_s, zt_s = host64(zd[sel]), host64(zt[sel])
    scale = len(idx) / N
    tol = loss_tol(zd.dtype)
    if mode == "wtv":
        o = O.wtv_loss(zd_s, zt_s, 1.0, 1.0)
        np.testing.assert_allclose(host64(r["accept"][sel]), o["a"], rtol=tol, atol=1e-4)
        coef = wtv_coef(o, len(idx), 1.0) * scale
        extra, near = wtv_flips(zd_s, zt_s, 1.0, 1.0, coef)
        check_grad(host64(r["grad"][sel]), o["grad"] * scale, coef, zd.dtype, zd.dtype, extra_tol=extra)
    else:
        o = O.eal_loss(zd_s, zt_s, 1.0)
        assert np.array_equal(r["xstar"][sel].cpu().numpy(), o["xstar"])
        np.testing.assert_allclose(host64(r["accept"][sel]), o["a"], rtol=tol, atol=1e-7)
        coef = eal_coef(o, len(idx), 1.0) * scale
        check_grad(host64(r["grad"][sel]), o["grad"] * scale, coef, zd.dtype, zd.dtype)
    assert rel_err(host64(r["E"][sel]), o["E"]) <= tol
    del r, inp, zd, zt
    gc.collect()
    torch.cuda.empty_cache()


def test_vp_rows_past_the_grid(A, dev):
    # more rows than row workgroups launched (65,536): the row kernels visit the rest grid-stride
    zd, zt = _inputs("c2", (70001, 1, 40), BF16, seed=8, dev=dev)
    check_eal(A, zd, zt, [16, 24], 1.0, F32)
    check_wtv(A, zd, zt, [16, 24], 1.0, 1.0, F32)


@pytest.mark.parametrize("dtype,widths", [(BF16, [1024] * 4), (F32, [300, 301, 399]), (BF16, [16032] * 8)])
def test_vp_eal_labels(A, dev, dtype, widths):
    """Labels replace the greedy token (the target slices are not read); against
    the oracle's EAL term with labels."""
    N, K, V = 3, 5, sum(widths)
    zd, zt = _inputs("c2", (N, K, V), dtype, seed=17, dev=dev)
    g = torch.Generator().manual_seed(3)
    lab = torch.randint(0, V, (N * K,), generator=g, dtype=torch.int32)
    lab[0] = 0
    lab[-1] = V - 1
    r = run_vp(A, zd, zt, A.AAL_VP_EAL, widths, 0.8, 1.0, F32, labels=lab.to(dev))
    o = O.combined_loss(host64(zd), host64(zt), 0.8, 1.0, (0.0, 1.0, 0.0, 0.0), 0, N, K, K, labels=lab.numpy())
    assert np.array_equal(r["xstar"].cpu().numpy().reshape(-1), lab.numpy())
    tol = loss_tol(zd.dtype)
    assert rel_err(r["loss"].item(), o["loss"]) <= tol
    assert rel_err(host64(r["E"]), o["E_eal"]) <= tol
    np.testing.assert_allclose(host64(r["accept"]).reshape(-1), o["a_eal"], rtol=tol, atol=1e-7)
    check_grad(host64(r["grad"]), o["grad"], o["coef_eal"], zd.dtype, F32)


@pytest.mark.parametrize("widths", [[256, 256, 256, 256], [300, 301, 399]])
def test_vp_eal_labels_out_of_range_match_fused_call(A, dev, widths):
    """Labels outside [0, V) (an ignore index of -100, -1, V, V + 7) are clamped
    into the vocabulary exactly as aal_loss_fwd_bwd clamps them: the assembled
    vocabulary-parallel loss, E, acceptances, tokens and gradient equal the
    fused call's on the same labels."""
    N, K, V = 4, 3, sum(widths)
    zd, zt = _inputs("c2", (N, K, V), F32, seed=23, dev=dev)
    g = torch.Generator().manual_seed(5)
    lab = torch.randint(0, V, (N * K,), generator=g, dtype=torch.int32)
    lab[:5] = torch.tensor([-100, -1, V, V + 7, (1 << 31) - 1], dtype=torch.int32)
    lab_d = lab.to(dev)
    r = run_vp(A, zd, zt, A.AAL_VP_EAL, widths, 0.9, 1.0, F32, labels=lab_d)
    f = A.aal_loss_fwd_bwd(zd, zt, K, weights=(0.0, 1.0, 0.0, 0.0), temp_draft=0.9, labels=lab_d,
                           grad_dtype=F32)
    torch.cuda.synchronize()
    clamped = lab.clamp(0, V - 1).numpy()
    assert np.array_equal(r["xstar"].cpu().numpy().reshape(-1), clamped)
    assert np.array_equal(f["xstar"].cpu().numpy().reshape(-1), clamped)
    assert rel_err(r["loss"].item(), f["loss"].item()) <= 1e-5
    np.testing.assert_allclose(host64(r["E"]), host64(f["E_eal"]), rtol=1e-5)
    np.testing.assert_allclose(host64(r["accept"]).reshape(-1), host64(f["accept_eal"]), rtol=1e-5, atol=1e-7)
    o = O.combined_loss(host64(zd), host64(zt), 0.9, 1.0, (0.0, 1.0, 0.0, 0.0), 0, N, K, K, labels=clamped)
    check_grad(host64(r["grad"]), o["grad"], o["coef_eal"], zd.dtype, F32)
    check_grad(host64(f["grad"]), o["grad"], o["coef_eal"], zd.dtype, F32)


def run_vp_seq(A, zd, zt, mode, widths, K, Td=1.0, Tt=1.0, gdtype=None, scale=None):
    """The vocabulary-parallel steps over B sequences [B, S, V] with windows sliding by one."""
    B, S, V = zd.shape
    rows = B * S
    sl = [(v0, w, zd.reshape(rows, V)[:, v0:v0 + w].contiguous(), zt.reshape(rows, V)[:, v0:v0 + w].contiguous())
          for v0, w in _bounds(V, widths)]
    parts = torch.stack([A.aal_vp_row_partials(d, t, v0, mode, Td, Tt, V_total=V) for v0, w, d, t in sl])
    row = A.aal_vp_merge_rows(parts, mode, Td, Tt)
    acc = None
    if mode == A.AAL_VP_WTV:
        acc = torch.stack([A.aal_vp_accept_partials(d, t, row, Td, Tt) for v0, w, d, t in sl])
    gs = None if scale is None else torch.tensor([scale], device=zd.device)
    r = A.aal_vp_sequence_scan(row, acc, B, S, K, mode, Td, grad_scale=gs)
    g = [A.aal_vp_grad(d, t if mode == A.AAL_VP_WTV else None, row, v0, mode, Td, Tt, grad_dtype=gdtype)
         for v0, w, d, t in sl]
    r["grad"] = torch.cat(g, dim=1).reshape(B, S, V)
    torch.cuda.synchronize()
    return r


SEQ_CASES = [
    ("wtv", BF16, 3, 20, 7, [1024] * 4),
    ("eal", BF16, 3, 20, 7, [1024] * 4),
    ("wtv", F32, 2, 9, 3, [300, 301, 399]),
    ("eal", F32, 2, 5, 5, [500, 500]),
    ("wtv", BF16, 2, 40, 7, [16032] * 8),
]


@pytest.mark.parametrize("mode,dtype,B,S,K,widths", SEQ_CASES)
def test_vp_sequences(A, dev, mode, dtype, B, S, K, widths):
    """Windows sliding over sequences (K <= S, down to one window per sequence)
    against the oracle's sequence-layout objective with that single term."""
    V = sum(widths)
    zd, zt = _inputs("c2" if dtype == BF16 else "c4", (B, S, V), dtype, seed=B * S + K, dev=dev)
    Td, Tt, scale = 0.9, 1.1, 0.5
    m = A.AAL_VP_WTV if mode == "wtv" else A.AAL_VP_EAL
    r = run_vp_seq(A, zd, zt, m, widths, K, Td, Tt, F32, scale)
    zd64, zt64 = host64(zd), host64(zt)
    w = (1.0, 0.0, 0.0, 0.0) if mode == "wtv" else (0.0, 1.0, 0.0, 0.0)
    o = O.combined_loss(zd64, zt64, Td, Tt, w, O.LAYOUT_SEQUENCES, B, S, K, grad_scale=scale)
    tol = loss_tol(zd.dtype)
    assert rel_err(r["loss"].item(), o["loss"]) <= tol
    key = "tv" if mode == "wtv" else "eal"
    assert rel_err(host64(r["E"]), o["E_" + key]) <= tol
    atol = (1e-6 if dtype == F32 else 1e-4) if mode == "wtv" else 1e-7
    np.testing.assert_allclose(host64(r["accept"]).reshape(-1), o["a_" + key], rtol=tol, atol=atol)
    coef = o["coef_" + key]
    if mode == "wtv":
        extra, near = wtv_flips(zd64, zt64, Td, Tt, coef.reshape(B, S))
        check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, F32, extra_tol=extra)
    else:
        assert np.array_equal(r["xstar"].cpu().numpy().reshape(-1), o["xstar"])
        check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, F32)
