"""GPU parity of the combined-objective entry point (aal_loss_fwd_bwd) with
the fp64 oracle: disjoint windows and sliding windows over sequences, every
term alone and in the paper's combinations, both dtypes, ragged and
multi-tile vocabularies, labels, grad_scale, and windows that do not fit —
each under both schedules (the register-resident kernel, used by default
where the shape allows, and the multi-kernel streaming schedule).

Tolerances are those of tests/parity.py; the gradient coefficient of a row
for the elementwise bound is |coef_tv| + |coef_eal| + |coef_kl| (each term's
gradient is that coefficient times a vector bounded by 1 in magnitude)."""
import numpy as np
import pytest
import torch

import oracle as O
from parity import check_grad, host64, rel_err, KAPPA

pytestmark = pytest.mark.gpu

WIN, SEQ = 0, 1


@pytest.fixture(params=[0, 1], ids=["resident", "streaming"])
def flags(request):
    return request.param  # AAL_FLAG_STREAMING = 1


@pytest.fixture(scope="module")
def A():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_24150_amd as lib
    return lib


def _inputs(B, S, V, dtype, seed, peaks=True):
    g = torch.Generator(device="cpu").manual_seed(seed)
    zt = torch.randn(B, S, V, generator=g) * 2.5
    if peaks:
        idx = torch.randint(0, V, (B, S, 3), generator=g)
        zt.scatter_add_(-1, idx, torch.full((B, S, 3), 6.0))
    zd = 0.7 * zt + torch.randn(B, S, V, generator=g) * 1.5
    return zd.to(dtype).cuda(), zt.to(dtype).cuda()


def _check(A, zd, zt, K, weights, layout, Td=1.0, Tt=1.0, labels=None, gdt=None, scale=None, pass_target=True,
           flags=0):
    B, S, V = zd.shape
    r = A.aal_loss_fwd_bwd(zd, zt if pass_target else None, K, weights=weights, temp_draft=Td, temp_target=Tt,
                           layout=layout, labels=labels, grad_dtype=gdt, flags=flags,
                           grad_scale=None if scale is None else torch.tensor([scale], device=zd.device))
    torch.cuda.synchronize()
    zd64, zt64 = host64(zd), host64(zt)
    lab = None if labels is None else labels.cpu().numpy()
    o = O.combined_loss(zd64, zt64, Td, Tt, weights, layout, B, S, K, labels=lab,
                        grad_scale=1.0 if scale is None else scale)
    f32 = zd.dtype == torch.float32
    rtol, atol = (1e-5, 1e-6) if f32 else (1e-3, 1e-5)
    terms = host64(r["terms"])
    on = np.array([w != 0 for w in weights])
    assert np.all(terms[~on] == 0.0)  # terms with weight 0 are not evaluated
    assert np.all(np.abs(terms - o["terms"])[on] <= (rtol * np.abs(o["terms"]) + atol)[on]), (terms, o["terms"])
    assert abs(r["loss"].item() - o["loss"]) <= rtol * abs(o["loss"]) + atol * 4
    W = len(o["E_tv"])
    if W and (weights[0] or weights[3]):
        assert rel_err(host64(r["E_tv"]), o["E_tv"]) <= rtol
    if W and weights[1]:
        assert rel_err(host64(r["E_eal"]), o["E_eal"]) <= rtol
    if weights[1]:
        assert np.array_equal(r["xstar"].cpu().numpy(), o["xstar"])
        np.testing.assert_allclose(host64(r["accept_eal"]), o["a_eal"], rtol=rtol, atol=1e-7)
    if weights[0] or weights[2] or weights[3]:
        np.testing.assert_allclose(host64(r["accept_tv"]), o["a_tv"], rtol=rtol, atol=1e-6 if f32 else 1e-4)
    else:
        assert not r["accept_tv"].any()
    if not weights[1]:
        assert not r["accept_eal"].any() and bool((r["xstar"] == -1).all())
    coef = np.abs(o["coef_tv"]) + np.abs(o["coef_eal"]) + np.abs(o["coef_kl"])
    q = np.exp(O.tempered_log_softmax(zd64.reshape(-1, V), Td))
    p = np.exp(O.tempered_log_softmax(zt64.reshape(-1, V), Tt))
    near = np.abs(q - p) <= 1e-5 * np.maximum(p, q)
    qtie = np.max(np.where(near, q, 0.0), axis=-1)
    rows = np.abs(o["coef_tv"]) * qtie * q.max(-1) > 0.25 * KAPPA * coef
    elems = near if (weights[0] or weights[3]) else None
    return check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, r["grad"].dtype,
                      exclude_rows=rows if elems is not None else None, exclude_elems=elems)


WEIGHTS = [(1, 0, 0, 0), (0, 1, 0, 0), (0, 0, 1, 0), (0, 0, 0, 1), (0, 0.1, 1, 0), (0, 0, 1, 1),
           (0.7, 0.4, 1.3, 0.9)]


@pytest.mark.parametrize("weights", WEIGHTS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_sequences_all_terms(A, weights, dtype, flags):
    zd, zt = _inputs(3, 11, 1000, dtype, seed=1)
    _check(A, zd, zt, 4, weights, SEQ, Td=0.8, Tt=1.2, flags=flags)


@pytest.mark.parametrize("weights", WEIGHTS)
def test_windows_all_terms(A, weights, flags):
    zd, zt = _inputs(5, 4, 3000, torch.bfloat16, seed=2)
    _check(A, zd, zt, 4, weights, WIN, flags=flags)


@pytest.mark.parametrize("S,K", [(7, 7), (5, 7), (1, 1), (9, 1), (40, 16), (23, 5), (16, 8), (17, 8)])
@pytest.mark.parametrize("V", [256, 257])
def test_sequence_edges(A, S, K, V, flags):
    zd, zt = _inputs(2, S, V, torch.float32, seed=3 + S + K)
    _check(A, zd, zt, K, (0.7, 0.4, 1.3, 0.9), SEQ, Td=0.7, Tt=0.7, flags=flags)


@pytest.mark.parametrize("S,K", [(16, 8), (17, 8), (23, 7), (40, 16), (9, 6), (13, 6)])
@pytest.mark.parametrize("weights", [(1, 0, 0, 0), (0, 0, 0, 1), (1, 0.5, 0, 0)])
def test_sequence_edges_tv_without_kl(A, S, K, weights, flags):
    """A TV term and no KL term: the resident schedule keeps [q < p] as bits
    from phase B, refills the target early and (K = 7, 8, no greedy token)
    evaluates the next chunk's first-group target partials ahead; sequences
    whose length K does not divide, on a vocabulary of several members."""
    zd, zt = _inputs(3, S, 20480, torch.bfloat16, seed=5 + S + K)
    _check(A, zd, zt, K, weights, SEQ, Td=0.9, Tt=0.9, flags=flags)


@pytest.mark.parametrize("V", [1, 3, 8, 130, 2047, 2051, 2056])
def test_ragged_vocab(A, V, flags):
    zd, zt = _inputs(2, 6, V, torch.bfloat16, seed=10 + V, peaks=V > 8)
    _check(A, zd, zt, 3, (0.7, 0.4, 1.3, 0.9), SEQ, Td=1.1, Tt=0.9, flags=flags)


@pytest.mark.parametrize("V", [777, 776])
def test_fp32_grad_from_bf16_and_scale(A, V, flags):
    zd, zt = _inputs(2, 9, V, torch.bfloat16, seed=20)
    _check(A, zd, zt, 3, (0.7, 0.4, 1.3, 0.9), SEQ, gdt=torch.float32, scale=3.5, flags=flags)


def test_labels_and_target_free_eal(A, flags):
    zd, zt = _inputs(2, 9, 512, torch.float32, seed=21)
    g = torch.Generator(device="cpu").manual_seed(5)
    lab = torch.randint(0, 512, (2 * 9,), generator=g, dtype=torch.int32).cuda()
    _check(A, zd, zt, 3, (0, 1, 0, 0), SEQ, labels=lab, flags=flags)
    _check(A, zd, zt, 3, (0, 1, 0, 0), SEQ, labels=lab, pass_target=False, flags=flags)
    _check(A, zd, zt, 3, (0.5, 0.1, 1.0, 0.3), SEQ, labels=lab, flags=flags)


@pytest.mark.parametrize("weights", [(0, 1, 0, 0), (0, 0.1, 1, 0), (0.5, 0.3, 0, 0.2)])
def test_labels_with_a_ragged_last_chunk(A, weights, flags):
    """S = 10 positions in chunks of K = 3 (the last chunk holds one row), x*
    from labels (including out-of-range ones, which are clamped)."""
    B, S, K, V = 3, 10, 3, 1024
    zd, zt = _inputs(B, S, V, torch.bfloat16, seed=24)
    g = torch.Generator(device="cpu").manual_seed(6)
    lab = torch.randint(-5, V + 5, (B * S,), generator=g, dtype=torch.int32)
    _check(A, zd, zt, K, weights, SEQ, labels=lab.clamp(0, V - 1).cuda(), flags=flags)
    r1 = A.aal_loss_fwd_bwd(zd, zt, K, weights=weights, layout=SEQ, labels=lab.cuda(), flags=flags)
    r2 = A.aal_loss_fwd_bwd(zd, zt, K, weights=weights, layout=SEQ, labels=lab.clamp(0, V - 1).cuda(), flags=flags)
    torch.cuda.synchronize()
    for k in ("loss", "terms", "grad", "xstar"):
        assert torch.equal(r1[k], r2[k]), k


def test_kl_of_identical_distributions_is_zero(A, flags):
    zd, _ = _inputs(2, 5, 300, torch.float32, seed=22)
    r = A.aal_loss_fwd_bwd(zd, zd.clone(), 3, weights=(0, 0, 1, 1), layout=SEQ, flags=flags)
    torch.cuda.synchronize()
    assert abs(r["terms"][2].item()) < 1e-6 and abs(r["terms"][3].item()) < 1e-6
    assert r["grad"].abs().max().item() < 1e-6


def test_sequences_match_resident_wtv_for_single_window_sequences(A, flags):
    """S = K: every sequence is one window, so the combined entry point and the
    fused WTV kernel compute the same loss and gradient."""
    zd, zt = _inputs(64, 7, 4096, torch.bfloat16, seed=23)
    r = A.aal_loss_fwd_bwd(zd, zt, 7, weights=(1, 0, 0, 0), layout=SEQ, flags=flags)
    w = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0)
    torch.cuda.synchronize()
    assert rel_err(r["loss"].item(), w["loss"].item()) < 1e-5
    d = (r["grad"].float() - w["grad"].float()).abs().max().item()
    assert d <= 2 * w["grad"].float().abs().max().item() * 2 ** -8


@pytest.mark.parametrize("weights", [(1, 0, 0, 0), (0, 0.1, 1, 0), (0, 0, 1, 1), (0.7, 0.4, 1.3, 0.9)])
def test_many_chunks_and_members(A, weights, flags):
    """Sequences of 150 positions (22 chunks of 7, the last of 3 rows) with a
    vocabulary split over 4 workgroups per chunk, so that chunks outnumber the
    teams that run together and neighbouring chunks come from the next round."""
    zd, zt = _inputs(3, 150, 32768, torch.bfloat16, seed=30)
    _check(A, zd, zt, 7, weights, SEQ, flags=flags)


@pytest.mark.parametrize("weights", [(0, 0.1, 1, 0), (0, 0, 1, 1)])
def test_many_chunks_ragged_last_member(A, weights):
    """As above with V = 32000: the team's last workgroup holds 928 of its 1024
    vectors, so the rows evaluated ahead from the staged copies are masked past
    the row end as the rows in registers are."""
    zd, zt = _inputs(3, 150, 32000, torch.bfloat16, seed=33)
    _check(A, zd, zt, 7, weights, SEQ)


def test_greedy_ties_across_members_many_windows(A, flags):
    """KL + 0.1 EAL over 40 windows of 7 rows at V = 128256 (16-member teams,
    so windows 16-39 are a team's second or third window) with tied greedy
    maxima in different members, in rows whose token is taken ahead during
    the previous window's merge (rows 0-3) and in rows taken in phase A: the
    lowest index wins, and a_eal = q(x*) matches the oracle."""
    N, K, V = 40, 7, 128256
    g = torch.Generator(device="cpu").manual_seed(35)
    zt = torch.randn(N, K, V, generator=g) * 2.5
    zd = 0.7 * zt + torch.randn(N, K, V, generator=g) * 1.5
    ties = [(0, 0, [100, 125000]), (17, 1, [8191, 8192]), (17, 5, [64, 512, 128000]),
            (33, 3, [24576, 127000, 3]), (39, 2, list(range(0, V, 8192))), (20, 6, [125000, 128255])]
    for n, k, cols in ties:
        zt[n, k, cols] = 40.0
    a, b = zd.to(torch.bfloat16).cuda(), zt.to(torch.bfloat16).cuda()
    r = A.aal_loss_fwd_bwd(a, b, K, weights=(0, 0.1, 1, 0), layout=WIN, flags=flags)
    torch.cuda.synchronize()
    xs = r["xstar"].cpu().numpy().reshape(N, K)
    for n, k, cols in ties:
        assert xs[n, k] == min(cols), (n, k, xs[n, k])
    zd64, zt64 = host64(a), host64(b)
    assert np.array_equal(xs, O.greedy_token(zt64))
    a_o, _, _ = O.acceptance_greedy(zd64, zt64, 1.0)
    np.testing.assert_allclose(host64(r["accept_eal"]).reshape(N, K), a_o,
                               rtol=1e-3, atol=1e-7)


@pytest.mark.parametrize("weights", [(0, 0, 1, 0), (0, 0.1, 1, 0), (0, 0.1, 1, 0.5), (0.5, 0, 1, 0)])
@pytest.mark.parametrize("layout,shape", [(WIN, (6, 5, 4096)), (SEQ, (2, 33, 4096))])
def test_without_per_row_outputs(A, weights, layout, shape, flags):
    """Loss and gradient when the per-row and per-window outputs are not
    requested (the KL term then skips sum min(p, q) in the resident schedule)."""
    B, S, V = shape
    zd, zt = _inputs(B, S, V, torch.bfloat16, seed=32)
    r = A.aal_loss_fwd_bwd(zd, zt, 5, weights=weights, layout=layout, flags=flags, outputs=False)
    torch.cuda.synchronize()
    o = O.combined_loss(host64(zd), host64(zt), 1.0, 1.0, weights, layout, B, S, 5)
    assert abs(r["loss"].item() - o["loss"]) <= 1e-3 * abs(o["loss"]) + 4e-5
    coef = np.abs(o["coef_tv"]) + np.abs(o["coef_eal"]) + np.abs(o["coef_kl"])
    q = np.exp(O.tempered_log_softmax(host64(zd).reshape(-1, V), 1.0))
    p = np.exp(O.tempered_log_softmax(host64(zt).reshape(-1, V), 1.0))
    near = np.abs(q - p) <= 1e-5 * np.maximum(p, q)
    qtie = np.max(np.where(near, q, 0.0), axis=-1)
    rows = np.abs(o["coef_tv"]) * qtie * q.max(-1) > 0.25 * KAPPA * coef
    tv = weights[0] or weights[3]
    check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, r["grad"].dtype,
               exclude_rows=rows if tv else None, exclude_elems=near if tv else None)


def test_resident_is_deterministic_and_agrees_with_streaming(A):
    zd, zt = _inputs(2, 61, 8192, torch.bfloat16, seed=31)
    w = (0.7, 0.4, 1.3, 0.9)
    r1 = A.aal_loss_fwd_bwd(zd, zt, 5, weights=w, layout=SEQ)
    r2 = A.aal_loss_fwd_bwd(zd, zt, 5, weights=w, layout=SEQ)
    rc = A.aal_loss_fwd_bwd(zd, zt, 5, weights=w, layout=SEQ, flags=A.AAL_FLAG_COOPERATIVE)
    s = A.aal_loss_fwd_bwd(zd, zt, 5, weights=w, layout=SEQ, flags=1)
    torch.cuda.synchronize()
    for k in ("loss", "terms", "E_tv", "E_eal", "accept_tv", "accept_eal", "xstar", "grad"):
        assert torch.equal(r1[k], r2[k]), k
        assert torch.equal(r1[k], rc[k]), k  # the cooperative launch: same grid, same bits
    assert rel_err(r1["loss"].item(), s["loss"].item()) < 1e-5
    assert torch.equal(r1["xstar"], s["xstar"])
    d = (r1["grad"].float() - s["grad"].float()).abs().max().item()
    assert d <= 2 * s["grad"].float().abs().max().item() * 2 ** -8
