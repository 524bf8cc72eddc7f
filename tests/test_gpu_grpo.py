"""GPU parity of aal_grpo_fwd_bwd with the fp64 oracle: both layouts, both
dtypes, labels instead of target logits, clipping active and inactive,
ragged vocabularies, and grad_scale.

Accepted lengths are compared exactly (greedy tokens are decided on the raw
stored logits).  Advantages and log rho within 1e-5 (fp32 logits) / 1e-4
(bf16 logits, whose log-probabilities are computed in fp32 from exact values).
The gradient uses the tolerance of tests/parity.py with the row coefficient
|dloss/dlog rho| / (K T); rows of windows whose ratio lies within 1e-4 of a
clip boundary (where the derivative legitimately switches) are excluded."""
import numpy as np
import pytest
import torch

import oracle as O
from parity import check_grad, host64

pytestmark = pytest.mark.gpu

WIN, SEQ = 0, 1


@pytest.fixture(scope="module")
def A():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_24150_amd as lib
    return lib


def _inputs(shape, dtype, seed, noise=1.0):
    g = torch.Generator(device="cpu").manual_seed(seed)
    V = shape[-1]
    zt = torch.randn(*shape, generator=g) * 2.0
    idx = torch.randint(0, V, shape[:-1] + (1,), generator=g)
    zt.scatter_add_(-1, idx, torch.full(shape[:-1] + (1,), 5.0))
    zth = zt + torch.randn(*shape, generator=g) * noise
    zrf = zt + torch.randn(*shape, generator=g) * noise
    return [t.to(dtype).cuda() for t in (zth, zrf, zt)]


def _check(A, zth, zrf, zt, m, K, layout, anchors=None, labels=None, T=1.0, scale=None, pass_target=True, **prm):
    B, S, V = zth.shape
    r = A.aal_grpo_fwd_bwd(zth, zrf, zt if pass_target else None, m, K, layout=layout, anchors=anchors,
                           labels=labels, temperature=T,
                           grad_scale=None if scale is None else torch.tensor([scale], device=zth.device), **prm)
    torch.cuda.synchronize()
    kw = {k: prm[k] for k in ("eps", "adv_clip", "eps_clip", "rho_min", "rho_max") if k in prm}
    o = O.grpo_loss(host64(zth).reshape(-1, V), host64(zrf).reshape(-1, V), host64(zt).reshape(-1, V), T, layout,
                    B, S, m, K, anchors=None if anchors is None else anchors.cpu().numpy(),
                    labels=None if labels is None else labels.cpu().numpy(),
                    grad_scale=1.0 if scale is None else scale, **kw)
    f32 = zth.dtype == torch.float32
    tol = 1e-5 if f32 else 1e-4
    assert np.array_equal(r["tau_theta"].cpu().numpy(), o["tau_theta"])
    assert np.array_equal(r["tau_ref"].cpu().numpy(), o["tau_ref"])
    np.testing.assert_allclose(host64(r["log_rho"]), o["log_rho"], rtol=tol, atol=tol)
    np.testing.assert_allclose(host64(r["advantage"]), o["adv"], rtol=1e-5, atol=1e-5)
    assert abs(r["loss"].item() - o["loss"]) <= tol * max(1.0, abs(o["loss"]))
    # windows near a kink of the clipped surrogate
    eps_clip = kw.get("eps_clip", 0.2)
    edges = [1 - eps_clip, 1 + eps_clip, kw.get("rho_min", 0.0), kw.get("rho_max", np.inf)]
    rho_e = np.exp(o["log_rho"])
    near = np.zeros(o["rho"].shape, bool)
    for e in edges:
        near |= np.abs(o["rho"] - e) <= 1e-4 * max(1.0, abs(e)) if np.isfinite(e) else False
        near |= np.abs(rho_e - e) <= 1e-4 * max(1.0, abs(e)) if np.isfinite(e) else False
    near |= np.abs(np.abs(o["log_rho"]) - 10.0) <= 1e-4
    win = O.grpo_windows(layout, B, S, m, K, None if anchors is None else anchors.cpu().numpy())
    R = B * S
    excl = np.zeros(R, bool)
    excl[win[near].reshape(-1)] = True
    coef = np.zeros(R)
    np.add.at(coef, win.reshape(-1), np.repeat(np.abs(o["coef"]).reshape(-1), K) / K)
    coef *= (1.0 if scale is None else scale) / T
    return check_grad(host64(r["grad"]).reshape(R, V), o["grad"], coef, zth.dtype, r["grad"].dtype,
                      exclude_rows=excl)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("prm", [dict(), dict(eps_clip=0.5, rho_min=0.3, rho_max=2.5, adv_clip=1.2),
                                 dict(eps_clip=100.0)])
def test_windows_layout(A, dtype, prm):
    m, K = 4, 3
    zth, zrf, zt = _inputs((6, m * K, 1000), dtype, seed=1)
    _check(A, zth, zrf, zt, m, K, WIN, T=0.9, **prm)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_sequences_layout(A, dtype):
    B, S, G, m, K = 2, 40, 3, 4, 3
    zth, zrf, zt = _inputs((B, S, 777), dtype, seed=2)
    anchors = torch.tensor([[0, 12, 30], [5, 18, 31]], dtype=torch.int32).cuda()
    _check(A, zth, zrf, zt, m, K, SEQ, anchors=anchors, eps_clip=0.3, rho_max=4.0)


def test_overlapping_groups_and_clamped_anchors(A):
    B, S, G, m, K = 1, 16, 3, 4, 3
    zth, zrf, zt = _inputs((B, S, 300), torch.float32, seed=3)
    anchors = torch.tensor([[2, 4, 9]], dtype=torch.int32).cuda()  # groups overlap; 9 is the last valid start
    _check(A, zth, zrf, zt, m, K, SEQ, anchors=anchors)


@pytest.mark.parametrize("V", [1, 7, 2049])
def test_ragged_vocab(A, V):
    m, K = 3, 2
    zth, zrf, zt = _inputs((3, m * K, V), torch.bfloat16, seed=4 + V)
    _check(A, zth, zrf, zt, m, K, WIN)


def test_labels_without_target_and_scale(A):
    m, K = 4, 3
    zth, zrf, zt = _inputs((5, m * K, 512), torch.float32, seed=5)
    lab = zt.argmax(-1).to(torch.int32).reshape(-1).contiguous()
    _check(A, zth, zrf, zt, m, K, WIN, labels=lab, pass_target=False, scale=2.0)


def test_reference_equal_to_policy_is_zero(A):
    m, K = 4, 3
    zth, _, zt = _inputs((4, m * K, 256), torch.bfloat16, seed=6)
    r = A.aal_grpo_fwd_bwd(zth, zth.clone(), zt, m, K)
    torch.cuda.synchronize()
    assert r["loss"].item() == 0.0 and not r["grad"].float().abs().max().item()
    assert not r["log_rho"].any() and not r["advantage"].any()


def test_out_of_range_anchors_are_clamped(A):
    """Anchors outside [0, S - (m-1) - K] are clamped into the sequence (the
    documented convention): the result equals the oracle on clamped anchors."""
    B, S, m, K = 2, 30, 4, 3
    zth, zrf, zt = _inputs((B, S, 500), torch.float32, seed=7)
    hi = S - (m - 1) - K
    raw = torch.tensor([[-5, 7], [hi + 9, 2**30]], dtype=torch.int32).cuda()
    r = A.aal_grpo_fwd_bwd(zth, zrf, zt, m, K, layout=SEQ, anchors=raw)
    c = A.aal_grpo_fwd_bwd(zth, zrf, zt, m, K, layout=SEQ, anchors=raw.clamp(0, hi))
    torch.cuda.synchronize()
    for k in ("loss", "tau_theta", "tau_ref", "advantage", "log_rho", "grad"):
        assert torch.equal(r[k], c[k]), k
    _check(A, zth, zrf, zt, m, K, SEQ, anchors=raw.clamp(0, hi))
