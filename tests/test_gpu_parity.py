"""GPU parity of the HIP library (through its C ABI) against the fp64 oracle on
small seeded inputs that span several tiles and ragged tails.  Tolerances are
documented in tests/parity.py."""
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


def _flags(A, path):
    return A.AAL_FLAG_STREAMING if path == "stream" else 0


def _check_eal(A, zd, zt, T, gdtype, flags, scale=None):
    r = A.aal_eal_fwd_bwd(zd, zt, T, grad_dtype=gdtype, flags=flags,
                          grad_scale=None if scale is None else torch.tensor([scale], device=zd.device))
    torch.cuda.synchronize()
    o = O.eal_loss(host64(zd), host64(zt), T, grad_scale=1.0 if scale is None else scale)
    assert np.array_equal(r["xstar"].cpu().numpy(), o["xstar"]), "greedy tokens differ"
    tol = loss_tol(zd.dtype)
    assert rel_err(r["loss"].item(), o["loss"]) <= tol
    assert rel_err(host64(r["E"]), o["E"]) <= tol
    np.testing.assert_allclose(host64(r["accept"]), o["a"], rtol=tol, atol=1e-7)
    coef = eal_coef(o, zd.shape[0], T, 1.0 if scale is None else scale)
    return check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, gdtype)


def _check_wtv(A, zd, zt, Td, Tt, gdtype, flags, scale=None):
    r = A.aal_wtv_fwd_bwd(zd, zt, Td, Tt, grad_dtype=gdtype, flags=flags,
                          grad_scale=None if scale is None else torch.tensor([scale], device=zd.device))
    torch.cuda.synchronize()
    zd64, zt64 = host64(zd), host64(zt)
    o = O.wtv_loss(zd64, zt64, Td, Tt, grad_scale=1.0 if scale is None else scale)
    tol = loss_tol(zd.dtype)
    assert rel_err(r["loss"].item(), o["loss"]) <= tol
    assert rel_err(host64(r["E"]), o["E"]) <= tol
    np.testing.assert_allclose(host64(r["accept"]), o["a"], rtol=tol, atol=1e-6 if zd.dtype == F32 else 1e-4)
    coef = wtv_coef(o, zd.shape[0], Td, 1.0 if scale is None else scale)
    extra, near = wtv_flips(zd64, zt64, Td, Tt, coef)
    return check_grad(host64(r["grad"]), o["grad"], coef, zd.dtype, gdtype, extra_tol=extra)


# (V, K, N) spanning: V below one vector, ragged vectors, exact vector multiples,
# several 256-thread tiles with ragged tails, and the workloads' vocabularies.
SHAPES = [(1, 1, 3), (2, 2, 3), (3, 7, 2), (7, 3, 3), (8, 4, 2), (9, 2, 3), (1023, 4, 3),
          (1024, 4, 5), (1025, 7, 3), (4099, 2, 2), (32000, 16, 2), (128256, 7, 1), (151936, 5, 1),
          # K = 6 and 8 on teams of several members: the fused WTV schedule splits their
          # unstaged pairs differently (at K = 6 every unstaged draft pair is restaged; at
          # K = 8 the first row group's target partials are evaluated one window ahead)
          (20000, 6, 3), (32000, 8, 2),
          # window lengths the resident kernel does not take (the streaming schedule
          # runs them in both paths), up to the largest K the boundary accepts
          (3000, 12, 2), (1000, 64, 2)]


@pytest.mark.parametrize("path", ["auto", "stream"])
@pytest.mark.parametrize("dtype,gdtype", [(F32, F32), (BF16, BF16), (BF16, F32), (F32, BF16)])
@pytest.mark.parametrize("V,K,N", SHAPES)
def test_eal_parity_shapes(A, dev, V, K, N, dtype, gdtype, path):
    zd, zt = _inputs("c1" if dtype == F32 else "c2", (N, K, V), dtype, seed=V + K, dev=dev)
    _check_eal(A, zd, zt, 1.0, gdtype, _flags(A, path))


@pytest.mark.parametrize("path", ["auto", "stream"])
@pytest.mark.parametrize("dtype,gdtype", [(F32, F32), (BF16, BF16), (BF16, F32), (F32, BF16)])
@pytest.mark.parametrize("V,K,N", SHAPES)
def test_wtv_parity_shapes(A, dev, V, K, N, dtype, gdtype, path):
    zd, zt = _inputs("c4" if dtype == F32 else "c2", (N, K, V), dtype, seed=V * 3 + K, dev=dev)
    _check_wtv(A, zd, zt, 1.0, 1.0, gdtype, _flags(A, path))


# Small vocabularies with many windows: one workgroup per team and two to four
# windows per team, so the fused schedule runs several windows per team (the
# alternating slot planes, the row-group merges and the windows that follow
# each other without a barrier), checked element by element.
MANY = [(BF16, BF16, 1024, 7, 700), (BF16, F32, 4096, 5, 600), (F32, F32, 2048, 16, 800),
        (BF16, BF16, 2048, 8, 500), (F32, BF16, 1024, 6, 600), (BF16, BF16, 8192, 4, 400)]


@pytest.mark.parametrize("dtype,gdtype,V,K,N", MANY)
def test_many_windows_per_team(A, dev, dtype, gdtype, V, K, N):
    zd, zt = _inputs("c1" if dtype == F32 else "c2", (N, K, V), dtype, seed=N + K, dev=dev)
    _check_eal(A, zd, zt, 1.0, gdtype, 0)
    _check_wtv(A, zd, zt, 0.7, 0.7, gdtype, 0)


@pytest.mark.parametrize("T", [0.05, 0.5, 0.7, 1.0, 2.0])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_temperatures(A, dev, T, dtype):
    zd, zt = _inputs("c3", (3, 5, 3001), dtype, seed=int(T * 100), dev=dev)
    _check_eal(A, zd, zt, T, dtype, 0)
    _check_wtv(A, zd, zt, T, T, dtype, 0)
    _check_wtv(A, zd, zt, T, 1.0, dtype, 0)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_grad_scale(A, dev, dtype):
    zd, zt = _inputs("c2", (4, 3, 2048), dtype, seed=5, dev=dev)
    _check_eal(A, zd, zt, 1.0, F32, 0, scale=-2.5)
    _check_wtv(A, zd, zt, 0.9, 1.1, F32, 0, scale=0.125)


def test_masked_vocabulary(A, dev):
    zd, zt = _inputs("c4", (3, 4, 1000), F32, seed=11, dev=dev)
    zd[:, :, 500:] = float("-inf")
    zt[:, :, :250] = float("-inf")
    _check_eal(A, zd, zt, 1.0, F32, 0)
    _check_wtv(A, zd, zt, 0.8, 0.8, F32, 0)


def test_extreme_logits(A, dev):
    g = torch.Generator().manual_seed(3)
    zt = (torch.rand(2, 3, 777, generator=g) * 2e4 - 1e4)
    zd = (torch.rand(2, 3, 777, generator=g) * 2e4 - 1e4)
    for dtype in (F32, BF16):
        a, b = zd.to(dtype).to(dev), zt.to(dtype).to(dev)
        for T in (0.05, 1.0):
            _check_eal(A, a, b, T, F32, 0)
            _check_wtv(A, a, b, T, T, F32, 0)


def test_identical_inputs_accept_everything(A, dev):
    zd, _ = _inputs("c2", (3, 7, 5000), BF16, seed=2, dev=dev)
    r = A.aal_wtv_fwd_bwd(zd, zd.clone(), 0.7, 0.7, grad_dtype=F32)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host64(r["accept"]), 1.0, atol=2e-6)
    np.testing.assert_allclose(r["loss"].item(), -7.0, rtol=1e-5)
    assert host64(r["grad"]).__abs__().max() < 1e-6


def test_one_hot_target_wtv_equals_eal(A, dev):
    zd, _ = _inputs("c4", (3, 4, 999), F32, seed=4, dev=dev)
    xs = torch.randint(0, 999, (3, 4), generator=torch.Generator().manual_seed(1))
    zt = torch.full((3, 4, 999), float("-inf"))
    zt.scatter_(2, xs[..., None], 0.0)
    zt = zt.to(dev)
    e = A.aal_eal_fwd_bwd(zd, zt, 0.8, grad_dtype=F32)
    w = A.aal_wtv_fwd_bwd(zd, zt, 0.8, 0.8, grad_dtype=F32)
    torch.cuda.synchronize()
    assert np.array_equal(e["xstar"].cpu().numpy(), xs.numpy())
    np.testing.assert_allclose(host64(w["accept"]), host64(e["accept"]), rtol=1e-5)
    np.testing.assert_allclose(host64(w["grad"]), host64(e["grad"]), atol=1e-7)
    _check_wtv(A, zd, zt, 0.8, 0.8, F32, 0)


def test_argmax_ties_lowest_index(A, dev):
    zt = torch.zeros(2, 3, 300)
    zt[0, 0, [7, 100, 299]] = 5.0
    zt[0, 1, :] = 1.0
    zt[1, 2, [299, 298]] = 2.0
    zd = torch.randn(2, 3, 300, generator=torch.Generator().manual_seed(0))
    for dtype in (F32, BF16):
        a, b = zd.to(dtype).to(dev), zt.to(dtype).to(dev)
        r = A.aal_eal_fwd_bwd(a, b, 1.0)
        torch.cuda.synchronize()
        xs = r["xstar"].cpu().numpy()
        assert xs[0, 0] == 7 and xs[0, 1] == 0 and xs[1, 2] == 298
        assert np.array_equal(xs, O.greedy_token(host64(b)))


@pytest.mark.parametrize("path", ["auto", "stream"])
@pytest.mark.parametrize("dtype", [BF16, F32])
def test_argmax_ties_across_team_members(A, dev, dtype, path):
    """Tied greedy maxima at V = 128256 placed in different members of a
    resident team (8192 bf16 / 4096 fp32 columns per member at K = 7), at
    member boundaries and in different waves of one member: the lowest index
    wins in both schedules."""
    N, K, V = 3, 7, 128256
    zd, zt = _inputs("c2", (N, K, V), F32, seed=31, dev="cpu")
    ties = [(0, 0, [100, 125000]),            # member 0 and the last member
            (0, 1, [125000, 128255]),         # both in the last member, the second at the row end
            (0, 2, [8191, 8192]),             # either side of the first member boundary
            (0, 3, [4095, 4096, 70000]),      # member boundaries at fp32 widths
            (1, 0, [24576, 127000, 3]),       # three members, the lowest index listed last
            (1, 6, [64, 512, 1024, 128000]),  # different waves and members
            (2, 4, list(range(0, V, 8192)))]  # one tie in every bf16 member
    for n, k, cols in ties:
        zt[n, k, cols] = 40.0
    a, b = zd.to(dtype).to(dev), zt.to(dtype).to(dev)
    r = A.aal_eal_fwd_bwd(a, b, 1.0, flags=_flags(A, path))
    torch.cuda.synchronize()
    xs = r["xstar"].cpu().numpy()
    for n, k, cols in ties:
        assert xs[n, k] == min(cols), (n, k, xs[n, k])
    assert np.array_equal(xs, O.greedy_token(host64(b)))
    _check_eal(A, a, b, 1.0, dtype, _flags(A, path))


def test_forward_only_and_stream_and_determinism(A, dev):
    zd, zt = _inputs("c2", (5, 7, 4096), BF16, seed=9, dev=dev)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        r1 = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0, grad=False)
        r2 = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0)
        r3 = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0)
        e1 = A.aal_eal_fwd_bwd(zd, zt, 1.0)
        e2 = A.aal_eal_fwd_bwd(zd, zt, 1.0)
    s.synchronize()
    assert r1["grad"] is None
    assert torch.equal(r1["loss"], r2["loss"]) and torch.equal(r1["E"], r2["E"])
    assert torch.equal(r2["grad"], r3["grad"]) and torch.equal(r2["accept"], r3["accept"])
    assert torch.equal(e1["grad"], e2["grad"]) and torch.equal(e1["loss"], e2["loss"])


@pytest.mark.parametrize("dtype,V,K,N", [(BF16, 128256, 7, 40), (BF16, 151936, 5, 30), (F32, 32000, 16, 20)])
def test_cooperative_launch_gives_the_same_bits(A, dev, dtype, V, K, N):
    """The resident kernel launched plainly (the default) and through the
    runtime's cooperative launch (AAL_FLAG_COOPERATIVE): same grid, same bits,
    and both agree with the oracle on a few windows."""
    zd, zt = _inputs("c2", (N, K, V), dtype, seed=13, dev=dev)
    for fn, args in ((A.aal_wtv_fwd_bwd, (0.9, 1.1)), (A.aal_eal_fwd_bwd, (0.8,))):
        r0 = fn(zd, zt, *args, flags=0)
        r1 = fn(zd, zt, *args, flags=A.AAL_FLAG_COOPERATIVE)
        torch.cuda.synchronize()
        for k in r0:
            if r0[k] is not None:
                assert torch.equal(r0[k], r1[k]), (fn.__name__, k)
    _check_wtv(A, zd[:3], zt[:3], 0.9, 1.1, dtype, A.AAL_FLAG_COOPERATIVE)
    _check_eal(A, zd[:3], zt[:3], 0.8, dtype, A.AAL_FLAG_COOPERATIVE)


def test_boundary_errors_write_nothing(A, dev):
    from paper_2609_24150_amd import _lib
    zd, zt = _inputs("c2", (2, 3, 256), BF16, seed=1, dev=dev)
    small = torch.empty(16, dtype=torch.uint8, device=dev)
    with pytest.raises(A.AalError) as ei:
        A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0, ws=small)
    assert ei.value.status == _lib.AAL_ERR_WORKSPACE
    with pytest.raises(A.AalError) as ei:
        A.aal_eal_fwd_bwd(zd, zt, 0.0)
    assert ei.value.status == _lib.AAL_ERR_ARG
    with pytest.raises(A.AalError) as ei:
        A.aal_eal_fwd_bwd(zd, zt, float("nan"))
    assert ei.value.status == _lib.AAL_ERR_ARG
    # misaligned logits: a view starting 2 bytes into a bf16 buffer
    big = torch.zeros(2 * 3 * 256 + 1, dtype=BF16, device=dev)
    mis = big[1:].view(2, 3, 256)
    with pytest.raises(A.AalError) as ei:
        A.aal_eal_fwd_bwd(mis, zt, 1.0)
    assert ei.value.status == _lib.AAL_ERR_ALIGN
    # nothing was written on error
    loss = torch.full((1,), 123.0, device=dev)
    lib = _lib.lib()
    st = lib.aal_eal_fwd_bwd(zd.data_ptr(), zt.data_ptr(), 0, 2, 3, 256, 1.0, loss.data_ptr(), None, None, None,
                             None, 0, None, 0, small.data_ptr(), 16, None)
    torch.cuda.synchronize()
    assert st == _lib.AAL_ERR_WORKSPACE and loss.item() == 123.0


# ------------------------------------------------------------- simulation
SIM_SHAPES = [(3, 4, 3, 3), (2, 8, 7, 7), (2, 5, 2, 8), (3, 8, 7, 1000), (2, 4, 3, 1025), (2, 8, 7, 128256),
              (1, 3, 2, 70001)]


def _check_sim(A, zd, zt, u1, u2, T, ddof=0, clip=0.0):
    r = A.aal_sim_accept_grpo(zd, zt, u1, u2, T, std_ddof=ddof, adv_clip=clip)
    torch.cuda.synchronize()
    zd64, zt64, u164, u264 = host64(zd), host64(zt), host64(u1), host64(u2)
    o = O.sim_accept_grpo(zd64, zt64, T, u164, u264, ddof=ddof, clip=clip if clip > 0 else None)
    flag = O.sim_near_threshold(zd64, zt64, T, u164, u264)
    tok, acc = r["token"].cpu().numpy(), r["accept"].cpu().numpy().astype(bool)
    ok = ~flag
    assert np.array_equal(tok[ok], o["token"][ok]), "sampled tokens differ"
    assert np.array_equal(acc[ok], o["accept"][ok]), "accept decisions differ"
    # a group is exact when no flagged decision sits at or before its first rejection
    K = zd.shape[2]
    first_rej = np.where(o["accept"].all(-1), K - 1, np.argmin(o["accept"], -1))
    upto = np.arange(K)[None, None, :] <= first_rej[..., None]
    gflag = (flag & upto).any(-1)  # [P, G]
    pflag = gflag.any(-1)  # groups (prefixes) with any flagged rollout
    rew = r["reward"].cpu().numpy()
    assert np.array_equal(rew[~gflag], o["reward"][~gflag])
    adv = host64(r["advantage"])
    np.testing.assert_allclose(adv[~pflag], o["advantage"][~pflag], atol=1e-5, rtol=0)
    return int(flag.sum())


@pytest.mark.parametrize("dtype", [BF16, F32])
@pytest.mark.parametrize("P,G,K,V", SIM_SHAPES)
def test_sim_parity(A, dev, P, G, K, V, dtype):
    from paper_2609_24150_amd.inputs import make_uniforms
    zd, zt = _inputs("c5", (P, G, K, V), dtype, seed=V + G, dev=dev)
    u1, u2 = make_uniforms((P, G, K), seed=V, device="cpu")
    _check_sim(A, zd, zt, u1.to(dev), u2.to(dev), 1.0)


def test_sim_options_and_edges(A, dev):
    from paper_2609_24150_amd.inputs import make_uniforms
    zd, zt = _inputs("c2", (4, 8, 5, 3000), BF16, seed=1, dev=dev)
    u1, u2 = make_uniforms((4, 8, 5), seed=2, device="cpu")
    u1, u2 = u1.to(dev), u2.to(dev)
    _check_sim(A, zd, zt, u1, u2, 0.7, ddof=1)
    _check_sim(A, zd, zt, u1, u2, 1.0, clip=0.5)
    # identical distributions: always accepted, reward K, advantage 0
    r = A.aal_sim_accept_grpo(zd, zd.clone(), u1, u2, 1.0)
    torch.cuda.synchronize()
    assert (r["reward"] == 5).all() and (r["advantage"] == 0).all()
    # u1 = 0 picks the first token with positive mass; masked prefix
    zm = zd.clone()
    zm[..., :17] = float("-inf")
    z0 = torch.zeros_like(u1)
    r = A.aal_sim_accept_grpo(zm, zt, z0, u2, 1.0)
    torch.cuda.synchronize()
    assert (r["token"] == 17).all()
    _check_sim(A, zm, zt, u1, u2, 1.0)
