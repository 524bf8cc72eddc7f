"""Pins for the fp64 oracle: hand cases, closed forms, identities the paper
states, finite differences and brute-force enumeration.  CPU only."""
import json
import os
from fractions import Fraction
from itertools import product

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

import oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")))


def fr(x):
    return float(Fraction(x))


def frs(a):
    return np.vectorize(fr, otypes=[np.float64])(np.asarray(a, dtype=object))


# ---------------------------------------------------------------- golden cases
def test_golden_temperature():
    c = GOLD["temperature_v2"]
    q = np.exp(O.tempered_log_softmax(np.array(c["z"]), c["T"]))
    np.testing.assert_allclose(q, frs(c["q"]), rtol=0, atol=1e-15)


def test_golden_eal_single_and_window():
    for key in ("eal_v2_single", "eal_window_k2"):
        c = GOLD[key]
        r = O.eal_loss(np.array(c["z_draft"]), np.array(c["z_target"]), c["T_draft"])
        assert r["xstar"].tolist() == c["xstar"]
        np.testing.assert_allclose(r["a"], frs(c["a"]), atol=1e-15)
        np.testing.assert_allclose(r["loss"], fr(c["loss"]), atol=1e-15)
        np.testing.assert_allclose(r["grad"], frs(c["grad"]), atol=1e-15)
        if "E" in c:
            np.testing.assert_allclose(r["E"], frs(c["E"]), atol=1e-15)


def test_golden_wtv_single():
    c = GOLD["wtv_v2_single"]
    r = O.wtv_loss(np.array(c["z_draft"]), np.array(c["z_target"]), c["T_draft"], c["T_target"])
    np.testing.assert_allclose(r["a"], frs(c["a"]), atol=1e-15)
    np.testing.assert_allclose(r["tv"], frs(c["tv"]), atol=1e-15)
    np.testing.assert_allclose(r["qlt"], frs(c["qlt"]), atol=1e-15)
    np.testing.assert_allclose(r["loss"], fr(c["loss"]), atol=1e-15)
    np.testing.assert_allclose(r["grad"], frs(c["grad"]), atol=1e-15)


def test_golden_window_gamma3():
    c = GOLD["window_gamma3"]
    a = frs(c["a"])
    np.testing.assert_allclose(O.length_distribution(a), frs(c["length_distribution"]), atol=1e-15)
    np.testing.assert_allclose(O.expected_length_full(a), fr(c["E"]), atol=1e-15)
    np.testing.assert_allclose(O.expected_length(a), fr(c["E"]), atol=1e-15)
    np.testing.assert_allclose(O.expected_length_grad(a), frs(c["dE_da"]), atol=1e-15)


def test_golden_uniform_draft():
    c = GOLD["uniform_draft"]
    V, K = c["V"], c["K"]
    rng = np.random.default_rng(1)
    zt = rng.normal(size=(1, K, V))
    zd = np.zeros((1, K, V))
    r = O.eal_loss(zd, zt, 1.0)
    exact = sum(Fraction(1, V ** k) for k in range(1, K + 1))
    np.testing.assert_allclose(r["E"][0], float(exact), rtol=1e-14)
    np.testing.assert_allclose(r["E"][0], c["E_value"], rtol=1e-12)


def test_golden_sim_cases():
    c = GOLD["sim_v3"]
    zd = np.array(c["z_draft"])[None, :]
    zt = np.array(c["z_target"])[None, :]
    for case in c["cases"]:
        x, acc, r, q, p = O.simulate_acceptance(zd, zt, c["T"], np.array([case["u1"]]), np.array([case["u2"]]))
        assert int(x[0]) == case["token"], case
        assert bool(acc[0]) == case["accept"], case
        assert int(r) == int(case["accept"])


def test_golden_advantage():
    c = GOLD["advantage"]
    r = np.array(c["reward"], np.float64)
    for ddof, key in ((0, "var_ddof0"), (1, "var_ddof1")):
        A = O.group_advantage(r, 1e-6, ddof)
        mean = frs(c["mean"])[:, None]
        std = np.sqrt(frs(c[key]))[:, None]
        np.testing.assert_allclose(A, (r - mean) / (std + 1e-6), atol=1e-15)
    assert np.all(O.group_advantage(r)[1] == 0.0)


# ------------------------------------------------------- temperature and lse
def test_tempered_softmax_matches_library_and_is_shift_invariant():
    rng = np.random.default_rng(0)
    z = rng.normal(scale=3, size=(5, 37))
    for T in (0.05, 0.5, 1.0, 2.0):
        ref = softmax(z / T, axis=-1)
        got = np.exp(O.tempered_log_softmax(z, T))
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(O.tempered_log_softmax(z, T),
                                   z / T - logsumexp(z / T, axis=-1, keepdims=True), atol=1e-10)
        shifted = np.exp(O.tempered_log_softmax(z + 123.25, T))
        np.testing.assert_allclose(shifted, got, rtol=1e-10, atol=1e-300)


def test_v2_is_logistic():
    for d in (-3.0, -0.2, 0.0, 1.7):
        for T in (0.3, 1.0, 2.5):
            q = np.exp(O.tempered_log_softmax(np.array([d, 0.0]), T))
            np.testing.assert_allclose(q[0], 1.0 / (1.0 + np.exp(-d / T)), rtol=1e-14)


def test_greedy_limit_concentrates_on_argmax():
    rng = np.random.default_rng(3)
    z = rng.normal(size=(4, 50))
    q = np.exp(O.tempered_log_softmax(z, 1e-4))
    assert np.all(np.argmax(q, -1) == np.argmax(z, -1))
    assert np.all(q.max(-1) > 1 - 1e-12)


def test_argmax_lowest_index_on_ties():
    z = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0]])
    assert O.greedy_token(z).tolist() == [1, 0]


# ---------------------------------------------------------- acceptance terms
def test_sampling_acceptance_is_one_minus_tv_and_in_unit_interval():
    rng = np.random.default_rng(4)
    zd = rng.normal(scale=2, size=(6, 3, 101))
    zt = rng.normal(scale=2, size=(6, 3, 101))
    for T in (0.5, 1.0):
        a, q, p = O.acceptance_sampling(zd, zt, T, T)
        np.testing.assert_allclose(a, 1.0 - 0.5 * np.abs(p - q).sum(-1), atol=1e-12)
        assert np.all(a >= 0) and np.all(a <= 1 + 1e-15)


def test_identical_distributions_accept_everything():
    rng = np.random.default_rng(5)
    z = rng.normal(size=(3, 4, 64))
    r = O.wtv_loss(z, z, 0.7, 0.7)
    np.testing.assert_allclose(r["a"], 1.0, atol=1e-14)
    np.testing.assert_allclose(r["E"], 4.0, atol=1e-13)
    np.testing.assert_allclose(r["loss"], -4.0, atol=1e-13)
    assert np.max(np.abs(r["grad"])) < 1e-12


def test_disjoint_supports_accept_nothing():
    V = 16
    zd = np.full((2, 3, V), -np.inf)
    zt = np.full((2, 3, V), -np.inf)
    zd[..., : V // 2] = 0.0
    zt[..., V // 2:] = 1.0
    r = O.wtv_loss(zd, zt, 1.0, 1.0)
    assert np.all(r["a"] == 0.0) and np.all(r["E"] == 0.0)


def test_one_hot_target_makes_wtv_equal_eal():
    rng = np.random.default_rng(6)
    N, K, V = 3, 4, 50
    zd = rng.normal(scale=1.5, size=(N, K, V))
    xs = rng.integers(0, V, size=(N, K))
    zt = np.full((N, K, V), -np.inf)
    np.put_along_axis(zt, xs[..., None], 0.0, axis=-1)
    for T in (0.6, 1.0):
        w = O.wtv_loss(zd, zt, T, T)
        e = O.eal_loss(zd, zt, T)
        assert np.all(e["xstar"] == xs)
        np.testing.assert_allclose(w["a"], e["a"], rtol=1e-13)
        np.testing.assert_allclose(w["loss"], e["loss"], rtol=1e-13)
        np.testing.assert_allclose(w["grad"], e["grad"], atol=1e-15)


def test_draft_one_hot_on_greedy_token():
    rng = np.random.default_rng(7)
    N, K, V = 2, 5, 40
    zt = rng.normal(size=(N, K, V))
    xs = np.argmax(zt, -1)
    zd = np.zeros((N, K, V))
    np.put_along_axis(zd, xs[..., None], 1000.0, axis=-1)
    r = O.eal_loss(zd, zt, 1.0)
    np.testing.assert_allclose(r["a"], 1.0)
    np.testing.assert_allclose(r["E"], K)
    assert np.max(np.abs(r["grad"])) == 0.0


# -------------------------------------------------------------------- window
def test_window_identities_random():
    rng = np.random.default_rng(8)
    for K in (1, 2, 3, 7, 16):
        a = rng.uniform(size=(20, K))
        d = O.length_distribution(a)
        np.testing.assert_allclose(d.sum(-1), 1.0, atol=1e-14)
        np.testing.assert_allclose(O.expected_length_full(a), O.expected_length(a), atol=1e-13)
        if K == 1:
            np.testing.assert_allclose(O.expected_length(a), a[:, 0])


def test_window_constant_a_closed_form():
    for a0 in (0.1, 0.5, 0.93):
        for K in (1, 4, 7, 16):
            E = O.expected_length(np.full((1, K), a0))
            np.testing.assert_allclose(E, a0 * (1 - a0 ** K) / (1 - a0), rtol=1e-13)


def test_window_gradient_finite_difference_and_zero_a():
    rng = np.random.default_rng(9)
    a = rng.uniform(size=(5, 6))
    g = O.expected_length_grad(a)
    h = 1e-6
    for j in range(6):
        ap, am = a.copy(), a.copy()
        ap[:, j] += h
        am[:, j] -= h
        fd = (O.expected_length(ap) - O.expected_length(am)) / (2 * h)
        np.testing.assert_allclose(g[:, j], fd, atol=1e-9)
    a0 = np.array([[0.5, 0.0, 0.25]])
    # E = a0 + a0 a1 + a0 a1 a2; at a1 = 0: dE/da1 = a0 + a0 a2 = 0.625
    np.testing.assert_allclose(O.expected_length_grad(a0), [[1.0, 0.625, 0.0]])


# ------------------------------------------------------------------ gradients
def _fd_check(fn, zd, h=1e-6):
    base = fn(zd)
    G = base["grad"]
    fd = np.zeros_like(zd)
    it = np.nditer(zd, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        zp, zm = zd.copy(), zd.copy()
        zp[i] += h
        zm[i] -= h
        fd[i] = (fn(zp)["loss"] - fn(zm)["loss"]) / (2 * h)
    return G, fd


def test_eal_gradient_finite_differences():
    rng = np.random.default_rng(10)
    N, K, V = 3, 4, 7
    zt = rng.normal(size=(N, K, V))
    zd = 0.8 * zt + rng.normal(scale=0.7, size=(N, K, V))
    for T in (0.7, 1.0):
        G, fd = _fd_check(lambda z: O.eal_loss(z, zt, T), zd)
        assert np.max(np.abs(G - fd)) < 1e-8


def test_wtv_gradient_finite_differences_away_from_kinks():
    rng = np.random.default_rng(11)
    N, K, V = 2, 3, 6
    for T in (0.7, 1.0):
        while True:
            zt = rng.normal(size=(N, K, V))
            zd = 0.8 * zt + rng.normal(scale=0.7, size=(N, K, V))
            q = np.exp(O.tempered_log_softmax(zd, T))
            p = np.exp(O.tempered_log_softmax(zt, T))
            if np.min(np.abs(q - p)) > 1e-4:
                break
        G, fd = _fd_check(lambda z: O.wtv_loss(z, zt, T, T), zd)
        assert np.max(np.abs(G - fd)) < 1e-8


def test_gradient_rows_sum_to_zero_and_scale():
    rng = np.random.default_rng(12)
    zt = rng.normal(size=(4, 5, 33))
    zd = rng.normal(size=(4, 5, 33))
    e = O.eal_loss(zd, zt, 0.8)
    w = O.wtv_loss(zd, zt, 0.8, 1.2)
    assert np.max(np.abs(e["grad"].sum(-1))) < 1e-16
    assert np.max(np.abs(w["grad"].sum(-1))) < 1e-16
    np.testing.assert_allclose(O.wtv_loss(zd, zt, 0.8, 1.2, grad_scale=-2.5)["grad"], -2.5 * w["grad"])


# ---------------------------------------------------------------- simulation
def test_inverse_cdf_matches_linear_scan_and_searchsorted():
    rng = np.random.default_rng(13)
    q = rng.dirichlet(np.ones(11), size=200)
    u = rng.uniform(size=200)
    x = O.inverse_cdf_token(q, u)
    for i in range(200):
        c, v = 0.0, None
        for j in range(11):
            c += q[i, j]
            if c > u[i]:
                v = j
                break
        assert x[i] == v
        assert x[i] == np.searchsorted(np.cumsum(q[i]), u[i], side="right")


def test_inverse_cdf_rounding_fallback():
    q = np.array([[0.5, 0.5, 0.0]])
    assert O.inverse_cdf_token(q, np.array([1.0])).tolist() == [1]


def _exact_expected_reward(zd, zt, T):
    """Exact E[reward] of the simulation over independent u1, u2 ~ U[0,1) per
    position: on each position the (u1, u2) square splits into cells (token x,
    accepted or not) of measure q_x min(1, p_x/q_x) and q_x (1 - min(...)).
    The simulation is evaluated at one interior point of every cell of every
    position and weighted by the product of cell measures."""
    K, V = zd.shape
    q = softmax(zd / T, axis=-1)
    p = softmax(zt / T, axis=-1)
    cells = []
    for k in range(K):
        C = np.concatenate([[0.0], np.cumsum(q[k])])
        ck = []
        for x in range(V):
            r = min(1.0, p[k, x] / q[k, x])
            u1 = 0.5 * (C[x] + C[x + 1])
            if r > 0:
                ck.append((u1, 0.5 * r, q[k, x] * r))
            if r < 1:
                ck.append((u1, 0.5 * (1 + r), q[k, x] * (1 - r)))
        cells.append(ck)
    tot = 0.0
    for combo in product(*cells):
        u1 = np.array([c[0] for c in combo])
        u2 = np.array([c[1] for c in combo])
        w = np.prod([c[2] for c in combo])
        _, _, rew, _, _ = O.simulate_acceptance(zd, zt, T, u1, u2)
        tot += w * float(rew)
    return tot


def test_simulation_expectation_equals_wtv_expected_length_brute_force():
    rng = np.random.default_rng(14)
    K, V = 3, 3
    for T in (0.7, 1.0):
        zt = rng.normal(scale=1.5, size=(K, V))
        zd = 0.5 * zt + rng.normal(size=(K, V))
        exact = _exact_expected_reward(zd, zt, T)
        E = O.wtv_loss(zd[None], zt[None], T, T)["E"][0]
        np.testing.assert_allclose(exact, E, atol=1e-12)


def test_simulation_monte_carlo_matches_wtv():
    rng = np.random.default_rng(15)
    K, V, M = 4, 9, 200000
    zt = rng.normal(scale=1.0, size=(K, V))
    zd = 0.8 * zt + rng.normal(scale=0.4, size=(K, V))
    E = O.wtv_loss(zd[None], zt[None], 1.0, 1.0)["E"][0]
    u1 = rng.uniform(size=(M, K))
    u2 = rng.uniform(size=(M, K))
    _, _, rew, _, _ = O.simulate_acceptance(np.broadcast_to(zd, (M, K, V)), np.broadcast_to(zt, (M, K, V)),
                                            1.0, u1, u2)
    se = rew.std() / np.sqrt(M)
    assert abs(rew.mean() - E) < 5 * se


def test_identical_distributions_always_accept_and_zero_advantage():
    rng = np.random.default_rng(16)
    z = rng.normal(size=(2, 8, 5, 30))
    u1 = rng.uniform(size=(2, 8, 5))
    u2 = rng.uniform(size=(2, 8, 5))
    r = O.sim_accept_grpo(z, z, 1.0, u1, u2)
    assert np.all(r["reward"] == 5)
    assert np.all(r["advantage"] == 0.0)


def test_advantages_have_zero_group_mean_and_clip():
    rng = np.random.default_rng(17)
    r = rng.integers(0, 8, size=(50, 8))
    A = O.group_advantage(r)
    np.testing.assert_allclose(A.mean(-1), 0.0, atol=1e-12)
    assert np.max(np.abs(O.group_advantage(r, clip=0.5))) <= 0.5


def test_near_threshold_flags():
    zd = np.zeros((1, 4))
    zt = np.zeros((1, 4))
    assert O.sim_near_threshold(zd, zt, 1.0, np.array([0.25]), np.array([0.3]))[0]
    assert not O.sim_near_threshold(zd, zt, 1.0, np.array([0.3]), np.array([0.3]))[0]
    # u2 right at min(1, p/q) = 1 is flagged
    assert O.sim_near_threshold(zd, zt, 1.0, np.array([0.3]), np.array([1.0 - 1e-7]))[0]


# ------------------------------------------------- helpers pinned on their own
def test_greedy_acceptance_is_draft_mass_on_target_argmax_by_hand():
    """Eq. acc_greedy on a case worked by hand: target argmax is index 2, so
    a = q(2) = e^1 / (e^0 + e^0 + e^1) for draft logits (0, 0, 1) at T = 1."""
    zd = np.array([[0.0, 0.0, 1.0], [3.0, 0.0, 0.0]])
    zt = np.array([[0.1, -2.0, 5.0], [-1.0, 4.0, 4.0]])
    a, xs, q = O.acceptance_greedy(zd, zt, 1.0)
    assert xs.tolist() == [2, 1]
    e = np.e
    np.testing.assert_allclose(a, [e / (2 + e), 1 / (e ** 3 + 2)], rtol=0, atol=1e-15)
    np.testing.assert_allclose(q.sum(-1), 1.0, atol=1e-15)


def test_total_variation_by_hand_and_bounds():
    """TV is half the l1 distance: 0 on equal rows, 1 on disjoint supports,
    and 0.4 for (0.7, 0.3, 0) against (0.3, 0.3, 0.4)."""
    p = np.array([[0.7, 0.3, 0.0], [1.0, 0.0, 0.0], [0.2, 0.5, 0.3]])
    q = np.array([[0.3, 0.3, 0.4], [0.0, 0.5, 0.5], [0.2, 0.5, 0.3]])
    np.testing.assert_allclose(O.total_variation(p, q), [0.4, 1.0, 0.0], rtol=0, atol=1e-15)
    np.testing.assert_allclose(O.total_variation(p, q), O.total_variation(q, p), atol=0)


def test_survival_probabilities_by_hand():
    """P(L >= k) for a = (1/2, 1/3, 3/4): 1/2, 1/6, 1/8; with a zero, every
    later survival probability is zero."""
    s = O.prob_accepted_at_least(np.array([[0.5, 1 / 3, 0.75], [0.9, 0.0, 1.0]]))
    np.testing.assert_allclose(s, [[0.5, 1 / 6, 1 / 8], [0.9, 0.0, 0.0]], rtol=0, atol=1e-16)


def test_grpo_windows_by_enumeration():
    """Rows of each group's windows enumerated with plain loops: the windows
    layout numbers rows group by group, window by window; the sequences layout
    starts window j of group (b, g) at b*S + anchor[b, g] + j."""
    w = O.grpo_windows(O.LAYOUT_WINDOWS, 2, 0, 3, 4)
    r = 0
    for g in range(2):
        for j in range(3):
            for k in range(4):
                assert w[g, j, k] == r
                r += 1
    B, S, m, K = 2, 11, 3, 2
    anchors = np.array([[0, 5], [2, 6]])
    w = O.grpo_windows(O.LAYOUT_SEQUENCES, B, S, m, K, anchors)
    assert w.shape == (4, m, K)
    for b in range(B):
        for g in range(2):
            for j in range(m):
                for k in range(K):
                    assert w[b * 2 + g, j, k] == b * S + anchors[b, g] + j + k
