"""Pins for the oracle's GRPO loss on the debiased greedy acceptance length:
a hand case, brute-force accepted lengths, the reference-equals-policy
identity, the sequences layout against explicitly sliced windows, and finite
differences away from kinks.  CPU only."""
import json
import os

import numpy as np
import pytest

import oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")))


def test_golden_grpo_one_group():
    c = GOLD["grpo_one_group"]
    r = O.grpo_loss(np.array(c["z_theta"]), np.array(c["z_ref"]), np.array(c["z_target"]), c["T"],
                    O.LAYOUT_WINDOWS, c["groups"], 0, c["m"], c["K"], eps=c["eps"], eps_clip=c["eps_clip"])
    assert r["S_theta"].tolist() == c["S_theta"] and r["S_ref"].tolist() == c["S_ref"]
    assert r["tau_theta"].ravel().tolist() == c["tau_theta"] and r["tau_ref"].ravel().tolist() == c["tau_ref"]
    assert r["reward"].ravel().tolist() == c["reward"]
    for k in ("adv", "log_rho", "rho", "coef"):
        np.testing.assert_allclose(r[k].ravel(), c[k], atol=1e-15)
    np.testing.assert_allclose(r["loss"], c["loss"], atol=1e-15)
    np.testing.assert_allclose(r["grad"], c["grad"], atol=1e-15)


def test_accepted_length_brute_force():
    rng = np.random.default_rng(30)
    S = rng.integers(0, 3, size=(200, 5))
    x = rng.integers(0, 3, size=(200, 5))
    want = []
    for s, t in zip(S, x):
        n = 0
        while n < len(s) and s[n] == t[n]:
            n += 1
        want.append(n)
    assert O.greedy_accepted_length(S, x).tolist() == want


def test_reference_equal_to_policy_gives_zero():
    rng = np.random.default_rng(31)
    G, m, K, V = 3, 4, 3, 7
    z = rng.normal(size=(G * m * K, V))
    r = O.grpo_loss(z, z.copy(), rng.normal(size=z.shape), 0.9, O.LAYOUT_WINDOWS, G, 0, m, K)
    assert np.all(r["reward"] == 0) and np.all(r["log_rho"] == 0) and np.all(r["adv"] == 0)
    assert r["loss"] == 0 and not r["grad"].any()


def test_sequences_layout_equals_sliced_windows():
    """Groups of m sliding windows at anchors of B sequences equal the same
    windows copied out into the windows layout (gradients of a row that sits
    in several windows add up)."""
    rng = np.random.default_rng(32)
    B, S, G, m, K, V = 2, 20, 2, 3, 4, 6
    zt = rng.normal(size=(B * S, V))
    zth = zt + rng.normal(scale=0.8, size=zt.shape)
    zrf = zt + rng.normal(scale=0.8, size=zt.shape)
    anchors = np.array([[0, 9], [4, 13]])
    r = O.grpo_loss(zth, zrf, zt, 1.1, O.LAYOUT_SEQUENCES, B, S, m, K, anchors=anchors, eps_clip=0.3,
                    rho_min=0.2, rho_max=3.0, adv_clip=1.5)
    rows = []
    for b in range(B):
        for g in range(G):
            for i in range(m):
                rows.extend(b * S + anchors[b, g] + i + np.arange(K))
    rows = np.array(rows)
    w = O.grpo_loss(zth[rows], zrf[rows], zt[rows], 1.1, O.LAYOUT_WINDOWS, B * G, 0, m, K, eps_clip=0.3,
                    rho_min=0.2, rho_max=3.0, adv_clip=1.5)
    np.testing.assert_allclose(r["loss"], w["loss"], rtol=1e-14)
    np.testing.assert_array_equal(r["reward"], w["reward"])
    back = np.zeros_like(zth)
    np.add.at(back, rows, w["grad"])
    np.testing.assert_allclose(r["grad"], back, rtol=1e-13, atol=1e-18)


def _away_from_kinks(zth, zrf, zt, T, G, m, K, **kw):
    r = O.grpo_loss(zth, zrf, zt, T, O.LAYOUT_WINDOWS, G, 0, m, K, **kw)
    top2 = np.sort(zth, -1)[:, -2:]
    ok = np.min(top2[:, 1] - top2[:, 0]) > 1e-3
    rho = r["rho"]
    for edge in (1 - kw.get("eps_clip", 0.2), 1 + kw.get("eps_clip", 0.2), kw.get("rho_min", 0.0),
                 kw.get("rho_max", np.inf)):
        ok = ok and np.min(np.abs(rho - edge)) > 1e-4
    return ok and np.max(np.abs(r["log_rho"])) < 9.9


@pytest.mark.parametrize("kw", [dict(eps_clip=0.2), dict(eps_clip=0.5, rho_min=0.5, rho_max=2.0, adv_clip=1.0)])
def test_grpo_grad_finite_differences(kw):
    rng = np.random.default_rng(33)
    G, m, K, V, T = 2, 4, 3, 5, 0.8
    while True:
        zt = rng.normal(size=(G * m * K, V))
        zth = zt + rng.normal(scale=0.6, size=zt.shape)
        zrf = zt + rng.normal(scale=0.6, size=zt.shape)
        if _away_from_kinks(zth, zrf, zt, T, G, m, K, **kw):
            break
    r = O.grpo_loss(zth, zrf, zt, T, O.LAYOUT_WINDOWS, G, 0, m, K, **kw)
    assert np.any(r["coef"] != 0)
    h = 1e-6
    fd = np.zeros_like(zth)
    for i in range(zth.shape[0]):
        for v in range(V):
            zp, zm = zth.copy(), zth.copy()
            zp[i, v] += h
            zm[i, v] -= h
            fd[i, v] = (O.grpo_loss(zp, zrf, zt, T, O.LAYOUT_WINDOWS, G, 0, m, K, **kw)["loss"]
                        - O.grpo_loss(zm, zrf, zt, T, O.LAYOUT_WINDOWS, G, 0, m, K, **kw)["loss"]) / (2 * h)
    assert np.max(np.abs(r["grad"] - fd)) < 1e-8
    np.testing.assert_allclose(r["grad"].sum(-1), 0.0, atol=1e-15)


def test_labels_replace_the_target():
    rng = np.random.default_rng(34)
    G, m, K, V = 2, 3, 2, 6
    zt = rng.normal(size=(G * m * K, V))
    zth = zt + rng.normal(size=zt.shape)
    zrf = zt + rng.normal(size=zt.shape)
    a = O.grpo_loss(zth, zrf, zt, 1.0, O.LAYOUT_WINDOWS, G, 0, m, K)
    b = O.grpo_loss(zth, zrf, None, 1.0, O.LAYOUT_WINDOWS, G, 0, m, K, labels=np.argmax(zt, -1))
    np.testing.assert_array_equal(a["grad"], b["grad"])
    assert a["loss"] == b["loss"]
