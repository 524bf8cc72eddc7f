"""Pins for the oracle's sequence layout (sliding windows) and combined
objectives: hand cases, reductions to the single losses, brute force over
windows, an independent KL / TV computation, and finite differences.  CPU
only."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_cases.json")))


def val(x):
    return float(Fraction(x)) if isinstance(x, str) else float(x)


def vals(a):
    return np.vectorize(val, otypes=[np.float64])(np.asarray(a, dtype=object))


def _softmax_T(z, T):
    """exp(z/T) / sum exp(z/T), written out independently of the oracle."""
    z = np.asarray(z, np.float64) / T
    e = np.exp(z - z.max(-1, keepdims=True))
    return e / e.sum(-1, keepdims=True)


def test_window_rows_hand():
    assert O.window_rows(O.LAYOUT_WINDOWS, 2, 0, 3).tolist() == [[0, 1, 2], [3, 4, 5]]
    assert O.window_rows(O.LAYOUT_SEQUENCES, 2, 5, 3).tolist() == [
        [0, 1, 2], [1, 2, 3], [2, 3, 4], [5, 6, 7], [6, 7, 8], [7, 8, 9]]
    assert O.window_rows(O.LAYOUT_SEQUENCES, 3, 2, 3).shape == (0, 3)
    assert O.window_rows(O.LAYOUT_SEQUENCES, 1, 4, 4).tolist() == [[0, 1, 2, 3]]


def test_golden_sliding_gamma2():
    c = GOLD["sliding_gamma2"]
    win = O.window_rows(O.LAYOUT_SEQUENCES, c["B"], c["S"], c["K"])
    assert win.tolist() == c["windows"]
    E, per_row = O.window_length_coefficients(vals(c["a"]), win)
    np.testing.assert_allclose(E, vals(c["E"]), atol=1e-15)
    np.testing.assert_allclose(per_row, vals(c["dE_da_per_row"]), atol=1e-15)


def test_golden_combined_two_rows():
    c = GOLD["combined_two_rows"]
    r = O.combined_loss(np.array(c["z_draft"]), np.array(c["z_target"]), c["T_draft"], c["T_target"],
                        c["weights"], O.LAYOUT_SEQUENCES, c["B"], c["S"], c["K"])
    np.testing.assert_allclose(r["a_tv"], vals(c["a_tv"]), atol=1e-15)
    np.testing.assert_allclose(r["a_eal"], vals(c["a_eal"]), atol=1e-15)
    assert r["xstar"].tolist() == c["xstar"]
    np.testing.assert_allclose(r["kl"], vals(c["kl"]), atol=1e-15)
    np.testing.assert_allclose(r["terms"], vals(c["terms"]), atol=1e-15)
    np.testing.assert_allclose(r["loss"], vals(c["terms"]).sum(), atol=1e-15)
    np.testing.assert_allclose(r["grad"], vals(c["grad"]), atol=1e-15)


@pytest.mark.parametrize("Td,Tt,scale", [(1.0, 1.0, 1.0), (0.7, 1.3, 2.5)])
def test_windows_layout_reduces_to_single_losses(Td, Tt, scale):
    rng = np.random.default_rng(20)
    N, K, V = 3, 4, 9
    zt = rng.normal(size=(N, K, V))
    zd = 0.7 * zt + rng.normal(scale=0.8, size=(N, K, V))
    w = O.wtv_loss(zd, zt, Td, Tt, grad_scale=scale)
    c = O.combined_loss(zd, zt, Td, Tt, (1, 0, 0, 0), O.LAYOUT_WINDOWS, N, K, K, grad_scale=scale)
    np.testing.assert_allclose(c["loss"], w["loss"], rtol=1e-14)
    np.testing.assert_allclose(c["E_tv"], w["E"], rtol=1e-14)
    np.testing.assert_allclose(c["grad"], w["grad"].reshape(-1, V), rtol=1e-12, atol=1e-17)
    e = O.eal_loss(zd, zt, Td, grad_scale=scale)
    c = O.combined_loss(zd, zt, Td, Tt, (0, 1, 0, 0), O.LAYOUT_WINDOWS, N, K, K, grad_scale=scale)
    np.testing.assert_allclose(c["loss"], e["loss"], rtol=1e-14)
    np.testing.assert_allclose(c["grad"], e["grad"].reshape(-1, V), rtol=1e-12, atol=1e-17)


def test_sequences_of_one_window_equal_windows_layout():
    rng = np.random.default_rng(21)
    B, K, V = 4, 3, 7
    zt = rng.normal(size=(B * K, V))
    zd = rng.normal(size=(B * K, V))
    wts = (0.6, 0.3, 1.1, 0.4)
    a = O.combined_loss(zd, zt, 0.8, 0.9, wts, O.LAYOUT_SEQUENCES, B, K, K)
    b = O.combined_loss(zd, zt, 0.8, 0.9, wts, O.LAYOUT_WINDOWS, B, K, K)
    np.testing.assert_allclose(a["terms"], b["terms"], rtol=1e-14)
    np.testing.assert_allclose(a["grad"], b["grad"], rtol=1e-13, atol=1e-18)


def test_sliding_terms_brute_force():
    """Every window sliced out of the sequences and evaluated on its own;
    KL and TV from an independent softmax."""
    rng = np.random.default_rng(22)
    B, S, K, V = 2, 7, 3, 6
    Td, Tt = 0.8, 1.2
    zt = rng.normal(size=(B, S, V))
    zd = 0.5 * zt + rng.normal(size=(B, S, V))
    r = O.combined_loss(zd, zt, Td, Tt, (1, 1, 1, 1), O.LAYOUT_SEQUENCES, B, S, K)
    q = _softmax_T(zd, Td)
    p = _softmax_T(zt, Tt)
    Etv, Eeal, tv = [], [], []
    for b in range(B):
        for t in range(S - K + 1):
            sl = slice(t, t + K)
            a_tv = np.minimum(p[b, sl], q[b, sl]).sum(-1)
            xs = np.argmax(zt[b, sl], -1)
            a_eal = q[b, sl][np.arange(K), xs]
            Etv.append(sum(np.prod(a_tv[:k]) for k in range(1, K + 1)))
            Eeal.append(sum(np.prod(a_eal[:k]) for k in range(1, K + 1)))
            tv.append(np.mean(0.5 * np.abs(p[b, sl] - q[b, sl]).sum(-1)))
    kl = np.sum(p * (np.log(p) - np.log(q)), -1).mean()
    np.testing.assert_allclose(r["E_tv"], Etv, rtol=1e-13)
    np.testing.assert_allclose(r["E_eal"], Eeal, rtol=1e-13)
    np.testing.assert_allclose(r["terms"], [-np.mean(Etv), -np.mean(Eeal), kl, np.mean(tv)], rtol=1e-13)


def test_kl_properties():
    rng = np.random.default_rng(23)
    z = rng.normal(size=(5, 8))
    kl, _, _ = O.forward_kl(z, z, 0.9, 0.9)
    np.testing.assert_allclose(kl, 0.0, atol=1e-15)
    kl, _, _ = O.forward_kl(z, rng.normal(size=(5, 8)), 0.9, 1.4)
    assert np.all(kl > 0)


def test_combined_grad_finite_differences():
    rng = np.random.default_rng(24)
    B, S, K, V = 1, 5, 3, 5
    Td, Tt = 0.8, 1.1
    while True:
        zt = rng.normal(size=(B * S, V))
        zd = 0.6 * zt + rng.normal(scale=0.8, size=(B * S, V))
        if np.min(np.abs(_softmax_T(zd, Td) - _softmax_T(zt, Tt))) > 1e-4:
            break
    wts = (0.7, 0.4, 1.3, 0.9)
    r = O.combined_loss(zd, zt, Td, Tt, wts, O.LAYOUT_SEQUENCES, B, S, K, grad_scale=1.0)
    h = 1e-6
    fd = np.zeros_like(zd)
    for i in range(zd.shape[0]):
        for v in range(V):
            zp = zd.copy()
            zm = zd.copy()
            zp[i, v] += h
            zm[i, v] -= h
            lp = O.combined_loss(zp, zt, Td, Tt, wts, O.LAYOUT_SEQUENCES, B, S, K)["loss"]
            lm = O.combined_loss(zm, zt, Td, Tt, wts, O.LAYOUT_SEQUENCES, B, S, K)["loss"]
            fd[i, v] = (lp - lm) / (2 * h)
    assert np.max(np.abs(r["grad"] - fd)) < 1e-8
    np.testing.assert_allclose(r["grad"].sum(-1), 0.0, atol=1e-15)


def test_labels_replace_the_greedy_token():
    rng = np.random.default_rng(25)
    B, S, K, V = 2, 4, 2, 6
    zt = rng.normal(size=(B * S, V))
    zd = rng.normal(size=(B * S, V))
    a = O.combined_loss(zd, zt, 1.0, 1.0, (0, 1, 0, 0), O.LAYOUT_SEQUENCES, B, S, K)
    b = O.combined_loss(zd, zt, 1.0, 1.0, (0, 1, 0, 0), O.LAYOUT_SEQUENCES, B, S, K, labels=np.argmax(zt, -1))
    np.testing.assert_array_equal(a["grad"], b["grad"])
    lab = rng.integers(0, V, size=B * S)
    c = O.combined_loss(zd, zt, 1.0, 1.0, (0, 1, 0, 0), O.LAYOUT_SEQUENCES, B, S, K, labels=lab)
    np.testing.assert_allclose(c["a_eal"], _softmax_T(zd, 1.0)[np.arange(B * S), lab], rtol=1e-14)
