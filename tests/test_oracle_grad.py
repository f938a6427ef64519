"""Pins of the oracle's backward to hidden states and LM head."""

import numpy as np
import pytest

from oracle.grad import dW_from_rows, dhidden_rows, dz_rows, logprob_backward
from oracle.logprob import logprob
from oracle.loss import grpo_loss


def _setup(seed, T=12, d=6, V=40, w_std=0.4):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((T, d))
    W = rng.standard_normal((V, d)) * w_std
    y = rng.integers(0, V, T)
    lens = np.array([5, 4, 3])
    seq = np.concatenate([[i] * l for i, l in enumerate(lens)])[:T]
    adv = np.array([0.9, -1.3, 0.4])
    logp0, _ = logprob(h, W, y)
    old = logp0 + rng.normal(0, 0.05, T)
    return h, W, y, seq, adv, lens, old


def _composite(h, W, y, seq, adv, lens, old):
    logp, _ = logprob(h, W, y, seq)
    loss, _, _ = grpo_loss(logp, old, seq, adv, lens, 3)
    return loss


def test_finite_differences_of_the_whole_path():
    h, W, y, seq, adv, lens, old = _setup(0)
    logp, lse = logprob(h, W, y, seq)
    _, dlogp, _ = grpo_loss(logp, old, seq, adv, lens, 3)
    rho = np.exp(logp - old)
    assert np.all((np.abs(rho - 0.8) > 1e-3) & (np.abs(rho - 1.2) > 1e-3))
    dh, dW = logprob_backward(h, W, y, lse, dlogp, seq)
    eps = 1e-6
    for (t, k) in [(0, 0), (3, 5), (7, 2), (11, 4)]:
        hp, hm = h.copy(), h.copy()
        hp[t, k] += eps
        hm[t, k] -= eps
        fd = (_composite(hp, W, y, seq, adv, lens, old)
              - _composite(hm, W, y, seq, adv, lens, old)) / (2 * eps)
        assert fd == pytest.approx(dh[t, k], rel=1e-6, abs=1e-11)
    for (v, k) in [(int(y[0]), 1), (0, 0), (17, 3), (39, 5)]:
        Wp, Wm = W.copy(), W.copy()
        Wp[v, k] += eps
        Wm[v, k] -= eps
        fd = (_composite(h, Wp, y, seq, adv, lens, old)
              - _composite(h, Wm, y, seq, adv, lens, old)) / (2 * eps)
        assert fd == pytest.approx(dW[v, k], rel=1e-6, abs=1e-11)


def test_columns_of_dW_sum_to_zero():
    h, W, y, seq, adv, lens, old = _setup(1, T=30, V=100)
    rng = np.random.default_rng(9)
    _, lse = logprob(h, W, y)
    dlogp = rng.standard_normal(30)
    _, dW = logprob_backward(h, W, y, lse, dlogp)
    assert np.allclose(dW.sum(axis=0), 0.0, atol=1e-12 * np.abs(dW).max())


def test_dhidden_closed_form():
    h, W, y, seq, adv, lens, old = _setup(2)
    rng = np.random.default_rng(10)
    _, lse = logprob(h, W, y)
    dlogp = rng.standard_normal(len(y))
    dh, _ = logprob_backward(h, W, y, lse, dlogp)
    for t in range(len(y)):
        z = W @ h[t]
        p = np.exp(z - z.max())
        p /= p.sum()
        want = dlogp[t] * (W[y[t]] - p @ W)
        assert np.allclose(dh[t], want, rtol=1e-12, atol=1e-14)


def test_linearity_in_dlogp_and_mask():
    h, W, y, seq, adv, lens, old = _setup(3)
    rng = np.random.default_rng(11)
    _, lse = logprob(h, W, y)
    a = rng.standard_normal(len(y))
    b = rng.standard_normal(len(y))
    dha, dWa = logprob_backward(h, W, y, lse, a)
    dhb, dWb = logprob_backward(h, W, y, lse, b)
    dhc, dWc = logprob_backward(h, W, y, lse, 2 * a - b)
    assert np.allclose(dhc, 2 * dha - dhb, atol=1e-12)
    assert np.allclose(dWc, 2 * dWa - dWb, atol=1e-12)
    seq_m = np.array(seq)
    seq_m[[1, 4]] = -1
    dhm, dWm = logprob_backward(h, W, y, lse, a, seq_m)
    a2 = a.copy()
    a2[[1, 4]] = 0
    dh2, dW2 = logprob_backward(h, W, y, lse, a2)
    assert np.all(dhm[[1, 4]] == 0)
    assert np.array_equal(dWm, dW2)


def test_row_helpers_match_full_backward():
    h, W, y, seq, adv, lens, old = _setup(4, T=20, V=64)
    rng = np.random.default_rng(12)
    _, lse = logprob(h, W, y)
    dlogp = np.zeros(20)
    rows = [2, 7, 19]
    dlogp[rows] = rng.standard_normal(3)
    dh, dW = logprob_backward(h, W, y, lse, dlogp)
    assert np.allclose(dhidden_rows(h, W, y, lse, dlogp, rows), dh[rows], atol=1e-13)
    assert np.allclose(dW_from_rows(h, W, y, lse, dlogp, rows), dW, atol=1e-13)
    assert np.allclose(dW_from_rows(h, W, y, lse, dlogp, rows, 10, 30), dW[10:30],
                       atol=1e-13)
    dz = dz_rows(h, W, y, lse, dlogp, rows)
    assert np.allclose(dz.sum(axis=1), 0.0, atol=1e-14)
    assert np.allclose(dW_from_rows(h, W, y, lse, dlogp, rows, 5, 9, dz=dz), dW[5:9],
                       atol=1e-13)
