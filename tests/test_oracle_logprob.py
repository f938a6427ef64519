"""Pins of the oracle's per-token log-probabilities."""

import math

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle.logprob import entropy, logprob, logprob_rows


def _inputs(T, d, V, seed, w_std=0.5):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((T, d))
    W = rng.standard_normal((V, d)) * w_std
    y = rng.integers(0, V, T)
    return h, W, y


def test_normalisation_over_the_vocabulary():
    h, W, y = _inputs(20, 16, 300, 0)
    _, lse = logprob(h, W, y)
    z = h @ W.T
    total = np.exp(z - lse[:, None]).sum(axis=1)
    assert np.allclose(total, 1.0, rtol=0, atol=1e-12)


def test_zero_weight_gives_uniform():
    h, W, y = _inputs(7, 8, 1000, 1)
    logp, lse = logprob(h, np.zeros_like(W), y)
    assert np.allclose(logp, -math.log(1000), rtol=0, atol=1e-13)
    assert np.allclose(lse, math.log(1000), rtol=0, atol=1e-13)


def test_single_token_vocabulary():
    h, W, y = _inputs(5, 8, 1, 2)
    logp, lse = logprob(h, W, y)
    assert np.all(logp == 0.0)
    assert np.allclose(lse, (h @ W.T)[:, 0], rtol=0, atol=1e-12)


def test_against_scipy_logsumexp():
    h, W, y = _inputs(33, 24, 517, 3, w_std=2.0)  # peaked logits
    logp, lse = logprob(h, W, y, chunk=8)
    z = h @ W.T
    assert np.allclose(lse, logsumexp(z, axis=1), rtol=1e-14, atol=1e-12)
    assert np.allclose(logp, z[np.arange(33), y] - logsumexp(z, axis=1),
                       rtol=1e-13, atol=1e-12)


def test_pure_python_brute_force_tiny():
    h, W, y = _inputs(3, 4, 6, 4)
    logp, lse = logprob(h, W, y)
    for t in range(3):
        zs = [sum(W[v][k] * h[t][k] for k in range(4)) for v in range(6)]
        want = zs[y[t]] - math.log(sum(math.exp(z) for z in zs))
        assert logp[t] == pytest.approx(want, abs=1e-13)


def test_chunking_and_row_spot_checks_agree():
    h, W, y = _inputs(50, 16, 200, 5)
    a, la = logprob(h, W, y, chunk=7)
    b, lb = logprob(h, W, y, chunk=1000)
    assert np.allclose(a, b, rtol=0, atol=1e-13)
    rows = [0, 13, 49]
    c, lc = logprob_rows(h, W, y, rows)
    assert np.allclose(c, a[rows], rtol=0, atol=1e-12)
    assert np.allclose(lc, la[rows], rtol=0, atol=1e-12)


def test_mask_zeroes_outputs():
    h, W, y = _inputs(6, 8, 50, 6)
    seq = np.array([0, 0, -1, 1, -1, 1])
    logp, lse = logprob(h, W, y, seq)
    assert np.all(logp[seq < 0] == 0) and np.all(lse[seq < 0] == 0)
    full, _ = logprob(h, W, y)
    assert np.array_equal(logp[seq >= 0], full[seq >= 0])


def test_shift_invariance_in_a_direction_shared_by_all_rows_of_W():
    # adding the same vector c to every row of W shifts all logits of a token
    # by c.h, leaving logp unchanged
    h, W, y = _inputs(10, 12, 40, 7)
    c = np.random.default_rng(8).standard_normal(12)
    a, _ = logprob(h, W, y)
    b, _ = logprob(h, W + c[None, :], y)
    assert np.allclose(a, b, rtol=0, atol=1e-11)


# ---- entropy ----------------------------------------------------------------

def test_entropy_of_uniform_logits_is_log_v():
    h, W, _ = _inputs(5, 8, 37, 11)
    assert np.allclose(entropy(h, np.zeros_like(W)), math.log(37), rtol=0, atol=1e-13)


def test_entropy_two_logits_is_binary_entropy_of_a_sigmoid():
    # z = (a, 0): p = sigmoid(a), H = -p ln p - (1 - p) ln(1 - p)
    a = np.array([-3.0, -0.5, 0.0, 0.7, 4.0])
    h = a[:, None]
    W = np.array([[1.0], [0.0]])
    p = 1.0 / (1.0 + np.exp(-a))
    want = -(p * np.log(p) + (1 - p) * np.log(1 - p))
    assert np.allclose(entropy(h, W), want, rtol=1e-13, atol=0)


def test_entropy_matches_scipy_and_its_bounds():
    from scipy.stats import entropy as scipy_entropy
    h, W, _ = _inputs(40, 16, 300, 12, w_std=0.4)
    z = h @ W.T
    p = np.exp(z - z.max(axis=1, keepdims=True))
    want = np.array([scipy_entropy(row) for row in p])  # normalises, uses ln
    got = entropy(h, W, chunk=7)
    assert np.allclose(got, want, rtol=1e-12, atol=0)
    assert np.all(got >= 0) and np.all(got <= math.log(300) + 1e-12)


def test_entropy_of_a_peaked_distribution_and_masking():
    # one logit 30 above three zeros: H = ln(1 + 3e^-30) + 90 e^-30 / (1 + 3e^-30)
    h = np.array([[1.0], [1.0]])
    W = np.array([[30.0], [0.0], [0.0], [0.0]])
    e = math.exp(-30.0)
    want = math.log1p(3 * e) + 90 * e / (1 + 3 * e)
    got = entropy(h, W, seq_of_token=[0, -1])
    assert got[0] == pytest.approx(want, rel=1e-9) and got[1] == 0.0
