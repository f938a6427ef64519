"""Pins of the oracle's objective variants: AsymRE (App. D.2) and the
whole-sequence-ratio form of the clipped objective."""

import numpy as np
import pytest

from oracle.loss import asymre_coef, asymre_loss, grpo_loss, grpo_seq_loss


def _packed(seed, n_seq=5, max_len=7):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, max_len + 1, n_seq)
    cu = np.concatenate([[0], np.cumsum(lens)])
    seq = np.repeat(np.arange(n_seq), lens)
    return rng, lens, cu, seq


# ---- AsymRE ------------------------------------------------------------------

def test_asymre_coef_group_sum_fixes_the_sign_of_delta_v():
    # within a group, sum_i (r_i - V_hat) = 0, so sum_i c_i = -G * delta_V:
    # with the paper's delta_V = -0.1 every group's coefficients add to +0.1 G
    rewards = [1, 0, 0, 1, 1, 1, 1, 0, 0]
    off = [0, 4, 6, 9]
    c = asymre_coef(rewards, off, delta_v=-0.1)
    for g in range(3):
        lo, hi = off[g], off[g + 1]
        assert sum(c[lo:hi]) == pytest.approx(0.1 * (hi - lo), abs=1e-14)
    # a correct rollout in a half-correct group of 4: 1 - 0.5 + 0.1
    assert c[0] == pytest.approx(0.6, abs=1e-15)
    assert c[1] == pytest.approx(-0.4, abs=1e-15)


def test_asymre_gradient_is_constant_per_sequence_and_matches_finite_differences():
    rng, lens, cu, seq = _packed(1)
    n_seq = len(lens)
    coef = rng.standard_normal(n_seq)
    logp = -rng.random(len(seq)) * 4
    loss, dlogp, st = asymre_loss(logp, seq, coef, n_seq)
    for i in range(n_seq):
        block = dlogp[cu[i]:cu[i + 1]]
        assert np.all(block == block[0])
    h = 1e-6
    for t in range(len(seq)):
        e = np.zeros_like(logp)
        e[t] = h
        fd = (asymre_loss(logp + e, seq, coef, n_seq)[0]
              - asymre_loss(logp - e, seq, coef, n_seq)[0]) / (2 * h)
        assert fd == pytest.approx(dlogp[t], rel=1e-7, abs=1e-10)
    assert st[0] == len(seq)


def test_asymre_shift_identity_and_masking():
    # adding k to every log-prob of sequence i (its probability scaled by e^k
    # per token) changes the loss by -c_i * k * len_i / n_seq; masked tokens
    # take no part
    rng, lens, cu, seq = _packed(2)
    n_seq = len(lens)
    coef = rng.standard_normal(n_seq)
    logp = -rng.random(len(seq)) * 4
    base = asymre_loss(logp, seq, coef, n_seq)[0]
    for i in range(n_seq):
        sh = logp.copy()
        sh[cu[i]:cu[i + 1]] += 0.7
        got = asymre_loss(sh, seq, coef, n_seq)[0] - base
        assert got == pytest.approx(-coef[i] * 0.7 * lens[i] / n_seq, rel=1e-12)
    masked = np.where(np.arange(len(seq)) % 3 == 0, -1, seq)
    l2, d2, st2 = asymre_loss(logp, masked, coef, n_seq)
    assert np.all(d2[masked < 0] == 0) and st2[0] == np.sum(masked >= 0)


def test_asymre_equal_rewards_without_offset_give_no_signal():
    c = asymre_coef([1, 1, 1, 1], [0, 4], delta_v=0.0)
    assert c == [0.0, 0.0, 0.0, 0.0]


# ---- whole-sequence ratio --------------------------------------------------

def test_seq_ratio_on_policy_identity():
    rng, lens, cu, seq = _packed(3)
    n_seq = len(lens)
    adv = rng.standard_normal(n_seq)
    logp = -rng.random(len(seq)) * 3
    loss, dlogp, st = grpo_seq_loss(logp, logp, cu, adv, n_seq)
    assert loss == pytest.approx(-adv.sum() / n_seq, rel=1e-13)
    assert np.allclose(dlogp, -adv[seq] / n_seq, rtol=1e-14, atol=0)
    assert st[0] == pytest.approx(n_seq) and st[1] == 0 and st[2] == n_seq


def test_seq_ratio_reduces_to_token_ratio_for_one_token_sequences():
    rng = np.random.default_rng(4)
    n = 12
    cu = np.arange(n + 1)
    seq = np.arange(n)
    adv = rng.standard_normal(n)
    logp = -rng.random(n) * 3
    old = logp + rng.normal(0, 0.3, n)
    a = grpo_seq_loss(logp, old, cu, adv, n)
    b = grpo_loss(logp, old, seq, adv, np.ones(n), n)
    assert a[0] == pytest.approx(b[0], rel=1e-13)
    assert np.allclose(a[1], b[1], rtol=1e-13, atol=0)


def test_seq_ratio_clip_uses_the_product_of_token_ratios():
    # two tokens with log-ratios 0.15 each: rho = e^0.3 = 1.35 > 1.2
    logp = np.array([-1.0, -2.0])
    old = logp - 0.15
    cu = [0, 2]
    _, d_pos, st_pos = grpo_seq_loss(logp, old, cu, [1.0], 1)
    assert np.all(d_pos == 0) and st_pos[1] == 1          # clipped, A > 0
    _, d_neg, st_neg = grpo_seq_loss(logp, old, cu, [-1.0], 1)
    assert np.allclose(d_neg, np.exp(0.3))                 # unclipped, A < 0
    # per token each ratio (e^0.15 = 1.16) is inside the clip range
    _, d_tok, _ = grpo_loss(logp, old, [0, 0], [1.0], [2], 1)
    assert np.all(d_tok != 0)


def test_seq_ratio_matches_finite_differences_away_from_kinks():
    rng, lens, cu, seq = _packed(5, n_seq=6, max_len=5)
    n_seq = len(lens)
    adv = rng.standard_normal(n_seq)
    logp = -rng.random(len(seq)) * 3
    old = logp + rng.normal(0, 0.04, len(seq))
    loss, dlogp, _ = grpo_seq_loss(logp, old, cu, adv, n_seq)
    h = 1e-6
    for t in range(len(seq)):
        e = np.zeros_like(logp)
        e[t] = h
        fd = (grpo_seq_loss(logp + e, old, cu, adv, n_seq)[0]
              - grpo_seq_loss(logp - e, old, cu, adv, n_seq)[0]) / (2 * h)
        assert fd == pytest.approx(dlogp[t], rel=1e-6, abs=1e-10)


def test_seq_ratio_asymmetric_clip_range():
    """eps_low = 0.1, eps_high = 0.3: a sequence ratio of e^0.25 = 1.28 lies
    inside (it would be clipped with the bounds swapped), one of e^0.3 = 1.35
    above; e^-0.2 = 0.82 lies below the lower bound 0.9."""
    logp = np.array([-1.0, -2.0])
    cu = [0, 2]
    for shift, A, clipped in ((0.125, 1.0, False), (0.15, 1.0, True), (-0.1, -1.0, True),
                              (-0.1, 1.0, False)):
        old = logp - shift
        rho = np.exp(2 * shift)
        loss, d, st = grpo_seq_loss(logp, old, cu, [A], 1, eps_low=0.1, eps_high=0.3)
        if clipped:
            assert np.all(d == 0) and st[1] == 1
            bound = 1.3 if A > 0 else 0.9
            assert -loss == pytest.approx(bound * A, rel=1e-12)
        else:
            assert np.allclose(d, -A * rho, rtol=1e-12) and st[1] == 0
            assert -loss == pytest.approx(rho * A, rel=1e-12)
