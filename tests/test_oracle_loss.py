"""Pins of the oracle's clipped GRPO objective and its gradient (App. D.2)."""

import numpy as np
import pytest

from oracle.advantage import group_advantage
from oracle.loss import grpo_loss


def _batch(seed, n_seq=6, max_len=9):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, max_len + 1, n_seq)
    seq = np.concatenate([[i] * l for i, l in enumerate(lens)])
    T = len(seq)
    logp = -rng.random(T) * 5
    adv = rng.standard_normal(n_seq)
    return rng, lens, seq, logp, adv


def test_on_policy_identity():
    rng, lens, seq, logp, adv = _batch(0)
    n_seq = len(lens)
    loss, dlogp, st = grpo_loss(logp, logp, seq, adv, lens, n_seq)
    assert loss == pytest.approx(-adv.sum() / n_seq, rel=1e-13, abs=1e-15)
    want = np.array([-adv[s] / (n_seq * lens[s]) for s in seq])
    assert np.allclose(dlogp, want, rtol=1e-14, atol=0)
    assert st[0] == len(seq) and st[1] == 0 and st[2] == len(seq)


def test_whole_groups_of_equal_length_give_zero_loss_but_a_gradient():
    G, n_groups, L = 4, 3, 5
    rewards = np.array([1, 0, 0, 1, 1, 1, 0, 1, 0, 0, 0, 1], dtype=float)
    off = np.arange(0, G * n_groups + 1, G)
    adv = np.array(group_advantage(rewards, off))
    lens = np.full(G * n_groups, L)
    seq = np.repeat(np.arange(G * n_groups), L)
    logp = -np.ones(len(seq))
    loss, dlogp, _ = grpo_loss(logp, logp, seq, adv, lens, G * n_groups)
    assert abs(loss) < 1e-15
    assert np.abs(dlogp).max() > 0


@pytest.mark.parametrize("A,rho,active,term", [
    (1.0, 1.2 + 1e-3, False, 1.2),          # above the upper bound, A > 0: clipped
    (1.0, 1.2 - 1e-3, True, 1.2 - 1e-3),    # inside
    (1.0, 0.5, True, 0.5),                   # below the lower bound, A > 0: unclipped side
    (-1.0, 0.8 - 1e-3, False, -0.8),         # below the lower bound, A < 0: clipped
    (-1.0, 0.8 + 1e-3, True, -(0.8 + 1e-3)),
    (-1.0, 1.7, True, -1.7),                 # above the upper bound, A < 0: unclipped side
    (1.0, 1.2, True, 1.2),                   # exactly on the bound: closed interval
    (-1.0, 0.8, True, -0.8),
])
def test_clip_cases(A, rho, active, term):
    old = np.array([-2.0])
    logp = old + np.log(rho)
    seq = np.array([0])
    loss, dlogp, st = grpo_loss(logp, old, seq, np.array([A]), np.array([1]), 1)
    r = np.exp(logp[0] - old[0])
    assert -loss == pytest.approx(term, rel=1e-9)
    if active:
        assert dlogp[0] == pytest.approx(-A * r, rel=1e-12)
        assert st[1] == 0
    else:
        assert dlogp[0] == 0.0
        assert st[1] == 1


def test_finite_differences_away_from_kinks():
    rng, lens, seq, logp, adv = _batch(1, n_seq=8, max_len=12)
    old = logp + rng.normal(0, 0.3, len(seq))
    rho = np.exp(logp - old)
    # keep tokens at least 1e-3 away from both clip boundaries
    bad = (np.abs(rho - 0.8) < 1e-3) | (np.abs(rho - 1.2) < 1e-3)
    old[bad] += 0.01
    n_seq = 11
    _, dlogp, _ = grpo_loss(logp, old, seq, adv, lens, n_seq)
    h = 1e-7
    for t in range(len(seq)):
        e = np.zeros(len(seq))
        e[t] = h
        lp, _, _ = grpo_loss(logp + e, old, seq, adv, lens, n_seq)
        lm, _, _ = grpo_loss(logp - e, old, seq, adv, lens, n_seq)
        assert (lp - lm) / (2 * h) == pytest.approx(dlogp[t], rel=1e-6, abs=1e-10)


def test_micro_batches_add_up_and_mask_is_inert():
    rng, lens, seq, logp, adv = _batch(2, n_seq=10, max_len=20)
    old = logp + rng.normal(0, 0.2, len(seq))
    full, dfull, sfull = grpo_loss(logp, old, seq, adv, lens, 10)
    cut = len(seq) // 3
    a, da, sa = grpo_loss(logp[:cut], old[:cut], seq[:cut], adv, lens, 10)
    b, db, sb = grpo_loss(logp[cut:], old[cut:], seq[cut:], adv, lens, 10)
    assert a + b == pytest.approx(full, rel=1e-13, abs=1e-16)
    assert np.array_equal(np.concatenate([da, db]), dfull)
    assert np.allclose(sa + sb, sfull)
    seq_m = np.concatenate([seq, [-1, -1]])
    lp_m = np.concatenate([logp, [3.0, -9.0]])
    old_m = np.concatenate([old, [0.0, 5.0]])
    m, dm, sm = grpo_loss(lp_m, old_m, seq_m, adv, lens, 10)
    assert m == full and np.all(dm[-2:] == 0) and sm[2] == sfull[2]


def test_zero_advantage_contributes_nothing():
    rng, lens, seq, logp, adv = _batch(3)
    adv[:] = 0.0
    old = logp + 0.5
    loss, dlogp, _ = grpo_loss(logp, old, seq, adv, lens, len(lens))
    assert loss == 0.0 and np.all(dlogp == 0.0)


@pytest.mark.parametrize("A,rho,active,term", [
    (1.0, 1.3 + 1e-3, False, 1.3),          # above 1 + eps_high, A > 0: clipped
    (1.0, 1.25, True, 1.25),                 # inside (outside if the bounds were swapped)
    (1.0, 0.85, True, 0.85),                 # below 1 - eps_low, A > 0: unclipped side
    (-1.0, 0.9 - 1e-3, False, -0.9),         # below 1 - eps_low, A < 0: clipped
    (-1.0, 0.75, False, -0.9),               # (inside if the bounds were swapped)
    (-1.0, 0.95, True, -0.95),               # inside
    (-1.0, 1.4, True, -1.4),                 # above 1 + eps_high, A < 0: unclipped side
])
def test_asymmetric_clip_range(A, rho, active, term):
    """eps_low = 0.1, eps_high = 0.3: the lower bound is 0.9, the upper 1.3,
    so a mistake that swaps or merges the two ranges changes these cases."""
    old = np.array([-2.0])
    logp = old + np.log(rho)
    loss, dlogp, st = grpo_loss(logp, old, np.array([0]), np.array([A]), np.array([1]), 1,
                                eps_low=0.1, eps_high=0.3)
    r = np.exp(logp[0] - old[0])
    assert -loss == pytest.approx(term, rel=1e-9)
    if active:
        assert dlogp[0] == pytest.approx(-A * r, rel=1e-12)
        assert st[1] == 0
    else:
        assert dlogp[0] == 0.0
        assert st[1] == 1
