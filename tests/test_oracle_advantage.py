"""Pins of the oracle's group-normalised advantage (App. D.2)."""

import math

import numpy as np
import pytest

from oracle.advantage import group_advantage


@pytest.mark.parametrize("G", [2, 4, 8, 16])
def test_binary_rewards_closed_form(G):
    # k of G correct: mean k/G; sample std s = sqrt(k (G-k) / (G (G-1)))
    for k in range(G + 1):
        r = [1.0] * k + [0.0] * (G - k)
        adv = group_advantage(r, [0, G], ddof=1, eps=0.0)
        if k in (0, G):
            assert adv == [0.0] * G
            continue
        s = math.sqrt(k * (G - k) / (G * (G - 1)))
        for i in range(G):
            want = (1 - k / G) / s if r[i] > 0 else -(k / G) / s
            assert adv[i] == pytest.approx(want, rel=1e-13, abs=1e-13)


def test_population_std_closed_form():
    # ddof = 0: binary group with k of G correct has std sqrt(f (1 - f))
    G, k = 8, 3
    f = k / G
    r = [1.0] * k + [0.0] * (G - k)
    adv = group_advantage(r, [0, G], ddof=0, eps=0.0)
    s = math.sqrt(f * (1 - f))
    assert adv[0] == pytest.approx((1 - f) / s, rel=1e-13)
    assert adv[-1] == pytest.approx(-f / s, rel=1e-13)


def test_groups_sum_to_zero_and_are_independent():
    rng = np.random.default_rng(0)
    sizes = rng.integers(1, 12, 40)
    off = np.concatenate([[0], np.cumsum(sizes)])
    r = rng.standard_normal(int(off[-1]))
    adv = group_advantage(r, off)
    for g in range(40):
        a = adv[off[g]:off[g + 1]]
        assert abs(sum(a)) < 1e-12 * max(1.0, max(abs(x) for x in a))
        # a group's advantages do not depend on other groups
        alone = group_advantage(r[off[g]:off[g + 1]], [0, int(sizes[g])])
        assert alone == a


def test_all_equal_and_singleton_groups_are_zero():
    assert group_advantage([0.5] * 5, [0, 5]) == [0.0] * 5
    assert group_advantage([1.0], [0, 1]) == [0.0]
    assert group_advantage([1.0, 1.0, 0.0, 0.0], [0, 2, 4]) == [0.0] * 4


def test_affine_invariance_of_rewards():
    # A is unchanged by r -> a r + b with a > 0 (eps = 0)
    rng = np.random.default_rng(1)
    r = rng.standard_normal(16)
    base = group_advantage(r, [0, 16], eps=0.0)
    moved = group_advantage(3.0 * r + 7.0, [0, 16], eps=0.0)
    assert np.allclose(base, moved, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("G", [2, 3, 4, 7, 8, 16])
@pytest.mark.parametrize("r", [0.7, 0.1, 1.0 / 3.0, -2.5, float(np.float32(0.7))])
def test_equal_non_binary_rewards_are_exactly_zero(G, r):
    # identical rewards have std 0 whatever their binary expansion: the fp64
    # mean of three 0.7s is not 0.7, so the decision cannot rest on the spread
    assert group_advantage([r] * G, [0, G]) == [0.0] * G
    assert group_advantage([r] * G, [0, G], ddof=0) == [0.0] * G


@pytest.mark.parametrize("G", [2, 4, 8, 16])
@pytest.mark.parametrize("x, ulps", [(0.7, 1), (0.1, 3), (1.0 / 3.0, 1000), (5.0, 2 ** 20)])
def test_one_outlier_closed_form(G, x, ulps):
    # G - 1 rewards x and one x + delta: mean x + delta/G, deviations
    # -delta/G and delta (G-1)/G, sample std |delta| / sqrt(G).  Evaluated in
    # exact rationals from the two floats, so eps matters when delta is a few
    # ulps of x (std ~ 1e-16 against eps = 1e-6).
    from fractions import Fraction
    import math as m

    y = float(np.nextafter(np.float32(x), np.float32(np.inf)))  # keep in fp32 range
    for _ in range(ulps - 1):
        y = float(np.nextafter(np.float32(y), np.float32(np.inf)))
    x = float(np.float32(x))
    delta = Fraction(y) - Fraction(x)
    eps = 1e-6
    std = float(abs(delta)) / m.sqrt(G)
    hi = float(delta * (G - 1) / G) / (std + eps)
    lo = float(-delta / G) / (std + eps)
    adv = group_advantage([x] * (G - 1) + [y], [0, G], ddof=1, eps=eps)
    assert adv[-1] == pytest.approx(hi, rel=1e-9)
    for a in adv[:-1]:
        assert a == pytest.approx(lo, rel=1e-9)
