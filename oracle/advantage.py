"""Group-normalised advantage, computed when a group of rollouts is inserted.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

App. D.2: for each prompt the workers generate a group of G rollouts; rollout i
gets A_i = (r_i - mean of the group's rewards) / (std of the group's rewards),
computed at generation time and stored with the rollout (not recomputed when
the rollout is replayed).

The paper says only "std".  The standard deviation uses ``ddof``
(default 1, the sample estimate), ``eps`` (default 1e-6) is added to it, and a
group whose rewards are all equal (std exactly 0, which includes G = 1) gets
A = 0 exactly.

Parity: pinned by closed forms (binary rewards with k of G correct), the
zero-sum property of every group, and the all-equal case --
tests/test_oracle_advantage.py.
"""

import math


def group_advantage(rewards, group_off, ddof=1, eps=1e-6):
    """Advantages for groups ``[group_off[g], group_off[g+1])`` of ``rewards``.

    Plain loops in Python floats (fp64).
    """
    adv = [0.0] * len(rewards)
    for g in range(len(group_off) - 1):
        lo, hi = int(group_off[g]), int(group_off[g + 1])
        n = hi - lo
        if n <= 0:
            continue
        # identical rewards have std 0 by definition; decided on the rewards
        # themselves, since the fp64 mean of e.g. three 0.7s is not 0.7
        equal = all(float(rewards[i]) == float(rewards[lo]) for i in range(lo, hi))
        mean = sum(float(rewards[i]) for i in range(lo, hi)) / n
        ss = sum((float(rewards[i]) - mean) ** 2 for i in range(lo, hi))
        if equal or ss == 0.0 or n - ddof <= 0:
            # identical rewards (or no degrees of freedom): no signal
            for i in range(lo, hi):
                adv[i] = 0.0
            continue
        std = math.sqrt(ss / (n - ddof))
        for i in range(lo, hi):
            adv[i] = (float(rewards[i]) - mean) / (std + eps)
    return adv
