"""Clipped, importance-weighted GRPO objective for replayed (stale) samples.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

App. D.2 states the objective: the expectation of
min(rho * A, clip(rho, 1 - eps_low, 1 + eps_high) * A), with rho the ratio of
the current policy's probability of the rollout to the probability recorded
when the rollout was generated, A the rollout's group advantage (stored at
generation), eps_low = eps_high = 0.2 and no KL term.

Where the paper leaves a choice open:

* ratio level -- the ratio is taken per token, rho_t = exp(logp_t - old_logp_t), and
  each sequence contributes the mean of its token terms (the GRPO form the
  paper cites); a whole-sequence ratio is a different objective.
* normalisation -- sequence i is weighted 1 / (n_seq * len_i): len_i is its full length
  (also when a micro-batch holds only part of it), n_seq the number of sampled
  sequences in the optimizer batch (duplicated draws count twice).
* sign -- the paper maximises J; ``loss = -J`` and all gradients are of ``loss``.
* clip gradient -- the gradient of a token term is rho*A when the unclipped branch is
  taken or the ratio lies inside [1 - eps_low, 1 + eps_high] (closed), and 0
  when the clipped branch is taken strictly outside it:
  act_t = 0 iff (A > 0 and rho > 1 + eps_high) or (A < 0 and rho < 1 - eps_low).

So, for token t of sequence i,
    l_t      = min(rho_t A_i, clip(rho_t, 1 - eps_low, 1 + eps_high) A_i)
    J        = sum_t l_t / (n_seq len_i)
    dlogp_t  = d(-J)/d logp_t = -A_i rho_t act_t / (n_seq len_i).
Masked tokens (seq_of_token < 0) contribute nothing and get dlogp = 0.

Parity: pinned by the on-policy identity (old = current gives rho = 1,
loss = -(1/n_seq) sum_i A_i and dlogp_t = -A_i / (n_seq len_i)), zero loss on
whole groups with equal lengths, the clip cases on both sides of each boundary,
and central finite differences -- tests/test_oracle_loss.py.  The two variants
at the end of this module (AsymRE, whole-sequence ratio) are pinned by finite
differences, the sign of delta_V through the group sum of the coefficients,
shift identities, the on-policy identity and, for one-token sequences, by the
token-level objective above -- tests/test_oracle_loss_variants.py.
"""

import numpy as np


def grpo_loss(logp, old_logp, seq_of_token, adv, seq_len, n_seq, eps_low=0.2,
              eps_high=0.2):
    """Return (loss, dlogp [T], stats) in fp64.

    stats = [sum of rho over valid tokens, number of tokens on a clipped branch
    with zero gradient, number of valid tokens, sum of the unweighted l_t].
    """
    logp = np.asarray(logp, dtype=np.float64)
    old = np.asarray(old_logp, dtype=np.float64)
    seq = np.asarray(seq_of_token, dtype=np.int64)
    adv = np.asarray(adv, dtype=np.float64)
    seq_len = np.asarray(seq_len, dtype=np.float64)
    valid = seq >= 0
    s = np.where(valid, seq, 0)
    A = np.where(valid, adv[s], 0.0)
    L = np.where(valid, seq_len[s], 1.0)
    rho = np.where(valid, np.exp(logp - old), 0.0)
    unclipped = rho * A
    clipped = np.clip(rho, 1.0 - eps_low, 1.0 + eps_high) * A
    term = np.minimum(unclipped, clipped)
    cut = ((A > 0) & (rho > 1.0 + eps_high)) | ((A < 0) & (rho < 1.0 - eps_low))
    weight = np.where(valid, 1.0 / (float(n_seq) * L), 0.0)
    J = float(np.sum(term * weight))
    dlogp = np.where(valid & ~cut, -A * rho * weight, 0.0)
    stats = np.array([
        float(np.sum(rho[valid])),
        float(np.sum(cut & valid)),
        float(np.sum(valid)),
        float(np.sum(term[valid])),
    ])
    return -J, dlogp, stats


# ---- objective variants (the paper's AsymRE; a whole-sequence ratio) -------
#
# AsymRE (App. D.2): J = E[(1/G) sum_i (r_i - (V_hat + delta_V)) log pi(z_i|q)],
# V_hat the mean reward of rollout i's group (known at generation), delta_V =
# -0.1, log pi(z|q) the sum of the rollout's token log-probabilities.
# Readings (design notes R13, R15): the per-rollout coefficient
# c_i = r_i - V_hat_g - delta_V is stored at insert like the GRPO advantage;
# the group average over G becomes the average over the n_seq sampled
# rollouts of the optimizer batch (as for GRPO); no ratio, no clip, no
# per-token length normalisation (log pi is a sum over the rollout's tokens).
#
# Sequence-ratio GRPO (the printed formula taken literally): rho_i =
# pi(z_i|q) / pi_old(z_i|q) = exp(sum_{t in i} (logp_t - old_logp_t)),
# J = (1/n_seq) sum_i min(rho_i A_i, clip(rho_i, 1 - eps_low, 1 + eps_high) A_i),
# with the clip-gradient rule above applied to rho_i.  The sum runs over the
# whole rollout, so a call must hold complete sequences (given by cu_seqlens).


def asymre_coef(rewards, group_off, delta_v=-0.1):
    """c_i = r_i - (mean reward of i's group + delta_v), plain loops in fp64."""
    c = [0.0] * len(rewards)
    for g in range(len(group_off) - 1):
        lo, hi = int(group_off[g]), int(group_off[g + 1])
        if hi <= lo:
            continue
        v_hat = sum(float(rewards[i]) for i in range(lo, hi)) / (hi - lo)
        for i in range(lo, hi):
            c[i] = float(rewards[i]) - (v_hat + float(delta_v))
    return c


def asymre_loss(logp, seq_of_token, coef, n_seq):
    """Return (loss, dlogp [T], stats) in fp64 for the AsymRE objective.

    loss = -(1/n_seq) sum_t c_{s(t)} logp_t over valid tokens; dlogp_t =
    -c_{s(t)} / n_seq; stats = [number of valid tokens, sum_t c_{s(t)} logp_t].
    """
    logp = np.asarray(logp, dtype=np.float64)
    seq = np.asarray(seq_of_token, dtype=np.int64)
    coef = np.asarray(coef, dtype=np.float64)
    valid = seq >= 0
    c = np.where(valid, coef[np.where(valid, seq, 0)], 0.0)
    s = float(np.sum(c * logp))
    loss = -s / float(n_seq)
    dlogp = np.where(valid, -c / float(n_seq), 0.0)
    return loss, dlogp, np.array([float(np.sum(valid)), s])


def grpo_seq_loss(logp, old_logp, cu_seqlens, adv, n_seq, eps_low=0.2, eps_high=0.2):
    """Return (loss, dlogp [T], stats) in fp64 for the whole-sequence ratio.

    Sequence i holds tokens [cu_seqlens[i], cu_seqlens[i+1]); tokens outside
    every sequence get dlogp = 0.  stats = [sum_i rho_i, number of sequences
    on a clipped branch with zero gradient, number of sequences, sum_i l_i].
    """
    logp = np.asarray(logp, dtype=np.float64)
    old = np.asarray(old_logp, dtype=np.float64)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    adv = np.asarray(adv, dtype=np.float64)
    dlogp = np.zeros_like(logp)
    J = 0.0
    st = np.zeros(4)
    for i in range(len(cu) - 1):
        lo, hi = int(cu[i]), int(cu[i + 1])
        rho = float(np.exp(np.sum(logp[lo:hi] - old[lo:hi])))
        A = float(adv[i])
        term = min(rho * A, min(max(rho, 1.0 - eps_low), 1.0 + eps_high) * A)
        cut = (A > 0 and rho > 1.0 + eps_high) or (A < 0 and rho < 1.0 - eps_low)
        J += term / float(n_seq)
        if not cut:
            dlogp[lo:hi] = -A * rho / float(n_seq)
        st += [rho, 1.0 if cut else 0.0, 1.0, term]
    return -J, dlogp, st
