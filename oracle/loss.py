"""Clipped, importance-weighted GRPO objective for replayed (stale) samples.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

App. D.2 states the objective: the expectation of
min(rho * A, clip(rho, 1 - eps_low, 1 + eps_high) * A), with rho the ratio of
the current policy's probability of the rollout to the probability recorded
when the rollout was generated, A the rollout's group advantage (stored at
generation), eps_low = eps_high = 0.2 and no KL term.

Readings (each listed in the design notes):

* R1 -- the ratio is taken per token, rho_t = exp(logp_t - old_logp_t), and
  each sequence contributes the mean of its token terms (the GRPO form the
  paper cites); a whole-sequence ratio is a different objective.
* R2 -- sequence i is weighted 1 / (n_seq * len_i): len_i is its full length
  (also when a micro-batch holds only part of it), n_seq the number of sampled
  sequences in the optimizer batch (duplicated draws count twice).
* R3 -- the paper maximises J; ``loss = -J`` and all gradients are of ``loss``.
* R4 -- the gradient of a token term is rho*A when the unclipped branch is
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
and central finite differences -- tests/test_oracle_loss.py.
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
