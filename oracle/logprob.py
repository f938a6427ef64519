"""Per-token policy log-probabilities from final hidden states and the LM head.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The objective of App. D.2 needs pi_theta(z|q) of replayed tokens under the
current policy.  With an untied LM head W (App. D.2 trains without weight
tying) and temperature 1 (App. D.2), token t with hidden state h_t and sampled
token y_t has logits z_t = W h_t and

    lse_t  = log sum_v exp(z_{t,v})
    logp_t = z_{t,y_t} - lse_t.

Plain definition in fp64: the logits of a chunk of tokens are one matmul, the
log-sum-exp shifts by the row maximum.  Chunking over tokens only bounds the
memory of the fp64 logits; it changes no arithmetic.  Masked tokens
(seq_of_token < 0) get logp = 0 and lse = 0.

Per-token entropy of the policy, H_t = -sum_v p_{t,v} log p_{t,v} with
p_t = softmax(z_t): the training entropy the paper reports alongside accuracy
(App. E, the test / train / entropy dynamics figure), measured on the batches
the trainer updates on.  Written from the definition with log p = z - lse.

Parity: pinned by normalisation (sum_v exp(z_v - lse) = 1), W = 0 (logp = -ln V
exactly), V = 1 (logp = 0), a cross-check against scipy's logsumexp and a
pure-Python brute force on tiny inputs; the entropy by W = 0 (ln V), the
two-logit closed form (binary entropy of a sigmoid), scipy.stats.entropy of the
softmax and its bounds -- tests/test_oracle_logprob.py.
"""

import numpy as np


def logits(hidden, W):
    """z = hidden @ W^T in fp64 (hidden [T, d], W [V, d])."""
    return np.asarray(hidden, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def logprob(hidden, W, tokens, seq_of_token=None, chunk=512):
    """Return (logp [T], lse [T]) in fp64."""
    hidden = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    tokens = np.asarray(tokens, dtype=np.int64)
    T = hidden.shape[0]
    logp = np.zeros(T, dtype=np.float64)
    lse = np.zeros(T, dtype=np.float64)
    for a in range(0, T, chunk):
        b = min(a + chunk, T)
        z = hidden[a:b] @ W.T
        m = z.max(axis=1)
        lse[a:b] = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        logp[a:b] = z[np.arange(b - a), tokens[a:b]] - lse[a:b]
    if seq_of_token is not None:
        masked = np.asarray(seq_of_token) < 0
        logp[masked] = 0.0
        lse[masked] = 0.0
    return logp, lse


def logprob_rows(hidden, W, tokens, rows):
    """(logp, lse) of selected rows only, one row at a time (for spot checks
    at sizes where a full pass is too slow)."""
    W = np.asarray(W, dtype=np.float64)
    out_logp, out_lse = [], []
    for t in rows:
        z = W @ np.asarray(hidden[t], dtype=np.float64)
        m = z.max()
        lse = m + np.log(np.exp(z - m).sum())
        out_lse.append(lse)
        out_logp.append(z[int(tokens[t])] - lse)
    return np.array(out_logp), np.array(out_lse)


def entropy(hidden, W, seq_of_token=None, chunk=512):
    """H_t = -sum_v p_{t,v} log p_{t,v} in fp64 [T]; masked tokens get 0."""
    hidden = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    T = hidden.shape[0]
    H = np.zeros(T, dtype=np.float64)
    for a in range(0, T, chunk):
        b = min(a + chunk, T)
        z = hidden[a:b] @ W.T
        m = z.max(axis=1)
        lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1))
        logp = z - lse[:, None]
        H[a:b] = -(np.exp(logp) * logp).sum(axis=1)
    if seq_of_token is not None:
        H[np.asarray(seq_of_token) < 0] = 0.0
    return H
