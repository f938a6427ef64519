"""Backward of the per-token log-probabilities to hidden states and LM head.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

With z_t = W h_t, lse_t = log sum_v exp(z_{t,v}) and logp_t = z_{t,y_t} - lse_t
(see ``oracle.logprob``), an upstream gradient dlogp_t gives

    p_t       = exp(z_t - lse_t)                  (softmax of row t)
    dz_t      = dlogp_t (e_{y_t} - p_t)
    dhidden_t = W^T dz_t
    dW        = sum_t dz_t h_t^T.

This is the chain rule through log-softmax; it is what the trainer's
``forward_backward`` (App. B) computes for the LM head.  Plain fp64; the
logits are recomputed per chunk of tokens, which bounds memory only.  Masked
tokens (seq_of_token < 0) contribute nothing and get a zero dhidden row.

Parity: pinned by central finite differences of the composite loss in fp64 on
tiny inputs, by the vanishing column sums of dW (sum_v dz_{t,v} = 0), by the
closed form dhidden_t = dlogp_t (W_{y_t} - E_{p_t}[W]) and by linearity in
dlogp -- tests/test_oracle_grad.py.
"""

import numpy as np


def logprob_backward(hidden, W, tokens, lse, dlogp, seq_of_token=None,
                     chunk=512):
    """Return (dhidden [T, d], dW [V, d]) in fp64."""
    hidden = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    tokens = np.asarray(tokens, dtype=np.int64)
    lse = np.asarray(lse, dtype=np.float64)
    dlogp = np.asarray(dlogp, dtype=np.float64).copy()
    if seq_of_token is not None:
        dlogp[np.asarray(seq_of_token) < 0] = 0.0
    T = hidden.shape[0]
    dhidden = np.zeros_like(hidden)
    dW = np.zeros_like(W)
    for a in range(0, T, chunk):
        b = min(a + chunk, T)
        z = hidden[a:b] @ W.T
        p = np.exp(z - lse[a:b, None])
        dz = -dlogp[a:b, None] * p
        dz[np.arange(b - a), tokens[a:b]] += dlogp[a:b]
        dhidden[a:b] = dz @ W
        dW += dz.T @ hidden[a:b]
    return dhidden, dW


def dz_rows(hidden, W, tokens, lse, dlogp, rows):
    """dz_t = dlogp_t (e_{y_t} - softmax(W h_t)) for selected rows only,
    [len(rows), V] (for spot checks at sizes where a full pass is too slow)."""
    W = np.asarray(W, dtype=np.float64)
    rows = list(rows)
    H = np.asarray([np.asarray(hidden[t], dtype=np.float64) for t in rows])
    z = H @ W.T
    dl = np.array([float(dlogp[t]) for t in rows])
    ls = np.array([float(lse[t]) for t in rows])
    dz = -dl[:, None] * np.exp(z - ls[:, None])
    dz[np.arange(len(rows)), [int(tokens[t]) for t in rows]] += dl
    return dz


def dhidden_rows(hidden, W, tokens, lse, dlogp, rows, dz=None):
    """dhidden of selected rows only: W^T dz_t."""
    if dz is None:
        dz = dz_rows(hidden, W, tokens, lse, dlogp, rows)
    return dz @ np.asarray(W, dtype=np.float64)


def dW_from_rows(hidden, W, tokens, lse, dlogp, rows, v_lo=0, v_hi=None, dz=None):
    """Rows [v_lo, v_hi) of dW = sum over the given token rows of dz_t h_t^T
    (the exact dW when every other token has dlogp = 0)."""
    if dz is None:
        dz = dz_rows(hidden, W, tokens, lse, dlogp, rows)
    v_hi = dz.shape[1] if v_hi is None else v_hi
    H = np.asarray([np.asarray(hidden[t], dtype=np.float64) for t in rows])
    return dz[:, v_lo:v_hi].T @ H
