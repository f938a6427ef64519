"""Seeded sweep of the clipped objectives over random clip ranges
(eps_low, eps_high drawn independently, so asymmetric ranges too): the
token-ratio loss, the whole-sequence-ratio loss and the single pass, each
against the oracle with the same eps.  Ratios are kept away from both clip
boundaries, where fp32 and fp64 log-probs could take different branches."""

import numpy as np
import pytest
import torch

from oracle.loss import grpo_loss, grpo_seq_loss

from gpu_util import rel_l2, require_gpu, to_np
import test_gpu_fused as fused

pytestmark = pytest.mark.gpu


def _eps(rng):
    return float(rng.uniform(0.05, 0.4)), float(rng.uniform(0.05, 0.5))


def _away(logp, old, lo, hi, margin):
    """Moves old log-probs so that no ratio exp(logp - old) lies within margin
    of 1 - lo or 1 + hi."""
    rho = np.exp(logp.astype(np.float64) - old.astype(np.float64))
    near = (np.abs(rho - (1 - lo)) < margin) | (np.abs(rho - (1 + hi)) < margin)
    old[near] -= np.float32(5 * margin)
    return old


def _token_cases(n=12, seed=11):
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(1, 50001)), int(rng.integers(1, 301)),
             [0.02, 0.1, 0.3][i % 3], int(rng.integers(0, 2**31))) for i in range(n)]


@pytest.mark.parametrize("T,B,noise,seed", _token_cases())
def test_token_ratio_loss(T, B, noise, seed):
    rbp = require_gpu()
    rng = np.random.default_rng(seed)
    lo, hi = _eps(rng)
    print(f"[loss sweep] T={T} B={B} eps=({lo:.3f}, {hi:.3f})", flush=True)
    lens = rng.integers(1, max(2, 2 * T // B), B)
    seq = np.concatenate([[i] * int(k) for i, k in enumerate(lens)])[:T]
    if len(seq) < T:
        seq = np.concatenate([seq, -np.ones(T - len(seq), dtype=np.int64)])
    seq = seq.astype(np.int32)
    seq[rng.random(T) < 0.05] = -1
    logp = (-rng.random(T) * 12.0).astype(np.float32)
    old = _away(logp, (logp + rng.normal(0, noise, T)).astype(np.float32), lo, hi, 1e-3)
    adv = rng.standard_normal(B).astype(np.float32)
    n_seq = B + int(rng.integers(0, 5))
    d = {k: torch.from_numpy(v).cuda() for k, v in
         dict(logp=logp, old=old, seq=seq, adv=adv, lens=lens.astype(np.int32)).items()}
    loss = torch.zeros(1, device="cuda")
    stats = torch.zeros(4, device="cuda")
    dlogp = torch.empty(T, device="cuda")
    rbp.policy_loss_fwd_bwd(d["logp"], d["old"], d["seq"], d["adv"], d["lens"], n_seq, loss,
                            dlogp, stats, rbp.workspace(rbp.RBP_OP_LOSS, T), eps_low=lo,
                            eps_high=hi)
    torch.cuda.synchronize()
    w_loss, w_d, w_st = grpo_loss(logp, old, seq, adv, lens, n_seq, lo, hi)
    assert abs(to_np(loss)[0] - w_loss) <= 1e-2 * max(abs(w_loss), 1e-30) + 1e-6
    assert rel_l2(to_np(dlogp), w_d) < 1e-2
    assert np.allclose(to_np(dlogp), w_d, rtol=1e-4, atol=1e-9)
    st = to_np(stats)
    assert st[1] == w_st[1] and st[2] == w_st[2]


@pytest.mark.parametrize("B,mean_len,seed", [(1, 5, 1), (9, 40, 2), (64, 300, 3), (200, 900, 4),
                                              (3, 1, 5), (31, 2000, 6)])
def test_sequence_ratio_loss(B, mean_len, seed):
    rbp = require_gpu()
    rng = np.random.default_rng(seed)
    lo, hi = _eps(rng)
    lens = np.maximum(1, rng.poisson(mean_len, B))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    print(f"[loss sweep] seq ratio T={T} B={B} eps=({lo:.3f}, {hi:.3f})", flush=True)
    logp = (-rng.random(T) * 8).astype(np.float32)
    old = (logp + rng.normal(0, 0.15 / np.sqrt(mean_len), T)).astype(np.float32)
    for i in range(B):
        r = np.exp(np.sum(logp[cu[i]:cu[i + 1]].astype(np.float64) - old[cu[i]:cu[i + 1]]))
        if abs(r - (1 - lo)) < 5e-3 or abs(r - (1 + hi)) < 5e-3:
            old[cu[i]] -= np.float32(0.05)
    adv = rng.standard_normal(B).astype(np.float32)
    n_seq = B + 1
    loss = torch.zeros(1, device="cuda")
    stats = torch.zeros(4, device="cuda")
    dlogp = torch.empty(T, device="cuda")
    rbp.policy_loss_seq_fwd_bwd(torch.from_numpy(logp).cuda(), torch.from_numpy(old).cuda(),
                                torch.from_numpy(cu).cuda(), torch.from_numpy(adv).cuda(), n_seq,
                                loss, dlogp, stats, rbp.workspace(rbp.RBP_OP_LOSS_SEQ, B),
                                eps_low=lo, eps_high=hi)
    torch.cuda.synchronize()
    w_loss, w_d, w_st = grpo_seq_loss(logp, old, cu, adv, n_seq, lo, hi)
    assert abs(to_np(loss)[0] - w_loss) <= 1e-3 * max(abs(w_loss), 1e-3)
    assert rel_l2(to_np(dlogp), w_d) < 1e-2
    st = to_np(stats)
    assert st[1] == w_st[1] and st[2] == w_st[2]


@pytest.mark.parametrize("eps", [(0.1, 0.28), (0.35, 0.05)])
def test_single_pass_clip_range(eps):
    rbp = require_gpu()
    T, d, V = 700, 136, 2049
    print(f"[loss sweep] single pass eps={eps}", flush=True)
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = fused._case(T, d, V, 0.02, 41)
    old = _away(want_logp, old, eps[0], eps[1], 1e-3)
    n_seq = len(lens)
    out = fused._run(rbp, hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda(),
                     torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
                     torch.from_numpy(lens).cuda(), n_seq, eps=eps)
    fused._check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq, eps=eps)
