"""GPU vs oracle: AsymRE (coefficient at insert, objective, gradient) and the
whole-sequence-ratio objective, through the C ABI."""

import numpy as np
import pytest
import torch

from oracle.loss import asymre_coef, asymre_loss, grpo_seq_loss
from gpu_util import rel_l2, require_gpu, to_np


def _seqs(seed, B, mean_len, masked=0.0):
    rng = np.random.default_rng(seed)
    lens = np.maximum(1, rng.poisson(mean_len, B)).astype(np.int64)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    seq = np.repeat(np.arange(B), lens).astype(np.int32)
    if masked:
        seq = seq.copy()
        seq[rng.random(len(seq)) < masked] = -1
    return rng, lens, cu, seq


@pytest.mark.gpu
@pytest.mark.parametrize("n_groups,G", [(1, 1), (16, 4), (128, 8), (4096, 16)])
def test_asymre_coef(n_groups, G):
    rbp = require_gpu()
    rng = np.random.default_rng(n_groups)
    sizes = np.full(n_groups, G)
    sizes[::3] = np.maximum(1, G - 1)  # some short groups
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    rewards = (rng.random(off[-1]) < 0.4).astype(np.float32)
    rewards[: off[-1] // 5] = rng.random(off[-1] // 5).astype(np.float32)  # real-valued too
    coef = torch.empty(off[-1], device="cuda")
    rbp.rb_asymre_coef(torch.from_numpy(rewards).cuda(), torch.from_numpy(off).cuda(), coef,
                       delta_v=-0.1)
    want = np.array(asymre_coef(rewards, off, -0.1))
    assert np.allclose(to_np(coef), want, rtol=0, atol=2e-6)


@pytest.mark.gpu
@pytest.mark.parametrize("B,mean_len,masked", [(8, 20, 0.0), (13, 1300, 0.05),
                                               (256, 1800, 0.1), (1, 1, 0.0)])
def test_asymre_loss_matches_oracle(B, mean_len, masked):
    rbp = require_gpu()
    rng, lens, cu, seq = _seqs(B + mean_len, B, mean_len, masked)
    T = len(seq)
    print(f"[asymre] T={T} B={B}", flush=True)
    logp = (-rng.random(T) * 10).astype(np.float32)
    coef = rng.standard_normal(B).astype(np.float32)
    n_seq = B + 5
    loss = torch.full((1,), 0.5, device="cuda")
    stats = torch.zeros(2, device="cuda")
    dlogp = torch.empty(T, device="cuda")
    rbp.policy_asymre_fwd_bwd(torch.from_numpy(logp).cuda(), torch.from_numpy(seq).cuda(),
                              torch.from_numpy(coef).cuda(), n_seq, loss, dlogp, stats,
                              rbp.workspace(rbp.RBP_OP_LOSS, T))
    torch.cuda.synchronize()
    w_loss, w_d, w_st = asymre_loss(logp, seq, coef, n_seq)
    got = to_np(loss)[0] - 0.5
    assert abs(got - w_loss) <= 1e-4 * max(abs(w_loss), 1.0)
    assert rel_l2(to_np(dlogp), w_d) < 1e-6
    assert np.all(to_np(dlogp)[seq < 0] == 0)
    st = to_np(stats)
    assert st[0] == w_st[0]
    assert abs(st[1] - w_st[1]) <= 1e-4 * max(abs(w_st[1]), 1.0)


@pytest.mark.gpu
@pytest.mark.parametrize("B,mean_len,noise", [(8, 12, 0.02), (64, 300, 0.004),
                                              (256, 1800, 0.001), (3, 1, 0.2)])
def test_seq_ratio_loss_matches_oracle(B, mean_len, noise):
    rbp = require_gpu()
    rng, lens, cu, seq = _seqs(7 * B + mean_len, B, mean_len)
    T = int(cu[-1]) + 37  # tokens past the last sequence get dlogp = 0
    print(f"[seq ratio] T={T} B={B}", flush=True)
    logp = (-rng.random(T) * 8).astype(np.float32)
    old = (logp + rng.normal(0, noise, T)).astype(np.float32)
    adv = rng.standard_normal(B).astype(np.float32)
    # keep every sequence ratio away from the clip boundaries, where fp32 and
    # fp64 could take different branches
    s = np.array([np.sum(logp[cu[i]:cu[i + 1]].astype(np.float64) - old[cu[i]:cu[i + 1]])
                  for i in range(B)])
    for i in range(B):
        r = np.exp(s[i])
        if abs(r - 0.8) < 5e-3 or abs(r - 1.2) < 5e-3:
            old[cu[i]] -= np.float32(0.05)
    n_seq = B + 2
    loss = torch.zeros(1, device="cuda")
    stats = torch.zeros(4, device="cuda")
    dlogp = torch.full((T,), 7.0, device="cuda")
    rbp.policy_loss_seq_fwd_bwd(torch.from_numpy(logp).cuda(), torch.from_numpy(old).cuda(),
                                torch.from_numpy(cu).cuda(), torch.from_numpy(adv).cuda(), n_seq,
                                loss, dlogp, stats, rbp.workspace(rbp.RBP_OP_LOSS_SEQ, B))
    torch.cuda.synchronize()
    w_loss, w_d, w_st = grpo_seq_loss(logp, old, cu, adv, n_seq)
    assert abs(to_np(loss)[0] - w_loss) <= 1e-3 * max(abs(w_loss), 1e-3)
    assert rel_l2(to_np(dlogp), w_d) < 1e-2
    assert np.all(to_np(dlogp)[cu[-1]:] == 0)
    st = to_np(stats)
    assert st[1] == w_st[1] and st[2] == w_st[2]
    assert abs(st[0] - w_st[0]) <= 1e-3 * w_st[0]


@pytest.mark.gpu
def test_variants_are_deterministic_and_reject_bad_args():
    rbp = require_gpu()
    rng, lens, cu, seq = _seqs(3, 40, 50)
    T = len(seq)
    logp = torch.from_numpy((-rng.random(T) * 5).astype(np.float32)).cuda()
    adv = torch.from_numpy(rng.standard_normal(40).astype(np.float32)).cuda()
    cu_d = torch.from_numpy(cu).cuda()
    outs = []
    for _ in range(2):
        loss, stats, d = torch.zeros(1, device="cuda"), torch.zeros(4, device="cuda"), \
            torch.empty(T, device="cuda")
        rbp.policy_loss_seq_fwd_bwd(logp, logp - 0.001, cu_d, adv, 40, loss, d, stats,
                                    rbp.workspace(rbp.RBP_OP_LOSS_SEQ, 40))
        outs.append((to_np(loss).copy(), to_np(d).copy(), to_np(stats).copy()))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
    with pytest.raises(rbp.RbpError):
        rbp.policy_loss_seq_fwd_bwd(logp, logp, cu_d, adv, 0, torch.zeros(1, device="cuda"),
                                    torch.empty(T, device="cuda"), torch.zeros(4, device="cuda"),
                                    rbp.workspace(rbp.RBP_OP_LOSS_SEQ, 40))
    with pytest.raises(rbp.RbpError):
        rbp.policy_asymre_fwd_bwd(logp, torch.from_numpy(seq).cuda(), adv, 40,
                                  torch.zeros(1, device="cuda"), torch.empty(T, device="cuda"),
                                  torch.zeros(2, device="cuda"), torch.empty(4, device="cuda",
                                                                             dtype=torch.uint8))
