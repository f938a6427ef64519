"""GPU parity of rb_group_advantage and policy_loss_fwd_bwd against the oracle."""

import numpy as np
import pytest
import torch

from oracle.advantage import group_advantage
from oracle.loss import grpo_loss
from paper_2604_08706_amd import workloads as wlm

from gpu_util import rel_l2, require_gpu, to_np

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("G,n_groups,p", [(4, 16, 0.5), (8, 128, 0.4), (8, 4096, 0.3),
                                          (16, 60, 0.5), (8, 125_000, 0.4)])
def test_group_advantage(G, n_groups, p):
    rbp = require_gpu()
    rng = np.random.default_rng(G * 1000 + n_groups)
    rewards = (rng.random(G * n_groups) < p).astype(np.float32)
    off = np.arange(n_groups + 1, dtype=np.int32) * G
    print(f"[advantage] G={G} n_groups={n_groups}", flush=True)
    for ddof in (1, 0):
        adv = torch.empty(G * n_groups, dtype=torch.float32, device="cuda")
        rbp.rb_group_advantage(torch.from_numpy(rewards).cuda(), torch.from_numpy(off).cuda(),
                               adv, ddof=ddof, eps=1e-6)
        want = np.array(group_advantage(rewards, off, ddof=ddof, eps=1e-6))
        got = to_np(adv)
        assert np.allclose(got, want, rtol=1e-5, atol=1e-6)
        # all-equal groups give exactly zero on both sides
        eq = np.array([rewards[off[g]:off[g + 1]].min() == rewards[off[g]:off[g + 1]].max()
                       for g in range(n_groups)])
        for g in np.nonzero(eq)[0]:
            assert np.all(got[off[g]:off[g + 1]] == 0.0)


def test_group_advantage_ragged_and_real_valued():
    rbp = require_gpu()
    rng = np.random.default_rng(7)
    sizes = rng.integers(1, 20, 300)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    rewards = rng.standard_normal(int(off[-1])).astype(np.float32)
    adv = torch.empty(int(off[-1]), dtype=torch.float32, device="cuda")
    rbp.rb_group_advantage(torch.from_numpy(rewards).cuda(), torch.from_numpy(off).cuda(), adv)
    want = np.array(group_advantage(rewards, off))
    assert np.allclose(to_np(adv), want, rtol=1e-4, atol=1e-5)


def _equal_and_near_equal_groups(seed):
    """Groups of G = 4, 8, 16 rewards: all equal to 0.1, 0.7, 1/3 (not exact in
    binary, so an fp32 mean leaves r - mean != 0), and near-equal groups with
    one or two members a few fp32 ulps away."""
    rng = np.random.default_rng(seed)
    groups, equal = [], []
    for G in (4, 8, 16):
        for x in (0.1, 0.7, 1.0 / 3.0, 0.3, 2.2):
            groups.append(np.full(G, x, dtype=np.float32))
            equal.append(True)
            g = np.full(G, x, dtype=np.float32)
            for j in rng.choice(G, int(rng.integers(1, 3)), replace=False):
                step = int(rng.integers(1, 6))
                for _ in range(step):
                    g[j] = np.nextafter(g[j], np.float32(np.inf))
            groups.append(g)
            equal.append(False)
    rewards = np.concatenate(groups)
    off = np.concatenate([[0], np.cumsum([len(g) for g in groups])]).astype(np.int32)
    return rewards, off, np.array(equal)


def test_group_advantage_equal_and_near_equal_non_binary():
    rbp = require_gpu()
    rewards, off, equal = _equal_and_near_equal_groups(11)
    print(f"[advantage] equal/near-equal groups={len(off) - 1}", flush=True)
    for ddof in (1, 0):
        adv = torch.full((len(rewards),), 77.0, dtype=torch.float32, device="cuda")
        rbp.rb_group_advantage(torch.from_numpy(rewards).cuda(), torch.from_numpy(off).cuda(),
                               adv, ddof=ddof, eps=1e-6)
        got = to_np(adv)
        want = np.array(group_advantage(rewards, off, ddof=ddof, eps=1e-6))
        for g in range(len(off) - 1):
            a, w = got[off[g]:off[g + 1]], want[off[g]:off[g + 1]]
            if equal[g]:
                assert np.all(a == 0.0) and np.all(w == 0.0), (g, a)
            else:
                # one fp32 rounding of an fp64 result: well inside rtol 1e-5
                # (a member that equals the group mean gets 0 on both sides)
                assert np.any(w != 0.0)
                assert np.allclose(a, w, rtol=1e-6, atol=1e-12), (g, a, w)


def _loss_case(T, B, seed, noise, margin=1e-3):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, max(2, 2 * T // B), B)
    seq = np.concatenate([[i] * int(l) for i, l in enumerate(lens)])[:T]
    if len(seq) < T:
        seq = np.concatenate([seq, -np.ones(T - len(seq), dtype=np.int64)])
    seq[rng.random(T) < 0.05] = -1   # some padding inside the batch
    logp = (-rng.random(T) * 12.0).astype(np.float32)
    old = (logp + rng.normal(0, noise, T)).astype(np.float32)
    # keep every ratio >= margin away from the clip boundaries, where fp32 and
    # fp64 log-probs (within ~1e-6) could take different branches
    rho = np.exp(logp.astype(np.float64) - old.astype(np.float64))
    near = (np.abs(rho - 0.8) < margin) | (np.abs(rho - 1.2) < margin)
    old[near] -= np.float32(5 * margin)
    adv = rng.standard_normal(B).astype(np.float32)
    adv[rng.random(B) < 0.1] = 0.0
    return logp, old, seq.astype(np.int32), adv, lens.astype(np.int32)


@pytest.mark.parametrize("T,B,noise", [(160, 8, 0.05), (16384, 13, 0.1), (16384, 13, 0.5),
                                       (473_000, 256, 0.2), (1, 1, 0.1)])
def test_loss_matches_oracle(T, B, noise):
    rbp = require_gpu()
    logp, old, seq, adv, lens = _loss_case(T, B, T + B, noise)
    n_seq = B + 3
    print(f"[loss] T={T} B={B} noise={noise}", flush=True)
    d = {k: torch.from_numpy(v).cuda() for k, v in
         dict(logp=logp, old=old, seq=seq, adv=adv, lens=lens).items()}
    loss = torch.full((1,), 0.25, device="cuda")
    stats = torch.zeros(4, device="cuda")
    dlogp = torch.empty(T, device="cuda")
    ws = rbp.workspace(rbp.RBP_OP_LOSS, T)
    rbp.policy_loss_fwd_bwd(d["logp"], d["old"], d["seq"], d["adv"], d["lens"], n_seq, loss,
                            dlogp, stats, ws)
    torch.cuda.synchronize()
    w_loss, w_dlogp, w_stats = grpo_loss(logp, old, seq, adv, lens, n_seq)
    got = to_np(loss)[0] - 0.25  # accumulated into the existing value
    assert abs(got - w_loss) <= 1e-2 * max(abs(w_loss), 1e-30) + 1e-6
    assert rel_l2(to_np(dlogp), w_dlogp) < 1e-2
    assert np.allclose(to_np(dlogp), w_dlogp, rtol=1e-4, atol=1e-9)
    st = to_np(stats)
    assert st[1] == w_stats[1] and st[2] == w_stats[2]  # integer counts: exact
    assert abs(st[0] - w_stats[0]) <= 1e-4 * w_stats[0] + 1e-3
    assert np.all(to_np(dlogp)[seq < 0] == 0)


def test_loss_on_policy_and_determinism():
    rbp = require_gpu()
    T, B = 5000, 10
    logp, _, seq, adv, lens = _loss_case(T, B, 3, 0.1)
    d = {k: torch.from_numpy(v).cuda() for k, v in
         dict(logp=logp, seq=seq, adv=adv, lens=lens).items()}
    outs = []
    for _ in range(2):
        loss = torch.zeros(1, device="cuda")
        stats = torch.zeros(4, device="cuda")
        dlogp = torch.empty(T, device="cuda")
        rbp.policy_loss_fwd_bwd(d["logp"], d["logp"], d["seq"], d["adv"], d["lens"], B, loss,
                                dlogp, stats, rbp.workspace(rbp.RBP_OP_LOSS, T))
        outs.append((to_np(loss).copy(), to_np(dlogp).copy(), to_np(stats).copy()))
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a, b)
    # rho == 1: dlogp_t = -A_i / (n_seq len_i), nothing clipped
    want = np.where(seq >= 0, -adv[np.maximum(seq, 0)] / (B * lens[np.maximum(seq, 0)]), 0)
    assert np.allclose(outs[0][1], want, rtol=1e-6, atol=0)
    assert outs[0][2][1] == 0


def test_loss_empty_batch_adds_nothing():
    # T = 0: the accumulated loss and statistics stay as they were
    rbp = require_gpu()
    adv = torch.tensor([1.0, -1.0, 0.5], device="cuda")
    lens = torch.tensor([4, 5, 6], dtype=torch.int32, device="cuda")
    e = torch.empty(0, device="cuda")
    ei = torch.empty(0, dtype=torch.int32, device="cuda")
    loss = torch.full((1,), 0.25, device="cuda")
    stats = torch.full((4,), 2.0, device="cuda")
    rbp.policy_loss_fwd_bwd(e, e, ei, adv, lens, 3, loss, e, stats,
                            rbp.workspace(rbp.RBP_OP_LOSS, 0))
    torch.cuda.synchronize()
    assert to_np(loss)[0] == 0.25 and np.all(to_np(stats) == 2.0)


def test_group_advantage_large_groups_take_the_direct_path():
    # groups of 40..80 records: a block's 256 groups then span more records
    # than its LDS stage holds, so those blocks read the rewards directly; the
    # last block holds few groups and is staged
    rbp = require_gpu()
    rng = np.random.default_rng(11)
    sizes = rng.integers(40, 81, 600)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    rewards = (rng.random(int(off[-1])) < 0.5).astype(np.float32)
    adv = torch.empty(int(off[-1]), dtype=torch.float32, device="cuda")
    rbp.rb_group_advantage(torch.from_numpy(rewards).cuda(), torch.from_numpy(off).cuda(), adv)
    want = np.array(group_advantage(rewards, off))
    assert np.allclose(to_np(adv), want, rtol=1e-5, atol=1e-6)
