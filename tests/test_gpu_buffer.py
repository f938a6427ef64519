"""GPU parity of the buffer maintenance calls against the oracle: sampling
without replacement and never-used-first (bit-exact slots), steps since last
use and use counts (exact), and FIFO insertion with advantages at insert
(records, arena contents and ring bookkeeping exact; advantages rtol 1e-5)."""

import numpy as np
import pytest
import torch

from oracle import buffer as ob
from oracle.advantage import group_advantage

from gpu_util import require_gpu, to_np

pytestmark = pytest.mark.gpu


def _records(rbp, n_live, cap, head, seed, use=None):
    """A ring of n_live records with 1..8 tokens each; use = per-slot counts."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, 9, n_live).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    phys = (head + np.arange(n_live)) % cap

    def ring(vals, dtype, junk):
        a = np.full(cap, junk, dtype=dtype)
        a[phys] = vals
        return torch.from_numpy(a).cuda()

    t = {
        "off": ring(offs, np.int64, 0), "len": ring(lens, np.int32, 1),
        "rew": ring(rng.random(n_live).astype(np.float32), np.float32, 0.0),
        "adv": ring(rng.standard_normal(n_live).astype(np.float32), np.float32, 0.0),
        "ver": ring(np.zeros(n_live, np.int32), np.int32, 0),
        "tok": torch.from_numpy(rng.integers(0, 1000, int(lens.sum())).astype(np.int32)).cuda(),
        "old": torch.from_numpy(rng.random(int(lens.sum())).astype(np.float32)).cuda(),
        "use": None if use is None else ring(np.asarray(use, np.int32), np.int32, 99),
    }
    rec = rbp.make_records(n_live, cap, head, t["off"], t["len"], t["rew"], t["adv"], t["ver"],
                           t["tok"], t["old"], t["use"])
    return rec, t, lens, offs


def _draw(rbp, rec, cap, mode, seed, step, n_draw):
    cfg = rbp.make_sample_cfg(mode, rbp.RB_LAYOUT_PACKED, seed, step, n_draw,
                              max_tokens=8 * n_draw)
    out = rbp.alloc_batch(cfg)
    print(f"[buffer] mode={mode} n_live={rec.n_live} n_draw={n_draw} step={step}", flush=True)
    rbp.rb_sample_gather(rec, cfg, out, rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, cap))
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in out.items()}


@pytest.mark.parametrize("n_live,cap,head,n_draw", [
    (1, 1, 0, 1), (37, 50, 45, 10), (37, 37, 3, 37), (1000, 1500, 1234, 1),
    (5000, 5000, 17, 300), (100_000, 120_000, 99_999, 1024)])
def test_without_replacement_matches_oracle(n_live, cap, head, n_draw):
    rbp = require_gpu()
    rec, t, lens, offs = _records(rbp, n_live, cap, head, n_live)
    for step in (0, 5):
        got = _draw(rbp, rec, cap, rbp.RB_NO_REPLACE, 11, step, n_draw)
        want = ob.sample_without_replacement(11, step, n_live, n_draw)
        assert np.array_equal(got["idx"], want)
        g = ob.gather(want, offs, lens, np.zeros(n_live), np.zeros(n_live), to_np(t["tok"]),
                      to_np(t["old"]), 10, ob.LAYOUT_PACKED, max_tokens=8 * n_draw)
        assert np.array_equal(got["tokens"], g["tokens"])
        assert np.array_equal(got["cu_seqlens"], g["cu_seqlens"])


@pytest.mark.parametrize("frac_used", [0.0, 0.3, 0.9, 1.0])
def test_unused_first_matches_oracle(frac_used):
    rbp = require_gpu()
    n_live, cap, head = 3000, 4096, 4000
    rng = np.random.default_rng(int(frac_used * 10))
    use = np.where(rng.random(n_live) < frac_used, rng.integers(1, 5, n_live), 0)
    rec, *_ = _records(rbp, n_live, cap, head, 7, use=use)
    for n_draw in (1, 100, 2500):
        got = _draw(rbp, rec, cap, rbp.RB_UNUSED_FIRST, 3, 2, n_draw)
        want = ob.sample_without_replacement(3, 2, n_live, n_draw, use_count=use)
        assert np.array_equal(got["idx"], want)


@pytest.mark.parametrize("n_draw,n_used", [(700, 0), (12_000, 290_000)])
def test_without_replacement_large_buffer_matches_oracle(n_draw, n_used):
    # 300000 records: more than a thousand keys share the selected top digit,
    # so the select runs digit passes before ranking the survivors; with
    # 290000 used records the draw spans all unused ones and the smallest used
    rbp = require_gpu()
    n_live = 300_000
    use = np.zeros(n_live, dtype=np.int32)
    use[:n_used] = 1 + np.arange(n_used) % 3
    mode = rbp.RB_UNUSED_FIRST if n_used else rbp.RB_NO_REPLACE
    rec, *_ = _records(rbp, n_live, n_live, 12_345, 4, use=use if n_used else None)
    got = _draw(rbp, rec, n_live, mode, 5, 1, n_draw)
    want = ob.sample_without_replacement(5, 1, n_live, n_draw, use_count=use if n_used else None)
    assert np.array_equal(got["idx"], want)


def test_without_replacement_rejects_bad_requests():
    rbp = require_gpu()
    rec, *_ = _records(rbp, 10, 10, 0, 1)
    with pytest.raises(rbp.RbpError):
        _draw(rbp, rec, 10, rbp.RB_NO_REPLACE, 1, 0, 11)
    with pytest.raises(rbp.RbpError):
        _draw(rbp, rec, 10, rbp.RB_UNUSED_FIRST, 1, 0, 3)  # no use_count


def test_note_use_matches_steps_since_last_use():
    rbp = require_gpu()
    cap, head, n_live = 64, 50, 60
    use = torch.zeros(cap, dtype=torch.int32, device="cuda")
    last = torch.full((cap,), -1, dtype=torch.int64, device="cuda")
    ws = rbp.workspace(rbp.RBP_OP_NOTE_USE, cap)
    rng = np.random.default_rng(5)
    batches, counts = [], np.zeros(n_live, dtype=np.int64)
    for step in (0, 1, 3, 4, 9, 10, 10):
        idx = rng.integers(0, n_live, 40).astype(np.int32)  # with replacement: repeats
        since = torch.empty(40, dtype=torch.int32, device="cuda")
        rbp.rb_note_use(torch.from_numpy(idx).cuda(), head, cap, step, use, last, since, ws)
        torch.cuda.synchronize()
        batches.append((step, idx.tolist()))
        want = ob.steps_since_last_use(batches)[-1]
        assert np.array_equal(to_np(since), want), step
        np.add.at(counts, idx, 1)
    phys = (head + np.arange(n_live)) % cap
    assert np.array_equal(to_np(use)[phys], counts)
    last_want = {}
    for step, ids in batches:
        for s in ids:
            last_want[s] = step
    assert all(to_np(last)[phys[s]] == (last_want.get(s, -1)) for s in range(n_live))


def test_push_is_fifo_with_advantages_at_insert():
    rbp = require_gpu()
    cap, slot = 10, 6
    ring = rbp.make_ring(cap, slot)
    fifo = ob.FifoBuffer(cap)
    rng = np.random.default_rng(3)
    version = 0
    for sizes in ([4, 4], [3], [4, 2, 4], [1], [5, 5], [2]):
        version += 1
        n = sum(sizes)
        goff = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
        lens = rng.integers(1, 9, n).astype(np.int32)  # some longer than the slot
        src = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
        rew = (rng.random(n) < 0.5).astype(np.float32)
        tok = rng.integers(0, 500, int(lens.sum())).astype(np.int32)
        old = rng.random(int(lens.sum())).astype(np.float32)
        ring.t["use_count"].fill_(7)  # rows written by the push must be reset
        print(f"[buffer] push {sizes}", flush=True)
        rbp.rb_push(ring, torch.from_numpy(goff).cuda(), torch.from_numpy(lens).cuda(),
                    torch.from_numpy(src).cuda(), torch.from_numpy(rew).cuda(), version,
                    torch.from_numpy(tok).cuda(), torch.from_numpy(old).cuda())
        torch.cuda.synchronize()
        adv = group_advantage(rew, goff)
        for i in range(n):
            k = min(int(lens[i]), slot)
            fifo.push({"len": k, "rew": rew[i], "adv": adv[i], "ver": version,
                       "tok": tok[src[i]:src[i] + k], "old": old[src[i]:src[i] + k]})
        assert ring.n_live == len(fifo)
        t = {k: (None if v is None else to_np(v)) for k, v in ring.t.items()}
        for s, want in enumerate(fifo.records):
            r = (ring.head + s) % cap
            assert t["length"][r] == want["len"] and t["version"][r] == want["ver"]
            assert t["reward"][r] == want["rew"]
            assert abs(t["advantage"][r] - want["adv"]) <= 1e-5 * abs(want["adv"]) + 1e-6
            o = t["arena_off"][r]
            assert o == r * slot
            assert np.array_equal(t["arena_tokens"][o:o + want["len"]], want["tok"])
            assert np.array_equal(t["arena_old_logp"][o:o + want["len"]], want["old"])
        written = (ring.head + len(fifo) - n + np.arange(n)) % cap
        assert np.all(t["use_count"][written] == 0) and np.all(t["last_step"][written] == -1)
    # the filled ring feeds the sampler: a uniform draw gathers the FIFO records
    rec = rbp.ring_records(ring)
    cfg = rbp.make_sample_cfg(rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 2, 0, 6, max_tokens=64)
    out = rbp.alloc_batch(cfg)
    rbp.rb_sample_gather(rec, cfg, out, rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, cap))
    torch.cuda.synchronize()
    idx = ob.sample_indices([0.0] * cap, ob.RB_UNIFORM, 2, 0, 6)
    assert np.array_equal(to_np(out["idx"]), idx)
    want_tok = np.concatenate([fifo.records[s]["tok"] for s in idx])
    assert np.array_equal(to_np(out["tokens"])[:len(want_tok)], want_tok)
    with pytest.raises(rbp.RbpError):
        rbp.rb_push(ring, torch.tensor([0, 11], dtype=torch.int32, device="cuda"),
                    torch.ones(11, dtype=torch.int32, device="cuda"),
                    torch.zeros(11, dtype=torch.int64, device="cuda"),
                    torch.zeros(11, device="cuda"), 0,
                    torch.zeros(1, dtype=torch.int32, device="cuda"), torch.zeros(1, device="cuda"))


def test_push_equal_non_binary_groups_store_zero_advantage():
    # the push computes advantages at insert with the same helper as
    # rb_group_advantage: groups of equal rewards such as 0.7 store exact zeros
    rbp = require_gpu()
    G_list = [4, 8, 16, 4, 8, 16, 8]
    vals = [0.1, 0.7, 1.0 / 3.0, 0.3, 0.7, 0.1, None]
    rew = []
    for G, x in zip(G_list, vals):
        if x is None:  # one near-equal group: a member one ulp above the rest
            g = np.full(G, 0.7, dtype=np.float32)
            g[3] = np.nextafter(g[3], np.float32(np.inf))
        else:
            g = np.full(G, x, dtype=np.float32)
        rew.append(g)
    rew = np.concatenate(rew)
    n = len(rew)
    goff = np.concatenate([[0], np.cumsum(G_list)]).astype(np.int32)
    lens = np.ones(n, np.int32)
    ring = rbp.make_ring(n + 5, 2)
    print(f"[buffer] push of {len(G_list)} equal/near-equal groups", flush=True)
    rbp.rb_push(ring, torch.from_numpy(goff).cuda(), torch.from_numpy(lens).cuda(),
                torch.arange(n, dtype=torch.int64, device="cuda"), torch.from_numpy(rew).cuda(),
                1, torch.zeros(n, dtype=torch.int32, device="cuda"),
                torch.zeros(n, device="cuda"))
    torch.cuda.synchronize()
    got = to_np(ring.t["advantage"])[(ring.head + np.arange(n)) % (n + 5)]
    want = np.array(group_advantage(rew, goff))
    k = goff[-2]
    assert np.all(got[:k] == 0.0) and np.all(want[:k] == 0.0)
    assert np.all(want[k:] != 0.0)
    assert np.allclose(got[k:], want[k:], rtol=1e-6, atol=1e-12)


@pytest.mark.parametrize("n,n_bins,lo", [(0, 3, 0), (1, 1, 0), (1000, 7, -1), (300_000, 4096, 5),
                                         (300_000, 33, -1)])
def test_hist_accumulate_matches_oracle(n, n_bins, lo):
    rbp = require_gpu()
    rng = np.random.default_rng(n + n_bins)
    vals = rng.integers(-3, 5000, n).astype(np.int32)
    hist = torch.zeros(n_bins, dtype=torch.int64, device="cuda")
    print(f"[buffer] hist n={n} n_bins={n_bins} lo={lo}", flush=True)
    for _ in range(2):  # accumulates
        rbp.rb_hist_accumulate(torch.from_numpy(vals).cuda(), hist, lo)
    torch.cuda.synchronize()
    want = 2 * np.array(ob.histogram(vals, n_bins, lo), dtype=np.int64)
    assert np.array_equal(to_np(hist), want)


def test_buffer_statistics_over_a_run():
    # pushes with evictions, uniform draws and usage updates: the ring's
    # replay-ratio histogram of evicted records, the live use counts, and the
    # histograms of ages (off-policiness) and steps since last use
    rbp = require_gpu()
    cap, slot, bins = 12, 4, 6
    ring = rbp.make_ring(cap, slot, replay_bins=bins)
    ws = rbp.workspace(rbp.RBP_OP_NOTE_USE, cap)
    rng = np.random.default_rng(9)
    age_h = torch.zeros(8, dtype=torch.int64, device="cuda")
    since_h = torch.zeros(6, dtype=torch.int64, device="cuda")
    steps, ages, sinces, batches, versions = [], [], [], [], []
    for step in range(14):
        n_new = int(rng.integers(1, 6))
        lens = np.full(n_new, 2, dtype=np.int32)
        goff = np.array([0, n_new], dtype=np.int32)
        rbp.rb_push(ring, torch.from_numpy(goff).cuda(), torch.from_numpy(lens).cuda(),
                    torch.arange(n_new, dtype=torch.int64, device="cuda") * 2,
                    torch.zeros(n_new, device="cuda"), step,
                    torch.zeros(2 * n_new, dtype=torch.int32, device="cuda"),
                    torch.zeros(2 * n_new, device="cuda"))
        versions = (versions + [step] * n_new)[-cap:]
        n_draw = 7
        cfg = rbp.make_sample_cfg(rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 4, step, n_draw,
                                  cur_version=step, max_tokens=2 * n_draw)
        out = rbp.alloc_batch(cfg)
        print(f"[buffer] statistics step={step} n_live={ring.n_live}", flush=True)
        rbp.rb_sample_gather(rbp.ring_records(ring), cfg, out,
                             rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, cap))
        since = torch.empty(n_draw, dtype=torch.int32, device="cuda")
        rbp.rb_note_use(out["idx"], ring.head, cap, step, ring.t["use_count"],
                        ring.t["last_step"], since, ws)
        rbp.rb_hist_accumulate(out["age"], age_h, 0)
        rbp.rb_hist_accumulate(since, since_h, -1)
        torch.cuda.synchronize()
        draws = ob.sample_indices([0.0] * ring.n_live, ob.RB_UNIFORM, 4, step, n_draw)
        assert np.array_equal(to_np(out["idx"]), draws)
        steps.append((n_new, draws))
        ages += [step - versions[s] for s in draws]
        # rollout ids: the k-th rollout ever pushed is id k
        first_id = sum(n for n, _ in steps) - ring.n_live
        batches.append((step, [first_id + s for s in draws]))
    evicted, live = ob.replay_ratios(cap, steps)
    assert len(evicted) > 0
    assert np.array_equal(to_np(ring.t["replay_hist"]), ob.histogram(evicted, bins))
    phys = (ring.head + np.arange(ring.n_live)) % cap
    assert np.array_equal(to_np(ring.t["use_count"])[phys], live)
    assert np.array_equal(to_np(age_h), ob.histogram(ages, 8))
    sinces = [v for b in ob.steps_since_last_use(batches) for v in b]
    assert np.array_equal(to_np(since_h), ob.histogram(sinces, 6, lo=-1))


def test_push_of_a_full_capacity_evicts_exactly_the_live_records():
    # ring of 8 holding 5 used records; a push of 8 overwrites every row and
    # evicts exactly the 5 (their use counts go to the replay histogram)
    rbp = require_gpu()
    cap = 8
    ring = rbp.make_ring(cap, 2, replay_bins=4)
    ws = rbp.workspace(rbp.RBP_OP_NOTE_USE, cap)

    def push(n, version):
        rbp.rb_push(ring, torch.tensor([0, n], dtype=torch.int32, device="cuda"),
                    torch.ones(n, dtype=torch.int32, device="cuda"),
                    torch.arange(n, dtype=torch.int64, device="cuda"),
                    torch.zeros(n, device="cuda"), version,
                    torch.zeros(n, dtype=torch.int32, device="cuda"), torch.zeros(n, device="cuda"))

    push(5, 0)
    draws = [0, 0, 0, 1, 1, 4, 4, 4, 4, 4]  # uses 3, 2, 0, 0, 5
    rbp.rb_note_use(torch.tensor(draws, dtype=torch.int32, device="cuda"), ring.head, cap, 0,
                    ring.t["use_count"], ring.t["last_step"], None, ws)
    push(cap, 1)
    torch.cuda.synchronize()
    ev, live = ob.replay_ratios(cap, [(5, draws), (cap, [])])
    assert ev == [3, 2, 0, 0, 5] and ring.n_live == cap
    assert np.array_equal(to_np(ring.t["replay_hist"]), ob.histogram(ev, 4))
    assert np.all(to_np(ring.t["use_count"]) == 0) and np.all(to_np(ring.t["version"]) == 1)


def test_push_long_records_and_note_use_at_full_capacity():
    # records of up to 9000 tokens into 8192-token rows: the copy splits each
    # row over 16 blocks that loop over it, and records past the row are cut
    rbp = require_gpu()
    cap, slot = 48, 8192
    ring = rbp.make_ring(cap, slot)
    fifo = ob.FifoBuffer(cap)
    rng = np.random.default_rng(13)
    for version, n in enumerate((20, 20, 20)):
        lens = rng.integers(1, 9001, n).astype(np.int32)
        src = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
        tok = rng.integers(0, 152064, int(lens.sum())).astype(np.int32)
        old = rng.standard_normal(int(lens.sum())).astype(np.float32)
        rew = (rng.random(n) < 0.4).astype(np.float32)
        print(f"[buffer] long push n={n}", flush=True)
        rbp.rb_push(ring, torch.tensor([0, n // 2, n], dtype=torch.int32, device="cuda"),
                    torch.from_numpy(lens).cuda(), torch.from_numpy(src).cuda(),
                    torch.from_numpy(rew).cuda(), version, torch.from_numpy(tok).cuda(),
                    torch.from_numpy(old).cuda())
        for i in range(n):
            k = min(int(lens[i]), slot)
            fifo.push({"tok": tok[src[i]:src[i] + k], "old": old[src[i]:src[i] + k]})
    torch.cuda.synchronize()
    t_tok, t_old = to_np(ring.t["arena_tokens"]), to_np(ring.t["arena_old_logp"])
    t_len = to_np(ring.t["length"])
    for s, want in enumerate(fifo.records):
        r = (ring.head + s) % cap
        n = len(want["tok"])
        assert t_len[r] == n
        assert np.array_equal(t_tok[r * slot:r * slot + n], want["tok"])
        assert np.array_equal(t_old[r * slot:r * slot + n], want["old"])

    # usage update at the stress buffer's capacity (10^6 rows, 256 draws with
    # repeats, the head near the end of the ring)
    cap2, head, n_live = 1_000_000, 999_000, 1_000_000
    use = torch.zeros(cap2, dtype=torch.int32, device="cuda")
    last = torch.full((cap2,), -1, dtype=torch.int64, device="cuda")
    ws = rbp.workspace(rbp.RBP_OP_NOTE_USE, cap2)
    batches = []
    for step in (0, 4, 5):
        idx = rng.integers(0, n_live, 256)
        idx[:40] = idx[40:80]  # repeats inside the batch
        since = torch.empty(256, dtype=torch.int32, device="cuda")
        rbp.rb_note_use(torch.from_numpy(idx.astype(np.int32)).cuda(), head, cap2, step, use,
                        last, since, ws)
        torch.cuda.synchronize()
        batches.append((step, idx.tolist()))
        assert np.array_equal(to_np(since), ob.steps_since_last_use(batches)[-1])
    counts = np.zeros(n_live, dtype=np.int64)
    for _, ids in batches:
        np.add.at(counts, ids, 1)
    phys = (head + np.arange(n_live)) % cap2
    assert np.array_equal(to_np(use)[phys], counts)
