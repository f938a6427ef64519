"""Pins of the oracle's replay buffer, sampling rules and gather."""

import json
import os

import numpy as np
import pytest
from scipy import stats

from oracle import buffer as ob
from oracle import philox


def test_fifo_push_evicts_oldest_and_sampling_keeps_records():
    # App. B "BufferStructure": push evicts the oldest once full
    b = ob.FifoBuffer(3)
    for r in range(5):
        b.push(r)
    assert b.records == [2, 3, 4]
    rewards = [1.0, 0.0, 1.0]
    ob.sample_indices(rewards, ob.RB_UNIFORM, seed=1, step=0, n_draw=10)
    assert b.records == [2, 3, 4]


def test_paper_worked_example_positive_bias(golden_dir):
    with open(os.path.join(golden_dir, "pos_retain_example.json")) as f:
        ex = json.load(f)
    rewards = [1.0 if c else 0.0 for c in ex["correct"]]
    n_fresh, n_pos_keep = ob.retain_split(ex["N"], ex["delta"])
    kept = ob.retained_set(rewards, n_fresh, n_pos_keep)
    assert [ex["names"][s] for s in kept] == ex["expected_buffer"]
    assert len(kept) == ex["N"]


def test_worked_example_at_printed_delta_differs():
    # at the printed delta = 0.75 the stated rule does not give the printed set
    correct = [False, True, True, False, True, True, False, True, False, False]
    rewards = [1.0 if c else 0.0 for c in correct]
    kept = ob.retained_set(rewards, *ob.retain_split(8, 0.75))
    assert 6 not in kept  # z_{t-3} dropped
    assert len(kept) == 7  # a sixth correct rollout would have to be older


def test_retain_delta_zero_is_plain_fifo_window():
    rng = np.random.default_rng(0)
    rewards = (rng.random(50) < 0.3).astype(float)
    kept = ob.retained_set(rewards, *ob.retain_split(20, 0.0))
    assert kept == list(range(30, 50))


def test_retain_brute_force_definition():
    # freshest n_fresh + freshest n_pos_keep positives among the rest, by
    # scanning from the newest record backwards
    rng = np.random.default_rng(1)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        rewards = (rng.random(n) < rng.random()).astype(float)
        nf = int(rng.integers(0, n + 3))
        npk = int(rng.integers(0, n + 3))
        want = set()
        for s in range(n - 1, -1, -1):
            if n - s <= nf:
                want.add(s)
        pos_taken = 0
        for s in range(n - 1, -1, -1):
            if s in want:
                continue
            if rewards[s] > 0 and pos_taken < npk:
                want.add(s)
                pos_taken += 1
        assert ob.retained_set(rewards, nf, npk) == sorted(want)


def test_uniform_chi_square():
    n_live, n_draw = 97, 200000
    rewards = [0.0] * n_live
    idx = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=11, step=4, n_draw=n_draw)
    counts = np.bincount(idx, minlength=n_live)
    chi2 = stats.chisquare(counts)
    assert chi2.pvalue > 1e-4


def test_uniform_draw_depends_only_on_seed_step_j():
    rewards = [0.0] * 1000
    a = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=5, step=9, n_draw=64)
    b = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=5, step=9, n_draw=128)
    assert a == b[:64]  # a prefix of a longer call: draws are independent
    c = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=5, step=10, n_draw=64)
    assert a != c
    for j in (0, 17, 63):
        x0 = philox.draw_block(5, 9, j)[0]
        assert a[j] == (x0 * 1000) >> 64


def test_pos_mix_p0_equals_uniform_and_p1_only_positives():
    rng = np.random.default_rng(3)
    rewards = (rng.random(500) < 0.3).astype(float)
    u = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=2, step=1, n_draw=400)
    m0 = ob.sample_indices(rewards, ob.RB_POS_MIX, seed=2, step=1, n_draw=400, p_q32=0)
    assert u == m0
    m1 = ob.sample_indices(rewards, ob.RB_POS_MIX, seed=2, step=1, n_draw=400,
                           p_q32=philox.p_to_q32(1.0))
    assert all(rewards[i] > 0 for i in m1)
    pos = ob.positive_slots(rewards)
    counts = np.bincount([pos.index(i) for i in m1], minlength=len(pos))
    assert stats.chisquare(counts).pvalue > 1e-4


def test_pos_mix_fraction_chi_square():
    # expected positive fraction p + (1 - p) f_pos
    rng = np.random.default_rng(4)
    rewards = (rng.random(1000) < 0.3).astype(float)
    f_pos = rewards.mean()
    p = 0.7
    n_draw = 50000
    idx = ob.sample_indices(rewards, ob.RB_POS_MIX, seed=8, step=2, n_draw=n_draw,
                            p_q32=philox.p_to_q32(p))
    n_pos = sum(rewards[i] > 0 for i in idx)
    expect = p + (1 - p) * f_pos
    z = (n_pos - n_draw * expect) / np.sqrt(n_draw * expect * (1 - expect))
    assert abs(z) < 4.5


def test_pos_mix_no_positives_falls_back_to_uniform():
    rewards = [0.0] * 64
    u = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=1, step=0, n_draw=32)
    m = ob.sample_indices(rewards, ob.RB_POS_MIX, seed=1, step=0, n_draw=32,
                          p_q32=philox.p_to_q32(1.0))
    assert u == m


def test_pos_retain_draws_cover_retained_set_uniformly():
    rng = np.random.default_rng(5)
    rewards = (rng.random(300) < 0.4).astype(float)
    nf, npk = ob.retain_split(100, 0.5)
    kept = ob.retained_set(rewards, nf, npk)
    idx = ob.sample_indices(rewards, ob.RB_POS_RETAIN, seed=3, step=7,
                            n_draw=50000, n_fresh=nf, n_pos_keep=npk)
    assert set(idx) <= set(kept)
    counts = np.bincount([kept.index(i) for i in idx], minlength=len(kept))
    assert stats.chisquare(counts).pvalue > 1e-4
    # delta = 0 over the whole table is uniform sampling, draw for draw
    u = ob.sample_indices(rewards, ob.RB_UNIFORM, seed=3, step=7, n_draw=100)
    r0 = ob.sample_indices(rewards, ob.RB_POS_RETAIN, seed=3, step=7, n_draw=100,
                           n_fresh=300, n_pos_keep=0)
    assert u == r0


def _table(rng, n, max_len):
    lens = rng.integers(1, max_len + 1, n)
    off = np.zeros(n, dtype=np.int64)
    off[1:] = np.cumsum(lens)[:-1]
    total = int(lens.sum())
    toks = rng.integers(0, 1000, total).astype(np.int32)
    old = rng.standard_normal(total).astype(np.float32)
    return off, lens, toks, old


def test_gather_packed_windows_tile_the_stream():
    rng = np.random.default_rng(6)
    off, lens, toks, old = _table(rng, 40, 30)
    adv = rng.standard_normal(40).astype(np.float32)
    ver = rng.integers(0, 5, 40)
    idx = [3, 3, 17, 0, 39, 22]
    total = int(sum(lens[i] for i in idx))
    win = 16
    pieces = []
    for wb in range(0, total + win, win):
        g = ob.gather(idx, off, lens, adv, ver, toks, old, cur_version=7,
                      layout=ob.LAYOUT_PACKED, max_tokens=win, token_begin=wb)
        nv = g["n_tokens"]
        assert nv == max(0, min(win, total - wb))
        assert np.all(g["seq_of_token"][nv:] == -1)
        pieces.append((g["tokens"][:nv], g["old_logp"][:nv], g["seq_of_token"][:nv]))
        assert list(g["len"]) == [lens[i] for i in idx]
        assert list(g["age"]) == [7 - ver[i] for i in idx]
    stream_tok = np.concatenate([p[0] for p in pieces])
    stream_seq = np.concatenate([p[2] for p in pieces])
    want_tok = np.concatenate([toks[off[i]:off[i] + lens[i]] for i in idx])
    want_seq = np.concatenate([[j] * lens[i] for j, i in enumerate(idx)])
    assert np.array_equal(stream_tok, want_tok)
    assert np.array_equal(stream_seq, want_seq)
    assert g["cu_seqlens"][-1] == total
    assert np.all(np.diff(g["cu_seqlens"]) == [lens[i] for i in idx])


def test_gather_padded_rows():
    rng = np.random.default_rng(7)
    off, lens, toks, old = _table(rng, 10, 20)
    adv = np.zeros(10, dtype=np.float32)
    ver = np.zeros(10, dtype=np.int64)
    idx = [9, 1, 1]
    g = ob.gather(idx, off, lens, adv, ver, toks, old, 0, ob.LAYOUT_PADDED, l_max=12)
    for j, i in enumerate(idx):
        k = min(lens[i], 12)
        assert np.array_equal(g["tokens"][j, :k], toks[off[i]:off[i] + k])
        assert np.all(g["seq_of_token"][j, :k] == j)
        assert np.all(g["seq_of_token"][j, k:] == -1)
    assert g["n_tokens"] == sum(min(lens[i], 12) for i in idx)


# ---- sampling without replacement / unused first (App. E variants) ---------

def test_without_replacement_is_a_subset_of_distinct_slots_and_covers_all():
    got = ob.sample_without_replacement(seed=3, step=1, n_live=50, n_draw=20)
    assert len(got) == 20 and len(set(got)) == 20 and got == sorted(got)
    assert all(0 <= s < 50 for s in got)
    assert ob.sample_without_replacement(3, 1, 50, 50) == list(range(50))
    with pytest.raises(ValueError):
        ob.sample_without_replacement(3, 1, 5, 6)


def test_without_replacement_single_draw_is_the_smallest_key():
    keys = [philox.philox4x64((s, 7, 1, 0), (9, 0))[0] >> 1 for s in range(300)]
    assert ob.sample_without_replacement(9, 7, 300, 1) == [int(np.argmin(keys))]


def test_without_replacement_inclusion_is_uniform():
    # every slot is in a B-subset with probability B / n: inclusion counts over
    # many steps follow a uniform multinomial
    n_live, n_draw, steps = 40, 10, 2000
    counts = np.zeros(n_live)
    for step in range(steps):
        counts[ob.sample_without_replacement(21, step, n_live, n_draw)] += 1
    assert counts.sum() == n_draw * steps
    assert stats.chisquare(counts).pvalue > 1e-4


def test_unused_first_takes_never_used_records_ahead_of_used_ones():
    n_live = 60
    rng = np.random.default_rng(0)
    use = rng.integers(0, 3, n_live)
    unused = [s for s in range(n_live) if use[s] == 0]
    k = len(unused)
    assert 5 < k < 40
    # fewer draws than unused records: only unused ones, as a plain
    # without-replacement draw restricted to them would rank them
    few = ob.sample_without_replacement(4, 2, n_live, 5, use_count=use)
    assert set(few) <= set(unused)
    keys = {s: ob.slot_key(4, 2, s) for s in unused}
    assert few == sorted(sorted(unused, key=lambda s: (keys[s], s))[:5])
    # more draws than unused records: all unused ones plus used ones
    many = ob.sample_without_replacement(4, 2, n_live, k + 7, use_count=use)
    assert set(unused) <= set(many) and len(many) == k + 7
    # nothing used (or everything used): the plain draw
    plain = ob.sample_without_replacement(4, 2, n_live, 13)
    assert ob.sample_without_replacement(4, 2, n_live, 13, use_count=[0] * n_live) == plain
    assert ob.sample_without_replacement(4, 2, n_live, 13, use_count=[5] * n_live) == plain


# ---- steps since last use (App. D.3) -----------------------------------------

def test_steps_since_last_use_paper_example(golden_dir):
    with open(os.path.join(golden_dir, "steps_since_last_use_example.json")) as f:
        ex = json.load(f)
    assert ob.steps_since_last_use([tuple(b) for b in ex["batches"]]) == ex["expected"]


def test_steps_since_last_use_brute_force():
    # against a scan of the whole sample history for each sample
    rng = np.random.default_rng(1)
    batches = [(int(step), list(rng.integers(0, 12, 6))) for step in sorted(
        rng.choice(100, 15, replace=False))]
    got = ob.steps_since_last_use(batches)
    history = []  # (step, rid) of every earlier sample, in order
    for (step, ids), vals in zip(batches, got):
        for rid, v in zip(ids, vals):
            prev = [s for s, r in history if r == rid]
            assert v == (-1 if not prev else step - prev[-1])
            history.append((step, rid))


def test_histogram_bins_by_hand():
    # since values with "new" = -1 in bin 0; the tail collects 5 and 9
    assert ob.histogram([-1, 0, 0, 2, 5, 9, -1], 5, lo=-1) == [2, 2, 0, 1, 2]
    assert ob.histogram([], 3) == [0, 0, 0]
    assert ob.histogram([3, -4, 1], 1) == [3]
    vals = np.random.default_rng(0).integers(-3, 40, 1000)
    h = ob.histogram(vals, 12, lo=-2)
    assert sum(h) == 1000
    assert h[0] == int(np.sum(vals <= -2)) and h[-1] == int(np.sum(vals >= 9))
    assert h[5] == int(np.sum(vals == 3))


def test_replay_ratios_by_hand():
    # capacity 3: push 2, use slot 0 twice and slot 1; push 2 (evicts the first,
    # used twice), use slots 0 and 2; push 1 (evicts the second, used twice)
    ev, live = ob.replay_ratios(3, [(2, [0, 0, 1]), (2, [0, 2]), (1, [])])
    assert ev == [2, 2] and live == [0, 1, 0]


def test_replay_ratios_conserve_draws():
    rng = np.random.default_rng(1)
    steps, total = [], 0
    for _ in range(50):
        n_new = int(rng.integers(0, 6))
        n_live = min(20, sum(s[0] for s in steps) + n_new)
        draws = rng.integers(0, n_live, int(rng.integers(0, 9))).tolist() if n_live else []
        steps.append((n_new, draws))
        total += len(draws)
    ev, live = ob.replay_ratios(20, steps)
    assert sum(ev) + sum(live) == total
    assert len(ev) + len(live) == sum(s[0] for s in steps) and len(live) == 20


def test_replay_ratio_mean_is_batch_over_inserts():
    # uniform draws with replacement: each record is drawn B/N times per step
    # in expectation (App. C.1) and stays N/R steps, so its replay ratio has
    # mean B/R
    N, R, B = 64, 8, 24
    rng = np.random.default_rng(2)
    steps = [(R, rng.integers(0, min(N, R * (k + 1)), B).tolist()) for k in range(4000)]
    ev, _ = ob.replay_ratios(N, steps)
    steady = ev[N:]
    assert abs(np.mean(steady) - B / R) < 0.03
