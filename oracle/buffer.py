"""Replay buffer, sampling rules and batch gather -- the plain CPU definition.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Paper passages followed:

* Sec. 3.1 and App. B ("BufferStructure"): the buffer is a list of trajectories
  with capacity N; ``push`` appends and, when full, evicts the oldest entry
  (first in, first out); sampling does not remove entries.
* Sec. 4 (synchronous analysis) and App. C.1: a minibatch of B draws is taken
  uniformly from the buffer *with replacement*; the pseudo-code's library call
  samples without replacement -- the analysis is followed here.
* Sec. 5 ("Further optimization") and App. D.4 ("Positive-bias sampling"): with
  coefficient delta the buffer keeps the freshest (1-delta)N rollouts and, among
  the rollouts not in that fresh part, the freshest delta*N correct ones; the
  sampler draws uniformly over what is kept.  delta = 0 is plain uniform.
  Pinned by the worked example of App. D.4, which the rule reproduces at
  delta = 0.5 (the example prints 0.75).
* Positive-prioritised mixture (p_pos): not in the paper.  A coin
  with probability p_pos picks the positive stratum, otherwise the draw is over
  all live records; with no positives the draw falls back to all records.

* Sampling variants compared in App. E (the "vanilla" / "No replacement" /
  "No replacement, at least once" figure): uniform *without* replacement, and
  the same after first taking records never used before.  Defined here as the
  B records with the smallest per-record random keys (a uniformly random
  B-subset), listed in slot order; "at least once" ranks never-used records
  ahead of used ones.
* Buffer statistics (Sec. 3.2, "Off-Policiness, Diversity, and Compute
  Efficiency"): off-policiness of a sample = steps since its rollout was
  generated; replay ratio of a rollout = number of gradient steps that used
  it over the run, final when the rollout leaves the buffer.  Kept as
  histograms of those integers.
* Steps-since-last-use (App. D.3, "Metrics"): samples are ordered batch by
  batch, in a random order inside a batch (here: draw order); a sample of a
  rollout seen for the first time is "new" (-1 here), any later one gets the
  number of gradient steps since that rollout's previous sample.  Pinned by
  the paper's worked example.

Record order: slot 0 is the oldest live record, slot n_live-1 the newest.  A
record is "positive" ("correct") when its reward is > 0 (binary rewards).

Random draws come from ``oracle.philox`` only; draw ``j`` of step ``step`` uses
its own counter block, so a draw depends on (seed, step, j) and the record
table and nothing else (this is what makes a resumed run repeat a step).

Parity: pinned (worked example, uniform/mixture identities, chi-square checks,
brute force on tiny tables) -- tests/test_oracle_buffer.py.
"""

import numpy as np

from . import philox

RB_UNIFORM = 0
RB_POS_MIX = 1
RB_POS_RETAIN = 2

LAYOUT_PACKED = 0
LAYOUT_PADDED = 1


class FifoBuffer:
    """List-backed FIFO replay buffer (App. B, "BufferStructure").

    ``push`` appends a record and evicts the oldest once ``capacity`` records
    are held; ``records`` lists the live records oldest first.
    """

    def __init__(self, capacity):
        if capacity < 1:
            raise ValueError("capacity must be >= 1")
        self.capacity = int(capacity)
        self.records = []

    def push(self, record):
        if len(self.records) >= self.capacity:
            self.records.pop(0)
        self.records.append(record)

    def __len__(self):
        return len(self.records)


def positive_slots(rewards):
    """Slots (ascending) whose reward is > 0."""
    return [s for s, r in enumerate(rewards) if r > 0]


def retained_set(rewards, n_fresh, n_pos_keep):
    """Slots kept by positive-bias retention (Sec. 5; App. D.4).

    The freshest ``n_fresh`` slots are kept; among the older slots, the
    freshest ``n_pos_keep`` positive ones are kept as well.  Returned in
    ascending slot order.  With too few positives the set is smaller than
    n_fresh + n_pos_keep.
    """
    n_live = len(rewards)
    first_fresh = max(n_live - int(n_fresh), 0)
    older_pos = [s for s in range(first_fresh) if rewards[s] > 0]
    keep = older_pos[len(older_pos) - min(int(n_pos_keep), len(older_pos)):]
    return keep + list(range(first_fresh, n_live))


def retain_split(n_buffer, delta):
    """Host split of a buffer of size N at coefficient delta: floor(delta*N)
    positive slots, the rest fresh."""
    n_pos_keep = int(np.floor(delta * n_buffer))
    return n_buffer - n_pos_keep, n_pos_keep


def sample_indices(rewards, mode, seed, step, n_draw, p_q32=0, n_fresh=0,
                   n_pos_keep=0):
    """Slot indices of ``n_draw`` draws, with replacement, in draw order."""
    n_live = len(rewards)
    if n_live < 1:
        raise ValueError("cannot sample from an empty buffer")
    if mode == RB_UNIFORM:
        pool = None
    elif mode == RB_POS_MIX:
        pos = positive_slots(rewards)
    elif mode == RB_POS_RETAIN:
        pool = retained_set(rewards, n_fresh, n_pos_keep)
        if not pool:
            raise ValueError("retained set is empty")
    else:
        raise ValueError("unknown sampling mode")
    out = []
    for j in range(n_draw):
        x0, x1, _, _ = philox.draw_block(seed, step, j)
        if mode == RB_UNIFORM:
            out.append(philox.uniform_index(x0, n_live))
        elif mode == RB_POS_MIX:
            if pos and philox.coin(x1, p_q32):
                out.append(pos[philox.uniform_index(x0, len(pos))])
            else:
                out.append(philox.uniform_index(x0, n_live))
        else:
            out.append(pool[philox.uniform_index(x0, len(pool))])
    return out


def slot_key(seed, step, s):
    """63-bit random key of slot ``s`` at sampling step ``step``: the first
    word of the Philox4x64-10 block with counter (s, step, 1, 0) and key
    (seed, 0), shifted right by one bit."""
    return philox.philox4x64((s, step, 1, 0), (seed, 0))[0] >> 1


def sample_without_replacement(seed, step, n_live, n_draw, use_count=None):
    """``n_draw`` distinct slots, ascending.  Plain: the slots with the
    ``n_draw`` smallest (key, slot) pairs.  With ``use_count`` ("at least
    once"): slots never used before rank ahead of used ones, i.e. the order is
    by (used, key, slot)."""
    if not 1 <= n_draw <= n_live:
        raise ValueError("need 1 <= n_draw <= n_live without replacement")
    rank = []
    for s in range(n_live):
        used = 0 if use_count is None else int(use_count[s] > 0)
        rank.append((used, slot_key(seed, step, s), s))
    rank.sort()
    return sorted(r[2] for r in rank[:n_draw])


def steps_since_last_use(batches):
    """``batches``: list of (step, rollout ids in draw order), in processing
    order.  Returns one list per batch: -1 for a rollout's first sample, else
    the steps since its previous sample (0 for a repeat inside a batch)."""
    last = {}
    out = []
    for step, ids in batches:
        vals = []
        for rid in ids:
            vals.append(-1 if rid not in last else step - last[rid])
            last[rid] = step
        out.append(vals)
    return out


def histogram(values, n_bins, lo=0):
    """Counts of integers in ``n_bins`` bins: value v lands in bin v - lo,
    values below ``lo`` in the first bin and values past the last bin in the
    last one.  The buffer statistics of Sec. 3.2 are distributions of small
    integers: off-policiness (a sample's age in steps), replay ratio (how
    often a rollout is used) and steps since last use, where lo = -1 gives
    "new" (-1) the first bin."""
    if n_bins < 1:
        raise ValueError("n_bins must be >= 1")
    h = [0] * n_bins
    for v in values:
        h[min(max(int(v) - lo, 0), n_bins - 1)] += 1
    return h


def replay_ratios(capacity, steps):
    """Replay ratio of each rollout (Sec. 3.2: the number of gradient steps
    that used it) in a FIFO buffer of ``capacity`` records.

    ``steps``: list of (n_new, draws) in processing order; each step first
    pushes ``n_new`` fresh rollouts (evicting the oldest ones past the
    capacity), then uses the records at slots ``draws`` (0 = oldest live
    record, with repeats counting once per draw).  Returns (use counts of the
    evicted rollouts in eviction order, use counts of the live ones oldest
    first)."""
    live, evicted = [], []
    for n_new, draws in steps:
        for _ in range(int(n_new)):
            if len(live) == capacity:
                evicted.append(live.pop(0))
            live.append(0)
        for s in draws:
            live[s] += 1
    return evicted, live


def gather(idx, rec_off, rec_len, rec_adv, rec_version, arena_tokens,
           arena_old_logp, cur_version, layout, max_tokens=0, token_begin=0,
           l_max=0):
    """Assemble the training batch of the drawn records, in draw order.

    Duplicated draws are kept (sampling is with replacement).  Packed layout:
    the drawn sequences are concatenated into one token stream; this call
    returns the window [token_begin, token_begin + max_tokens) of it (a
    micro-batch), padding positions past the end of the stream.  A sequence
    cut by the window keeps its full length for weighting.  Padded layout: row
    j holds the first min(len_j, l_max) tokens of draw j.

    Returns a dict of numpy arrays: idx, adv, len, age (per draw),
    cu_seqlens (packed: prefix sums of full lengths over the whole stream;
    padded: row starts), tokens, old_logp, seq_of_token (-1 on padding) and
    n_tokens (valid positions in the output).
    """
    idx = np.asarray(idx, dtype=np.int64)
    n_draw = len(idx)
    lens = np.asarray(rec_len, dtype=np.int64)[idx]
    offs = np.asarray(rec_off, dtype=np.int64)[idx]
    out = {
        "idx": idx.astype(np.int32),
        "adv": np.asarray(rec_adv, dtype=np.float32)[idx],
        "len": lens.astype(np.int32),
        "age": (int(cur_version)
                - np.asarray(rec_version, dtype=np.int64)[idx]).astype(np.int32),
    }
    if layout == LAYOUT_PACKED:
        cu = np.zeros(n_draw + 1, dtype=np.int64)
        for j in range(n_draw):
            cu[j + 1] = cu[j] + lens[j]
        tokens = np.zeros(max_tokens, dtype=np.int32)
        old = np.zeros(max_tokens, dtype=np.float32)
        seq = np.full(max_tokens, -1, dtype=np.int32)
        n_valid = 0
        for j in range(n_draw):
            for p in range(int(lens[j])):
                t = int(cu[j]) + p - token_begin
                if 0 <= t < max_tokens:
                    tokens[t] = arena_tokens[offs[j] + p]
                    old[t] = arena_old_logp[offs[j] + p]
                    seq[t] = j
                    n_valid += 1
        out["cu_seqlens"] = cu.astype(np.int32)
    elif layout == LAYOUT_PADDED:
        tokens = np.zeros((n_draw, l_max), dtype=np.int32)
        old = np.zeros((n_draw, l_max), dtype=np.float32)
        seq = np.full((n_draw, l_max), -1, dtype=np.int32)
        n_valid = 0
        for j in range(n_draw):
            for p in range(min(int(lens[j]), l_max)):
                tokens[j, p] = arena_tokens[offs[j] + p]
                old[j, p] = arena_old_logp[offs[j] + p]
                seq[j, p] = j
                n_valid += 1
        out["cu_seqlens"] = (np.arange(n_draw + 1, dtype=np.int64)
                             * l_max).astype(np.int32)
    else:
        raise ValueError("unknown layout")
    out["tokens"] = tokens
    out["old_logp"] = old
    out["seq_of_token"] = seq
    out["n_tokens"] = n_valid
    return out
